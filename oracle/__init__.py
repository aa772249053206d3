"""fp64 CPU oracle for SONIC's segment-structured attention path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this
package.  The HIP library never links, imports or falls back to it, and the
oracle shares no code with the HIP path: both read the same seeded inputs
from ``workloads.py`` and nothing else.

The method reaches results with plain definitions (a masked softmax
attention, a filter, attention over the filtered set), so the oracle writes
those definitions out, slowly and in float64:

* ``layout``     - the augmented-sequence grammar of Eq.(1) (Sec. 3.1) and the
                   per-segment index sets B_i, N_i of Sec. 3.2.
* ``mask``       - the explicit L x L visibility matrix from the three rules of
                   Sec. 3.2, Eqs.(3)-(5).
* ``attention``  - dense softmax attention under that mask (Sec. 3.2 with the
                   standard scaled dot product), fp64.
* ``compaction`` - the KV retention rule: keep system, Nexus and current-query
                   entries (Sec. 3, Fig. 2 caption; Sec. 3.2 Rule 2; App. C).
* ``decode``     - generation over the retained context {I_sys, N, Q_n}
                   (App. C, Eq.(15)) and the same step over the full cache with
                   the mask applied.
* ``extend``     - the next turn's Nexus rows over the compact cache (Sec. 3.2
                   mask restricted to the newest segment) and the cache update
                   that drops the turn's body and keeps its Nexus KV.
* ``stats``      - attention statistics behind the training objectives of
                   Sec. 4: the Nexus attention mass per query row and head, and
                   the head-averaged attention each key receives from the
                   current rows.
* ``projection`` - the role-routed linear layer: Nexus tokens use their own
                   projection matrices, every other token the standard ones
                   (Sec. 3.1).
* ``recon``      - the reconstruction targets of the information bottleneck
                   (Sec. 4): per Nexus token, a cosine-softmax pooling of its
                   body sub-interval, with the target's cosine and the
                   normalised entropy of the weights.

Inputs are bf16 bit patterns (uint16); they are widened exactly to float64.
"""
from . import layout, mask, attention, compaction, decode, extend, stats, projection, recon  # noqa: F401


