"""Generation over the retained context (oracle; test infrastructure only).

App. C, Eq.(15): the response R_n is generated from {I_sys, N, Q_n} only.  A
generated token belongs to the current turn (reading A8), so its mask row is
exactly "every retained entry, every earlier generated token and itself".

Two definitions are kept side by side:
* ``decode_step``          - attention of one new query over a cache whose rows
                             are all visible (the compact cache plus the new row);
* ``masked_decode_step``   - the same query over the full, uncompacted cache with
                             the mask applied (history body rows excluded by
                             Eq.(4), everything else visible).
In exact arithmetic the two agree; the test suite checks that.
"""
from __future__ import annotations

import numpy as np

from .attention import bf16_bits_to_f64, kv_head
from .layout import HISTORY_TEXT


def _attend(qf, kf, vf, visible, scale):
    """qf [Hq, d]; kf, vf [n, Hkv, d]; visible bool [n] -> out [Hq, d] (float64)."""
    Hq, d = qf.shape
    Hkv = kf.shape[1]
    out = np.zeros((Hq, d), dtype=np.float64)
    for h in range(Hq):
        g = kv_head(h, Hq, Hkv)
        s = scale * (kf[:, g, :] @ qf[h])
        s = np.where(visible, s, -np.inf)
        m = s.max()
        e = np.where(visible, np.exp(s - m), 0.0)
        out[h] = (e / e.sum()) @ vf[:, g, :]
    return out


def decode_step(q_bits, k_ctx_bits, v_ctx_bits, k_new_bits, v_new_bits, scale=None):
    """One step: append (k_new, v_new) to the context, attend with every row visible."""
    qf = bf16_bits_to_f64(q_bits)
    kf = np.concatenate([bf16_bits_to_f64(k_ctx_bits), bf16_bits_to_f64(k_new_bits)[None]], axis=0)
    vf = np.concatenate([bf16_bits_to_f64(v_ctx_bits), bf16_bits_to_f64(v_new_bits)[None]], axis=0)
    if scale is None:
        scale = 1.0 / np.sqrt(qf.shape[1])
    return _attend(qf, kf, vf, np.ones(kf.shape[0], dtype=bool), scale)


def masked_decode_step(q_bits, k_full_bits, v_full_bits, role_full, k_new_bits, v_new_bits, scale=None):
    """One step over the full cache: rows whose role is history text are masked; the
    appended row and every non-text row are visible."""
    qf = bf16_bits_to_f64(q_bits)
    kf = np.concatenate([bf16_bits_to_f64(k_full_bits), bf16_bits_to_f64(k_new_bits)[None]], axis=0)
    vf = np.concatenate([bf16_bits_to_f64(v_full_bits), bf16_bits_to_f64(v_new_bits)[None]], axis=0)
    visible = np.concatenate([np.asarray(role_full) != HISTORY_TEXT, [True]])
    if scale is None:
        scale = 1.0 / np.sqrt(qf.shape[1])
    return _attend(qf, kf, vf, visible, scale)


def decode_run(q_steps, k_steps, v_steps, k_ctx_bits, v_ctx_bits, scale=None):
    """Several steps for one request: step t appends its k/v, then attends over all rows.
    q_steps [T, Hq, d], k_steps/v_steps [T, Hkv, d] (bf16 bits).  Returns [T, Hq, d]."""
    kc = np.asarray(k_ctx_bits)
    vc = np.asarray(v_ctx_bits)
    outs = []
    for t in range(len(q_steps)):
        outs.append(decode_step(q_steps[t], kc, vc, k_steps[t], v_steps[t], scale))
        kc = np.concatenate([kc, np.asarray(k_steps[t])[None]], axis=0)
        vc = np.concatenate([vc, np.asarray(v_steps[t])[None]], axis=0)
    return np.stack(outs)
