"""Device-memory plumbing around the three entry points.

`SonicBatch` owns the device tensors of one packed batch (inputs, outputs,
workspaces, the compact cache and the status word) and calls the C ABI
through `sonic`.  torch is used only to allocate memory and to provide the
stream; every step of the path runs in libsonic.so.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np
import torch

from . import sonic


def bf16_to_device(bits: np.ndarray, device="cuda") -> torch.Tensor:
    """Upload raw bf16 bit patterns (uint16) as a bfloat16 tensor, unchanged."""
    a = np.ascontiguousarray(bits, dtype=np.uint16)
    return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)


def bf16_to_host(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def check(code: int, where: str):
    if code != sonic.OK:
        raise sonic.SonicError(code, where)


class SonicBatch:
    """One packed batch on the device.

    role uint8 [T], turn_id int32 [T], cu_seqlens int32 [B+1], q/k/v bf16 bits.
    """

    def __init__(self, role, turn_id, cu_seqlens, q_bits, k_bits, v_bits, device="cuda"):
        self.device = torch.device(device)
        self.cu_host = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
        self.batch = len(self.cu_host) - 1
        self.total_tokens = int(self.cu_host[-1])
        self.lengths = np.diff(self.cu_host)
        self.max_seqlen = int(self.lengths.max()) if self.batch else 0
        self.role = torch.from_numpy(np.ascontiguousarray(role, dtype=np.uint8)).to(self.device)
        self.turn_id = torch.from_numpy(np.ascontiguousarray(turn_id, dtype=np.int32)).to(self.device)
        self.cu = torch.from_numpy(self.cu_host).to(self.device)
        self.k = bf16_to_device(k_bits, self.device)
        self.v = bf16_to_device(v_bits, self.device)
        self.T, self.Hkv, self.d = self.k.shape
        self.status = torch.zeros(1, dtype=torch.int32, device=self.device)
        # a decode-only batch has no prefill queries
        self.q = None if q_bits is None else bf16_to_device(q_bits, self.device)
        self.Hq = 0 if self.q is None else self.q.shape[1]
        self.out = None if self.q is None else torch.empty((self.T, self.Hq, self.d), dtype=torch.float32,
                                                           device=self.device)
        ws = sonic.prefill_workspace_bytes(self.batch, self.total_tokens, max(self.Hq, 1), self.Hkv, self.d)
        self.prefill_ws = torch.empty(max(ws, 256), dtype=torch.uint8, device=self.device)
        self.cache = None

    # ------------------------------------------------------------- step 1
    def prefill(self, stream=None, nexus_scope: int = sonic.NEXUS_ALL, nexus_mass=None, key_weight=None) -> int:
        return sonic.segment_attn_prefill(self.cu, self.role, self.turn_id, self.q, self.k, self.v, self.out,
                                          self.prefill_ws, self.status, nexus_scope=nexus_scope,
                                          nexus_mass=nexus_mass, key_weight=key_weight, stream=stream)

    # ------------------------------------------------------------- step 2
    def alloc_cache(self, capacities: Sequence[int], fill_bits: int = 0xFFFF):
        cap = np.asarray(capacities, dtype=np.int64)
        off = np.concatenate([[0], np.cumsum(cap)[:-1]]).astype(np.int64)
        rows = int(cap.sum())
        self.cache = CompactCache(rows, self.Hkv, self.d, off, cap.astype(np.int32), self.device, fill_bits)
        return self.cache

    def compact(self, stream=None) -> int:
        c = self.cache
        return sonic.kv_compact(self.cu, self.role, self.k, self.v, c.k, c.v, c.row_off, c.row_cap, c.length,
                                c.keep_idx, self.status, self.max_seqlen, stream=stream)

    def read_status(self) -> int:
        return int(self.status.item())

    def clear_status(self):
        self.status.zero_()


class CompactCache:
    """Per-request cache rows [row_off[b], row_off[b] + row_cap[b]) of a [rows, Hkv, d] bf16 pair."""

    def __init__(self, rows, Hkv, d, row_off, row_cap, device, fill_bits=0xFFFF):
        self.rows, self.Hkv, self.d = rows, Hkv, d
        fill = np.int16(np.uint16(fill_bits).view(np.int16))
        self.k = torch.full((max(rows, 1), Hkv, d), int(fill), dtype=torch.int16, device=device).view(torch.bfloat16)
        self.v = torch.full((max(rows, 1), Hkv, d), int(fill), dtype=torch.int16, device=device).view(torch.bfloat16)
        self.keep_idx = torch.full((max(rows, 1),), -1, dtype=torch.int32, device=device)
        self.row_off_host = np.asarray(row_off, dtype=np.int64)
        self.row_cap_host = np.asarray(row_cap, dtype=np.int32)
        self.row_off = torch.from_numpy(self.row_off_host).to(device)
        self.row_cap = torch.from_numpy(self.row_cap_host).to(device)
        self.length = torch.zeros(len(row_cap), dtype=torch.int32, device=device)
        self.batch = len(row_cap)
        self.ws = None
        self.ws_key = None

    def decode(self, q, k_new, v_new, out, status, max_ctx: int, row_role: Optional[torch.Tensor] = None,
               stream=None) -> int:
        B, Hq, d = q.shape
        Hkv = k_new.shape[1]
        key = (B, Hq, Hkv, d, int(max_ctx))
        if self.ws_key != key:
            n = sonic.decode_workspace_bytes(B, Hq, d, int(max_ctx))
            self.ws = torch.zeros(max(n, 256), dtype=torch.uint8, device=q.device)   # counters start at zero
            self.ws_key = key
        return sonic.compressed_decode(self.k, self.v, self.row_off, self.row_cap, self.length, q, k_new, v_new,
                                       out, self.ws, status, max_ctx, row_role=row_role, stream=stream)
