"""Python binding of libsonic.so: argument marshalling only.

Every function here forwards torch tensors' device pointers, sizes and the
current HIP stream to the C entry point of the same name (see include/sonic.h)
and returns its status code.  No arithmetic of the path happens in Python, and
there is no fallback: if the library is missing or no GPU is present, calls
raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch  # loads the HIP runtime the library shares with torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsonic.so")

OK = 0
ERR_INVALID_ARG = 1
ERR_BAD_LAYOUT = 2
ERR_CAPACITY = 3
ERR_WORKSPACE = 4
ERR_UNSUPPORTED = 5
ERR_HIP = 6

ROLE_SYSTEM, ROLE_HISTORY_TEXT, ROLE_NEXUS, ROLE_CURRENT = 0, 1, 2, 3
NEXUS_ALL, NEXUS_UP_TO_OWN = 0, 1   # Nexus <-> Nexus visibility scope of the prefill mask

EXPORTS = (
    "sonic_abi_version", "sonic_status_string", "sonic_validate_layout_host", "sonic_layout_stats_host",
    "sonic_prefill_workspace_bytes", "sonic_segment_attn_prefill", "sonic_kv_compact",
    "sonic_decode_workspace_bytes", "sonic_compressed_decode", "sonic_compressed_decode_noalloc",
    "sonic_nexus_extend_workspace_bytes",
    "sonic_nexus_extend", "sonic_role_projection_workspace_bytes", "sonic_role_projection",
    "sonic_nexus_recon_workspace_bytes", "sonic_nexus_recon_targets",
)

_lib = None

_i32, _i64, _f32, _sz, _p = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t, ctypes.c_void_p


class SonicError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {status_string(code)} ({code})")


def lib() -> ctypes.CDLL:
    """Load libsonic.so once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2601_21927_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    L.sonic_abi_version.restype = _i32
    L.sonic_abi_version.argtypes = []
    L.sonic_status_string.restype = ctypes.c_char_p
    L.sonic_status_string.argtypes = [_i32]
    L.sonic_validate_layout_host.restype = _i32
    L.sonic_validate_layout_host.argtypes = [_i32, _p, _p, _p, _p]
    L.sonic_layout_stats_host.restype = _i32
    L.sonic_layout_stats_host.argtypes = [_i32, _p, _p, _p, _i32, _p, _p]
    L.sonic_prefill_workspace_bytes.restype = _sz
    L.sonic_prefill_workspace_bytes.argtypes = [_i32, _i32, _i32, _i32, _i32]
    L.sonic_segment_attn_prefill.restype = _i32
    L.sonic_segment_attn_prefill.argtypes = [_i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _p, _p, _f32, _i32, _p,
                                             _p, _p, _p, _sz, _p, _p]
    L.sonic_kv_compact.restype = _i32
    L.sonic_kv_compact.argtypes = [_i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p]
    L.sonic_decode_workspace_bytes.restype = _sz
    L.sonic_decode_workspace_bytes.argtypes = [_i32, _i32, _i32, _i32]
    L.sonic_compressed_decode.restype = _i32
    L.sonic_compressed_decode.argtypes = [_i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _p, _p, _p, _p, _p, _f32,
                                          _p, _p, _sz, _p, _p]
    L.sonic_compressed_decode_noalloc.restype = _i32
    L.sonic_compressed_decode_noalloc.argtypes = [_i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _p, _p, _p, _p, _p,
                                                  _f32, _p, _p, _p]
    L.sonic_nexus_extend_workspace_bytes.restype = _sz
    L.sonic_nexus_extend_workspace_bytes.argtypes = [_i32, _i32, _i32, _i32, _i32]
    L.sonic_nexus_extend.restype = _i32
    L.sonic_nexus_extend.argtypes = [_i32, _i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p,
                                     _f32, _p, _p, _sz, _p, _p]
    L.sonic_role_projection_workspace_bytes.restype = _sz
    L.sonic_role_projection_workspace_bytes.argtypes = [_i32]
    L.sonic_role_projection.restype = _i32
    L.sonic_role_projection.argtypes = [_i32, _i32, _i32, _p, _p, _p, _p, _p, _p, _sz, _p, _p]
    L.sonic_nexus_recon_workspace_bytes.restype = _sz
    L.sonic_nexus_recon_workspace_bytes.argtypes = [_i32, _i32]
    L.sonic_nexus_recon_targets.restype = _i32
    L.sonic_nexus_recon_targets.argtypes = [_i32, _i32, _i32, _p, _p, _p, _p, _i32, _p, _p, _p, _p, _sz, _p, _p]
    _lib = L
    return L


def status_string(code: int) -> str:
    return lib().sonic_status_string(int(code)).decode()


def abi_version() -> int:
    return int(lib().sonic_abi_version())


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libsonic must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _np_ptr(a):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dev(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("libsonic GPU entry points take device tensors")


_I32, _I64, _U8, _BF16, _F32 = torch.int32, torch.int64, torch.uint8, torch.bfloat16, torch.float32


def _types(**named):
    """named=(tensor, dtype): the C ABI reads raw memory, so a wrong element type is refused here."""
    for name, (t, dt) in named.items():
        if t is not None and t.dtype != dt:
            raise TypeError(f"{name} must be {dt}, got {t.dtype}")


# ----------------------------------------------------------------- host helpers
def validate_layout_host(cu_seqlens, role, turn_id):
    """(status, first bad request) for numpy int32 cu, uint8 role, int32 turn_id."""
    import numpy as np
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    r = np.ascontiguousarray(role, dtype=np.uint8)
    t = np.ascontiguousarray(turn_id, dtype=np.int32)
    bad = ctypes.c_int32(-1)
    st = lib().sonic_validate_layout_host(len(cu) - 1, _np_ptr(cu), _np_ptr(r), _np_ptr(t), ctypes.byref(bad))
    return int(st), int(bad.value)


def layout_stats_host(cu_seqlens, role, turn_id, nexus_scope: int = NEXUS_ALL):
    """(visible pairs per request int64[B], kept rows per request int32[B])."""
    import numpy as np
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
    r = np.ascontiguousarray(role, dtype=np.uint8)
    t = np.ascontiguousarray(turn_id, dtype=np.int32)
    B = len(cu) - 1
    vis = np.zeros(max(B, 1), np.int64)
    kept = np.zeros(max(B, 1), np.int32)
    st = lib().sonic_layout_stats_host(B, _np_ptr(cu), _np_ptr(r), _np_ptr(t), int(nexus_scope), _np_ptr(vis),
                                       _np_ptr(kept))
    if st != OK:
        raise SonicError(st, "sonic_layout_stats_host")
    return vis[:B], kept[:B]


# ----------------------------------------------------------------- step 1: prefill
def prefill_workspace_bytes(batch: int, total_tokens: int, num_q_heads: int, num_kv_heads: int, head_dim: int) -> int:
    return int(lib().sonic_prefill_workspace_bytes(batch, total_tokens, num_q_heads, num_kv_heads, head_dim))


def segment_attn_prefill(cu_seqlens, role, turn_id, q, k, v, out, workspace, dev_status, softmax_scale=None,
                         nexus_scope: int = NEXUS_ALL, nexus_mass=None, key_weight=None, stream=None) -> int:
    """q [T,Hq,d] bf16, k/v [T,Hkv,d] bf16, out [T,Hq,d] fp32; cu int32 [B+1]; role uint8 [T];
    turn_id int32 [T]; workspace uint8 [>= prefill_workspace_bytes]; dev_status int32 [1];
    optional statistics nexus_mass fp32 [T,Hq] and key_weight fp32 [T]."""
    _dev(cu_seqlens, role, turn_id, q, k, v, out, workspace, dev_status, nexus_mass, key_weight)
    _types(cu_seqlens=(cu_seqlens, _I32), role=(role, _U8), turn_id=(turn_id, _I32), q=(q, _BF16), k=(k, _BF16),
           v=(v, _BF16), out=(out, _F32), dev_status=(dev_status, _I32), nexus_mass=(nexus_mass, _F32),
           key_weight=(key_weight, _F32))
    T, Hq, d = q.shape
    Hkv = k.shape[1]
    scale = 0.0 if softmax_scale is None else float(softmax_scale)   # 0: the library's 1/sqrt(d)
    return int(lib().sonic_segment_attn_prefill(
        cu_seqlens.numel() - 1, T, Hq, Hkv, d, _ptr(cu_seqlens), _ptr(role), _ptr(turn_id), _ptr(q), _ptr(k),
        _ptr(v), scale, int(nexus_scope), _ptr(out), _ptr(nexus_mass), _ptr(key_weight), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(dev_status), _stream(stream)))


# ----------------------------------------------------------------- step 2: compaction
def kv_compact(cu_seqlens, role, k, v, k_cache, v_cache, cache_row_off, cache_row_cap, cache_len, keep_idx,
               dev_status, max_seqlen: int, stream=None) -> int:
    """k/v [T,Hkv,d] bf16 -> k_cache/v_cache [rows,Hkv,d]; cache_row_off int64 [B]; cache_row_cap int32 [B];
    cache_len int32 [B]; keep_idx int32 [rows]."""
    _dev(cu_seqlens, role, k, v, k_cache, v_cache, cache_row_off, cache_row_cap, cache_len, keep_idx, dev_status)
    _types(cu_seqlens=(cu_seqlens, _I32), role=(role, _U8), k=(k, _BF16), v=(v, _BF16), k_cache=(k_cache, _BF16),
           v_cache=(v_cache, _BF16), cache_row_off=(cache_row_off, _I64), cache_row_cap=(cache_row_cap, _I32),
           cache_len=(cache_len, _I32), keep_idx=(keep_idx, _I32), dev_status=(dev_status, _I32))
    T, Hkv, d = k.shape
    return int(lib().sonic_kv_compact(
        cu_seqlens.numel() - 1, T, int(max_seqlen), Hkv, d, _ptr(cu_seqlens), _ptr(role), _ptr(k), _ptr(v),
        _ptr(k_cache), _ptr(v_cache), _ptr(cache_row_off), _ptr(cache_row_cap), _ptr(cache_len), _ptr(keep_idx),
        _ptr(dev_status), _stream(stream)))


# ----------------------------------------------------------------- step 3: decode
def decode_workspace_bytes(batch: int, num_q_heads: int, head_dim: int, max_ctx: int) -> int:
    return int(lib().sonic_decode_workspace_bytes(batch, num_q_heads, head_dim, max_ctx))


def compressed_decode(k_cache, v_cache, cache_row_off, cache_row_cap, cache_len, q, k_new, v_new, out, workspace,
                      dev_status, max_ctx: int, row_role=None, softmax_scale=None, stream=None) -> int:
    """q [B,Hq,d] bf16; k_new/v_new [B,Hkv,d] bf16; out [B,Hq,d] fp32; row_role uint8 [rows] or None."""
    _dev(k_cache, v_cache, cache_row_off, cache_row_cap, cache_len, q, k_new, v_new, out, workspace, dev_status,
         row_role)
    _types(k_cache=(k_cache, _BF16), v_cache=(v_cache, _BF16), cache_row_off=(cache_row_off, _I64),
           cache_row_cap=(cache_row_cap, _I32), cache_len=(cache_len, _I32), q=(q, _BF16), k_new=(k_new, _BF16),
           v_new=(v_new, _BF16), out=(out, _F32), dev_status=(dev_status, _I32), row_role=(row_role, _U8))
    B, Hq, d = q.shape
    Hkv = k_new.shape[1]
    scale = 0.0 if softmax_scale is None else float(softmax_scale)   # 0: the library's 1/sqrt(d)
    return int(lib().sonic_compressed_decode(
        B, Hq, Hkv, d, int(max_ctx), _ptr(k_cache), _ptr(v_cache), _ptr(cache_row_off), _ptr(cache_row_cap),
        _ptr(cache_len), _ptr(row_role), _ptr(q), _ptr(k_new), _ptr(v_new), scale, _ptr(out), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(dev_status), _stream(stream)))


def compressed_decode_noalloc(k_cache, v_cache, cache_row_off, cache_row_cap, cache_len, q, k_new, v_new, out,
                              dev_status, max_ctx: int, row_role=None, softmax_scale=None, stream=None) -> int:
    """compressed_decode without a workspace: the library's fixed per-GPU scratch is used."""
    _dev(k_cache, v_cache, cache_row_off, cache_row_cap, cache_len, q, k_new, v_new, out, dev_status, row_role)
    _types(k_cache=(k_cache, _BF16), v_cache=(v_cache, _BF16), cache_row_off=(cache_row_off, _I64),
           cache_row_cap=(cache_row_cap, _I32), cache_len=(cache_len, _I32), q=(q, _BF16), k_new=(k_new, _BF16),
           v_new=(v_new, _BF16), out=(out, _F32), dev_status=(dev_status, _I32), row_role=(row_role, _U8))
    B, Hq, d = q.shape
    Hkv = k_new.shape[1]
    scale = 0.0 if softmax_scale is None else float(softmax_scale)   # 0: the library's 1/sqrt(d)
    return int(lib().sonic_compressed_decode_noalloc(
        B, Hq, Hkv, d, int(max_ctx), _ptr(k_cache), _ptr(v_cache), _ptr(cache_row_off), _ptr(cache_row_cap),
        _ptr(cache_len), _ptr(row_role), _ptr(q), _ptr(k_new), _ptr(v_new), scale, _ptr(out), _ptr(dev_status),
        _stream(stream)))


# ----------------------------------------------------------------- next turn: Nexus step
def nexus_extend_workspace_bytes(batch: int, total_new: int, max_rows: int, num_kv_heads: int,
                                 head_dim: int) -> int:
    return int(lib().sonic_nexus_extend_workspace_bytes(batch, total_new, max_rows, num_kv_heads, head_dim))


def nexus_extend(nexus_cu, keep_len, k_cache, v_cache, cache_row_off, cache_row_cap, cache_len, q, k, v, out,
                 workspace, dev_status, max_rows: int, body_len=None, softmax_scale=None, stream=None) -> int:
    """nexus_cu int32 [B+1]; keep_len int32 [B]; body_len int32 [B] or None (the whole tail);
    q [N,Hq,d] bf16; k/v [N,Hkv,d] bf16; out [N,Hq,d] fp32."""
    _dev(nexus_cu, keep_len, body_len, k_cache, v_cache, cache_row_off, cache_row_cap, cache_len, q, k, v, out,
         workspace, dev_status)
    _types(nexus_cu=(nexus_cu, _I32), keep_len=(keep_len, _I32), body_len=(body_len, _I32),
           k_cache=(k_cache, _BF16), v_cache=(v_cache, _BF16), cache_row_off=(cache_row_off, _I64),
           cache_row_cap=(cache_row_cap, _I32), cache_len=(cache_len, _I32), q=(q, _BF16), k=(k, _BF16),
           v=(v, _BF16), out=(out, _F32), dev_status=(dev_status, _I32))
    N, Hq, d = q.shape
    Hkv = k.shape[1]
    scale = 0.0 if softmax_scale is None else float(softmax_scale)   # 0: the library's 1/sqrt(d)
    return int(lib().sonic_nexus_extend(
        nexus_cu.numel() - 1, N, Hq, Hkv, d, int(max_rows), _ptr(nexus_cu), _ptr(keep_len), _ptr(body_len),
        _ptr(k_cache), _ptr(v_cache), _ptr(cache_row_off), _ptr(cache_row_cap), _ptr(cache_len), _ptr(q), _ptr(k),
        _ptr(v), scale, _ptr(out), _ptr(workspace), workspace.numel() * workspace.element_size(), _ptr(dev_status),
        _stream(stream)))


# ----------------------------------------------------------------- role-routed projection
def role_projection_workspace_bytes(total_tokens: int) -> int:
    return int(lib().sonic_role_projection_workspace_bytes(total_tokens))


def role_projection(role, x, w_text, w_nexus, y, workspace, dev_status, stream=None) -> int:
    """role uint8 [T]; x [T,K] bf16; w_text / w_nexus [N,K] bf16; y [T,N] fp32 (Nexus rows use w_nexus)."""
    _dev(role, x, w_text, w_nexus, y, workspace, dev_status)
    _types(role=(role, _U8), x=(x, _BF16), w_text=(w_text, _BF16), w_nexus=(w_nexus, _BF16), y=(y, _F32),
           dev_status=(dev_status, _I32))
    T, K = x.shape
    N = w_text.shape[0]
    if tuple(w_nexus.shape) != (N, K) or tuple(w_text.shape) != (N, K) or tuple(y.shape) != (T, N) or \
            role.numel() != T:
        raise ValueError("role_projection: inconsistent shapes")
    return int(lib().sonic_role_projection(
        T, K, N, _ptr(role), _ptr(x), _ptr(w_text), _ptr(w_nexus), _ptr(y), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(dev_status), _stream(stream)))


# ----------------------------------------------------------------- reconstruction targets
def nexus_recon_workspace_bytes(batch: int, total_tokens: int) -> int:
    return int(lib().sonic_nexus_recon_workspace_bytes(batch, total_tokens))


def nexus_recon_targets(cu_seqlens, role, turn_id, h, target, cos_target, entropy_ratio, workspace, dev_status,
                        stream=None) -> int:
    """h [T,Dm] bf16; target [n,Dm] fp32, cos_target [n] fp32, entropy_ratio [n] fp32 with n >= the
    batch's Nexus count (rows in packed position order)."""
    _dev(cu_seqlens, role, turn_id, h, target, cos_target, entropy_ratio, workspace, dev_status)
    _types(cu_seqlens=(cu_seqlens, _I32), role=(role, _U8), turn_id=(turn_id, _I32), h=(h, _BF16),
           target=(target, _F32), cos_target=(cos_target, _F32), entropy_ratio=(entropy_ratio, _F32),
           dev_status=(dev_status, _I32))
    T, Dm = h.shape
    n = target.shape[0]
    if target.shape[1] != Dm or cos_target.numel() < n or entropy_ratio.numel() < n:
        raise ValueError("nexus_recon_targets: inconsistent output shapes")
    return int(lib().sonic_nexus_recon_targets(
        cu_seqlens.numel() - 1, T, Dm, _ptr(cu_seqlens), _ptr(role), _ptr(turn_id), _ptr(h), n, _ptr(target),
        _ptr(cos_target), _ptr(entropy_ratio), _ptr(workspace), workspace.numel() * workspace.element_size(),
        _ptr(dev_status), _stream(stream)))
