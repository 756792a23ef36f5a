"""WIDE token-level dynamic-width masked projections on MI355X (gfx950).

Thin Python binding over ``libwide.so`` (see ``include/wide.h``): the same
entry-point names, torch tensors in and out, the current HIP stream.  The
binding only marshals arguments (pointers, sizes, stream) and allocates
outputs/workspaces with torch when the caller does not pass them; every step
of the computation runs in the library's HIP kernels.  There is no fallback:
if the library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os

__all__ = [
    "WideError", "lib", "wide_mask_reorder", "wide_ffn_masked", "wide_qkvo_masked", "wide_router",
    "wide_attention_masked", "wide_attention_workspace_size", "wide_attention_decode",
    "wide_attention_decode_workspace_size", "wide_workspace_size", "wide_set_option", "wide_get_option", "wide_timing_enable",
    "wide_timing_reset", "wide_timing_query", "wide_timing_filter", "wide_ffn_masked_noalloc", "wide_static_scratch_bytes", "LIB_PATH",
    "OP_REORDER", "OP_FFN", "OP_QKV", "OP_O", "OP_ROUTER", "PHASE_QKV", "PHASE_O", "F32", "BF16",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libwide.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = range(5)
F32, BF16 = 0, 1
PHASE_QKV, PHASE_O = 0, 1
OP_REORDER, OP_FFN, OP_QKV, OP_O, OP_ROUTER = 0, 1, 2, 3, 4
SIZE_MAX = 2 ** 64 - 1

_lib = None


class WideError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn} failed with status {status}: {msg}")
        self.status = status


def lib() -> ctypes.CDLL:
    """Load libwide.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing; build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, i32, ci, sz = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                ctypes.c_int, ctypes.c_size_t)
        L.wide_last_error.restype = ctypes.c_char_p
        L.wide_last_error.argtypes = []
        L.wide_mask_reorder.restype = ci
        L.wide_mask_reorder.argtypes = [vp, i64, i32, vp, vp, vp, sz, vp]
        L.wide_ffn_masked.restype = ci
        L.wide_ffn_masked.argtypes = [ci, i64, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                      vp, sz, vp]
        L.wide_ffn_masked_noalloc.restype = ci
        L.wide_ffn_masked_noalloc.argtypes = [ci, i64, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.wide_static_scratch_bytes.restype = sz
        L.wide_static_scratch_bytes.argtypes = []
        L.wide_qkvo_masked.restype = ci
        L.wide_qkvo_masked.argtypes = [ci, ci, i64, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp,
                                       vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.wide_router.restype = ci
        L.wide_router.argtypes = [ci, i64, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.wide_attention_masked.restype = ci
        L.wide_attention_masked.argtypes = [ci, i64, i32, i32, i32, i32, i32, i32, i32, vp, vp, vp, vp,
                                            vp, vp, vp, vp, vp, sz, vp]
        L.wide_attention_workspace_size.restype = sz
        L.wide_attention_workspace_size.argtypes = [i64, i32, i32, i32, i32, i32, i32, i32]
        L.wide_attention_decode.restype = ci
        L.wide_attention_decode.argtypes = [ci, i64, i32, i32, i32, i32, i32, vp, vp, ci, vp, vp, vp, vp, vp,
                                            sz, vp]
        L.wide_attention_decode_workspace_size.restype = sz
        L.wide_attention_decode_workspace_size.argtypes = [i64, i32, i32, i32, i32, i32]
        L.wide_workspace_size.restype = sz
        L.wide_workspace_size.argtypes = [ci, ci, i64, i32, i32, i32]
        L.wide_set_option.restype = ci
        L.wide_set_option.argtypes = [ctypes.c_char_p, i64]
        L.wide_get_option.restype = ci
        L.wide_get_option.argtypes = [ctypes.c_char_p, ctypes.POINTER(i64)]
        L.wide_timing_enable.restype = ci
        L.wide_timing_enable.argtypes = [ci]
        L.wide_timing_reset.restype = ci
        L.wide_timing_reset.argtypes = []
        L.wide_timing_filter.restype = ci
        L.wide_timing_filter.argtypes = [ctypes.c_char_p]
        L.wide_timing_query.restype = ci
        L.wide_timing_query.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(i64)]
        _lib = L
    return _lib


def _check(fn: str, status: int) -> None:
    if status != OK:
        raise WideError(fn, status, lib().wide_last_error().decode(errors="replace"))


def _torch():
    import torch
    return torch


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(t):
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype} (bf16 or fp32)")


def _mask_bytes(mask):
    torch = _torch()
    if mask.dtype == torch.bool:
        mask = mask.view(torch.uint8)
    if mask.dtype != torch.uint8:
        raise TypeError("mask must be uint8 or bool")
    if mask.numel() and mask.data_ptr() % 16:
        # the library reads mask rows with 16-byte loads and requires a
        # 16-byte aligned mask (a row slice of a mask may not be): copy it
        mask = mask.clone()
    return mask


def _workspace(nbytes: int, device):
    torch = _torch()
    if nbytes == SIZE_MAX:
        raise ValueError("arguments rejected by wide_workspace_size")
    if nbytes == 0:
        return None
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def _contig(*ts):
    for t in ts:
        if t is not None and not t.is_contiguous():
            raise ValueError("tensors must be contiguous")


# ---- entry points -------------------------------------------------------------

def wide_workspace_size(op: int, dtype: int, M: int, d_model: int, d_inner: int,
                        group_size: int) -> int:
    return int(lib().wide_workspace_size(op, dtype, M, d_model, d_inner, group_size))


def wide_set_option(key: str, value: int) -> None:
    _check("wide_set_option", lib().wide_set_option(key.encode(), int(value)))


def wide_get_option(key: str) -> int:
    v = ctypes.c_int64()
    _check("wide_get_option", lib().wide_get_option(key.encode(), ctypes.byref(v)))
    return int(v.value)


def wide_timing_enable(on: bool = True) -> None:
    _check("wide_timing_enable", lib().wide_timing_enable(int(on)))


def wide_timing_reset() -> None:
    _check("wide_timing_reset", lib().wide_timing_reset())


def wide_timing_filter(name=None) -> None:
    """Time only launches labelled `name` (query's matching rule); None: all."""
    _check("wide_timing_filter", lib().wide_timing_filter(name.encode() if name else None))


def wide_timing_query(name: str):
    """(total milliseconds, launches) of recorded kernels labelled `name`
    (exactly, or followed by a template argument list or a "/variant" suffix)."""
    ms, n = ctypes.c_double(), ctypes.c_int64()
    _check("wide_timing_query", lib().wide_timing_query(name.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return float(ms.value), int(n.value)


def wide_mask_reorder(mask, idx=None, counts=None, ws=None):
    """mask [M][n_groups] (uint8/bool, device) -> (idx int32 [n_groups][M], counts int32 [n_groups])."""
    torch = _torch()
    mask = _mask_bytes(mask)
    _contig(mask)
    M, ng = mask.shape
    if idx is None:
        idx = torch.empty((ng, M), dtype=torch.int32, device=mask.device)
    if counts is None:
        counts = torch.empty((ng,), dtype=torch.int32, device=mask.device)
    if ws is None:
        ws = _workspace(wide_workspace_size(OP_REORDER, BF16, M, 0, ng, 1), mask.device)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("wide_mask_reorder", lib().wide_mask_reorder(
        _p(mask), M, ng, _p(idx), _p(counts), _p(ws), nbytes, _stream(mask)))
    return idx, counts


def wide_ffn_masked(x, w_gate, w_up, w_down, mask, group_size, idx=None, counts=None,
                    h_out=None, y=None, ws=None):
    """Masked SwiGLU FFN; returns y [M][d_model] (same dtype as x)."""
    torch = _torch()
    mask = _mask_bytes(mask)
    _contig(x, w_gate, w_up, w_down, mask, idx, counts, h_out, y)
    dt = _dtype_code(x)
    M, D = x.shape
    Dff = w_gate.shape[0]
    if y is None:
        y = torch.empty((M, D), dtype=x.dtype, device=x.device)
    if ws is None:
        ws = _workspace(wide_workspace_size(OP_FFN, dt, M, D, Dff, group_size), x.device)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("wide_ffn_masked", lib().wide_ffn_masked(
        dt, M, D, Dff, group_size, _p(mask), _p(idx), _p(counts), _p(x), _p(w_gate), _p(w_up),
        _p(w_down), _p(h_out), _p(y), _p(ws), nbytes, _stream(x)))
    return y


def wide_ffn_masked_noalloc(x, w_gate, w_up, w_down, mask, group_size, idx=None, counts=None,
                            h_out=None, y=None):
    """wide_ffn_masked with the library's static per-GPU scratch instead of a
    workspace (for callers that cannot allocate: pass y, and h_out for long
    prefills, and the call allocates nothing)."""
    torch = _torch()
    mask = _mask_bytes(mask)
    _contig(x, w_gate, w_up, w_down, mask, idx, counts, h_out, y)
    M, D = x.shape
    if y is None:
        y = torch.empty((M, D), dtype=x.dtype, device=x.device)
    _check("wide_ffn_masked_noalloc", lib().wide_ffn_masked_noalloc(
        _dtype_code(x), M, D, w_gate.shape[0], group_size, _p(mask), _p(idx), _p(counts), _p(x), _p(w_gate),
        _p(w_up), _p(w_down), _p(h_out), _p(y), _stream(x)))
    return y


def wide_static_scratch_bytes() -> int:
    return int(lib().wide_static_scratch_bytes())


def wide_qkvo_masked(phase, inp, mask, group_size, n_q_heads, n_kv_heads, head_dim,
                     w_q=None, w_k=None, w_v=None, w_o=None, idx=None, counts=None,
                     q=None, k=None, v=None, y=None, d_model=None, ws=None):
    """PHASE_QKV: returns (q, k, v); PHASE_O: returns y."""
    torch = _torch()
    mask = _mask_bytes(mask)
    _contig(inp, mask, w_q, w_k, w_v, w_o, idx, counts, q, k, v, y)
    dt = _dtype_code(inp)
    M = inp.shape[0]
    Nq, Nkv = n_q_heads * head_dim, n_kv_heads * head_dim
    if phase == PHASE_QKV:
        D = inp.shape[1]
        if q is None:
            q = torch.empty((M, Nq), dtype=inp.dtype, device=inp.device)
        if k is None:
            k = torch.empty((M, Nkv), dtype=inp.dtype, device=inp.device)
        if v is None:
            v = torch.empty((M, Nkv), dtype=inp.dtype, device=inp.device)
        op = OP_QKV
    else:
        D = w_o.shape[0] if d_model is None else d_model
        if y is None:
            y = torch.empty((M, D), dtype=inp.dtype, device=inp.device)
        op = OP_O
    if ws is None:
        ws = _workspace(wide_workspace_size(op, dt, M, D, Nq, group_size), inp.device)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("wide_qkvo_masked", lib().wide_qkvo_masked(
        phase, dt, M, D, n_q_heads, n_kv_heads, head_dim, group_size, _p(mask), _p(idx),
        _p(counts), _p(inp), _p(w_q), _p(w_k), _p(w_v), _p(w_o), _p(q), _p(k), _p(v), _p(y),
        _p(ws), nbytes, _stream(inp)))
    return (q, k, v) if phase == PHASE_QKV else y


def wide_router(x, w1, w2, mask=None, logits=False, reorder=False, idx=None, counts=None, ws=None):
    """Bottleneck router (inference).  x [M][d_model] bf16, w1 [rank][d_model],
    w2 [2*n_groups][rank].  Returns the mask [M][n_groups] uint8, followed by
    the fp32 logits [M][2*n_groups] if `logits`, and (idx, counts) if
    `reorder`."""
    torch = _torch()
    _contig(x, w1, w2, mask, idx, counts)
    M, D = x.shape
    rank = w1.shape[0]
    ng = w2.shape[0] // 2
    if mask is None:
        mask = torch.empty((M, ng), dtype=torch.uint8, device=x.device)
    lg = torch.empty((M, 2 * ng), dtype=torch.float32, device=x.device) if logits else None
    if reorder:
        if idx is None:
            idx = torch.empty((ng, M), dtype=torch.int32, device=x.device)
        if counts is None:
            counts = torch.empty((ng,), dtype=torch.int32, device=x.device)
    else:
        idx = counts = None
    if ws is None and reorder:
        ws = _workspace(wide_workspace_size(OP_ROUTER, _dtype_code(x), M, D, ng, rank), x.device)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("wide_router", lib().wide_router(
        _dtype_code(x), M, D, rank, ng, _p(x), _p(w1), _p(w2), _p(mask), _p(lg), _p(idx),
        _p(counts), _p(ws), nbytes, _stream(x)))
    out = [mask]
    if logits:
        out.append(lg)
    if reorder:
        out += [idx, counts]
    return out[0] if len(out) == 1 else tuple(out)


def wide_attention_workspace_size(n_seq, T_q, T_k, n_q, n_kv, head_dim, group_size, with_reorder=True):
    return int(lib().wide_attention_workspace_size(n_seq, T_q, T_k, n_q, n_kv, head_dim, group_size,
                                                   int(bool(with_reorder))))


def wide_attention_masked(q, k, v, mask, n_seq, n_q, n_kv, head_dim, group_size, causal=True,
                          idx=None, counts=None, o=None, ws=None, leftpad=None):
    """Head-group masked attention (prefill).  q [n_seq*T_q][n_q*head_dim],
    k, v [n_seq*T_k][n_kv*head_dim], mask [n_seq*T_q][n_groups] uint8;
    idx/counts optional (a reorder of `mask`); leftpad optional int32
    [n_seq] (the first non-padding key of each sequence).  Returns o, same
    shape as q."""
    torch = _torch()
    _contig(q, k, v, mask, idx, counts, o, leftpad)
    mask = _mask_bytes(mask)
    if n_seq > 0 and (q.shape[0] % n_seq or k.shape[0] % n_seq):
        raise ValueError("q and k rows must split evenly into n_seq sequences")
    T_q = q.shape[0] // n_seq if n_seq > 0 else 0
    T_k = k.shape[0] // n_seq if n_seq > 0 else 0
    if o is None:
        o = torch.empty_like(q)
    if ws is None:
        need = wide_attention_workspace_size(n_seq, T_q, T_k, n_q, n_kv, head_dim, group_size, idx is None)
        # (shapes the library rejects: no workspace, the call reports why)
        ws = None if need == SIZE_MAX else _workspace(need, q.device)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("wide_attention_masked", lib().wide_attention_masked(
        _dtype_code(q), n_seq, T_q, T_k, n_q, n_kv, head_dim, group_size, int(bool(causal)), _p(leftpad),
        _p(mask), _p(idx), _p(counts), _p(q), _p(k), _p(v), _p(o), _p(ws), nbytes, _stream(q)))
    return o


def wide_attention_decode_workspace_size(batch, L, n_q, n_kv, head_dim, group_size):
    return int(lib().wide_attention_decode_workspace_size(batch, L, n_q, n_kv, head_dim, group_size))


KV_TOKEN_MAJOR, KV_HEAD_MAJOR = 0, 1


def wide_attention_decode(q, k_cache, v_cache, mask, n_q, n_kv, head_dim, group_size, kv_len=None,
                          o=None, ws=None, head_major=False):
    """Head-group masked attention at decode.  q [B][n_q*head_dim]; k_cache and
    v_cache [B][L][n_kv*head_dim] (or [B][n_kv][L][head_dim] with head_major);
    mask [B][n_groups] uint8; kv_len optional int32 [B].  Returns o, same
    shape as q."""
    _contig(q, k_cache, v_cache, mask, kv_len, o)
    mask = _mask_bytes(mask)
    B = q.shape[0]
    if head_major:
        L = k_cache.shape[2] if k_cache.dim() == 4 else 0
    else:
        L = k_cache.shape[1] if k_cache.dim() == 3 else 0
    if o is None:
        o = _torch().empty_like(q)
    if ws is None:
        need = wide_attention_decode_workspace_size(B, L, n_q, n_kv, head_dim, group_size)
        ws = None if need == SIZE_MAX else _workspace(need, q.device)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("wide_attention_decode", lib().wide_attention_decode(
        _dtype_code(q), B, L, n_q, n_kv, head_dim, group_size, _p(mask), _p(kv_len),
        KV_HEAD_MAJOR if head_major else KV_TOKEN_MAJOR, _p(q), _p(k_cache),
        _p(v_cache), _p(o), _p(ws), nbytes, _stream(q)))
    return o
