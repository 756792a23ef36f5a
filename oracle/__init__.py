"""fp64 CPU oracle for WIDE's masked projections (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding) never does, and this package never imports the product.

The arithmetic lives in ``wide_oracle.c`` (plain fp64 loops, OpenMP over
tokens).  This module builds it with gcc and marshals numpy arrays through
ctypes.  Floating-point inputs are either float32 arrays or bf16 bit patterns
held in uint16 arrays; outputs are float64 arrays.

Sources followed (WIDE, "Token-level Dynamic Width Pruning"):
  * ``mask_reorder``   Section 3.3 (per-column SortDesc) and Appendix B,
                       Algorithm 1.
  * ``nproj``          Section 3.1, equations (1)-(2), Figure 1: Q pruned over
                       out-features in head groups.
  * ``kproj``          Section 3.1 equations (2)-(3) and the GEMM-K sum of
                       Appendix B: W_o / W_down pruned over in-features.
  * ``ffn``            Section 3.1, equation (3), with phi = SiLU (SwiGLU).
  * ``linear``         dense K/V projections, equation (1).
  * ``attention``      Section 3.1 equations (1)-(2) and Appendix B,
                       Algorithm 4: per (token, head group) either standard
                       scaled dot-product attention or zeros.
  * ``router``         Section 3.1, Routing Components: logits X W1 W2 as
                       n_groups (execute, skip) pairs; the mask bit is 1 when
                       class 0 wins (argmax, first index on a tie).
  * ``bf16_round``     storage rounding of the bf16 data path (the paper states
                       no precision; the reading is recorded with the design
                       notes).

Every function is pinned by CPU tests against closed forms, special cases
that reduce to numpy/torch routines, invariants and independent formulations.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "wide_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2 -fopenmp, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
             "-fno-fast-math", "-ffp-contract=off", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        vp, i64, i32, ci = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int
        lib.oracle_bf16_round.restype = ctypes.c_double
        lib.oracle_bf16_round.argtypes = [ctypes.c_double]
        lib.oracle_mask_reorder.argtypes = [vp, i64, i32, vp, vp]
        lib.oracle_linear.argtypes = [ci, ci, i64, i32, i32, vp, vp, vp]
        lib.oracle_nproj.argtypes = [ci, ci, i64, i32, i32, i32, vp, vp, vp, vp]
        lib.oracle_kproj.argtypes = [ci, ci, i64, i32, i32, i32, vp, vp, vp, vp]
        lib.oracle_ffn.argtypes = [ci, ci, i64, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp]
        lib.oracle_router.argtypes = [ci, i64, i32, i32, i32, vp, vp, vp, vp, vp]
        lib.oracle_attention.argtypes = [ci, ci, i64, i32, i32, i32, i32, i32, i32, ci, vp, vp, vp, vp, vp, vp]
        lib.oracle_num_threads.restype = ci
        _lib = lib
    return _lib


def _fp(a: np.ndarray):
    """Return (dtype code, contiguous array) for a float32 or bf16-bits array."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return 1, a
    if a.dtype == np.float32:
        return 0, a
    raise TypeError(f"oracle takes float32 or bf16 bits (uint16), got {a.dtype}")


def _same_dtype(*arrs):
    codes = [_fp(a) for a in arrs]
    if len({c for c, _ in codes}) != 1:
        raise TypeError("all floating-point operands must share one dtype")
    return codes[0][0], [a for _, a in codes]


def _mask(m: np.ndarray) -> np.ndarray:
    m = np.ascontiguousarray(m)
    if m.dtype == np.bool_:
        m = m.view(np.uint8)
    if m.dtype != np.uint8:
        raise TypeError("mask must be uint8 or bool")
    return m


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def bf16_round(v: float) -> float:
    """Nearest bf16 value to v, ties to even, rounded once from fp64."""
    return float(_load().oracle_bf16_round(float(v)))


def mask_reorder(mask: np.ndarray):
    """mask [M][n_groups] -> (idx int32 [n_groups][M], cnt int32 [n_groups])."""
    mask = _mask(mask)
    M, ng = mask.shape
    idx = np.empty((ng, M), np.int32)
    cnt = np.empty((ng,), np.int32)
    _load().oracle_mask_reorder(_p(mask), M, ng, _p(idx), _p(cnt))
    return idx, cnt


def linear(x, w, round_bf16=False) -> np.ndarray:
    dt, (x, w) = _same_dtype(x, w)
    M, K = x.shape
    N = w.shape[0]
    assert w.shape == (N, K)
    out = np.empty((M, N), np.float64)
    _load().oracle_linear(dt, int(round_bf16), M, K, N, _p(x), _p(w), _p(out))
    return out


def nproj(x, w, mask, G, round_bf16=False) -> np.ndarray:
    dt, (x, w) = _same_dtype(x, w)
    mask = _mask(mask)
    M, K = x.shape
    N = w.shape[0]
    assert w.shape == (N, K) and N % G == 0 and mask.shape == (M, N // G)
    out = np.empty((M, N), np.float64)
    _load().oracle_nproj(dt, int(round_bf16), M, K, N, G, _p(mask), _p(x), _p(w), _p(out))
    return out


def kproj(a, w, mask, G, round_bf16=False) -> np.ndarray:
    dt, (a, w) = _same_dtype(a, w)
    mask = _mask(mask)
    M, K = a.shape
    N = w.shape[0]
    assert w.shape == (N, K) and K % G == 0 and mask.shape == (M, K // G)
    out = np.empty((M, N), np.float64)
    _load().oracle_kproj(dt, int(round_bf16), M, K, N, G, _p(mask), _p(a), _p(w), _p(out))
    return out


def ffn(x, w_gate, w_up, w_down, mask, G, round_bf16=False, want_h=True):
    """Masked SwiGLU FFN.  Returns (h [M][Dff] or None, y [M][D]) as float64."""
    dt, (x, w_gate, w_up, w_down) = _same_dtype(x, w_gate, w_up, w_down)
    mask = _mask(mask)
    M, D = x.shape
    Dff = w_gate.shape[0]
    assert w_gate.shape == (Dff, D) and w_up.shape == (Dff, D)
    assert w_down.shape == (D, Dff) and Dff % G == 0 and mask.shape == (M, Dff // G)
    h = np.empty((M, Dff), np.float64) if want_h else None
    y = np.empty((M, D), np.float64)
    _load().oracle_ffn(dt, int(round_bf16), M, D, Dff, G, _p(mask), _p(x), _p(w_gate),
                       _p(w_up), _p(w_down), _p(h) if h is not None else None, _p(y))
    return h, y


def router(x, w1, w2):
    """Bottleneck router, inference form.  x [M][D], w1 [r][D] (W1 transposed),
    w2 [2*n_groups][r] (W2 transposed; rows 2g and 2g+1 are group g's execute
    and skip classes).  Returns (logits float64 [M][2*n_groups], mask uint8
    [M][n_groups])."""
    dt, (x, w1, w2) = _same_dtype(x, w1, w2)
    M, D = x.shape
    r = w1.shape[0]
    J = w2.shape[0]
    assert w1.shape == (r, D) and w2.shape == (J, r) and J % 2 == 0
    logits = np.empty((M, J), np.float64)
    mask = np.empty((M, J // 2), np.uint8)
    _load().oracle_router(dt, M, D, r, J // 2, _p(x), _p(w1), _p(w2), _p(logits), _p(mask))
    return logits, mask


def attention(q, k, v, mask, n_seq, n_q, n_kv, d, causal, round_bf16=False, leftpad=None):
    """Head-group masked attention (prefill).  q [n_seq*T_q][n_q*d],
    k/v [n_seq*T_k][n_kv*d], mask [n_seq*T_q][n_groups]; with causal masking
    the queries are the last T_q of each sequence's T_k positions; leftpad
    (optional int [n_seq]) hides keys j < leftpad[b] of sequence b (a query
    left with no key gets zeros).  Returns o float64 [n_seq*T_q][n_q*d]."""
    dt, (q, k, v) = _same_dtype(q, k, v)
    mask = _mask(mask)
    Mq, Mk = q.shape[0], k.shape[0]
    assert Mq % n_seq == 0 and Mk % n_seq == 0
    assert q.shape[1] == n_q * d and k.shape == (Mk, n_kv * d) and v.shape == k.shape
    T_q, T_k = Mq // n_seq, Mk // n_seq
    assert not causal or T_k >= T_q
    ng = mask.shape[1]
    assert mask.shape[0] == Mq and n_q % ng == 0 and n_q % n_kv == 0
    lp = None
    if leftpad is not None:
        lp = np.ascontiguousarray(leftpad, dtype=np.int32)
        assert lp.shape == (n_seq,) and (lp >= 0).all() and (lp <= T_k).all()
    o = np.empty((Mq, n_q * d), np.float64)
    _load().oracle_attention(dt, int(round_bf16), n_seq, T_q, T_k, n_q, n_kv, d, ng, int(causal),
                             _p(mask), _p(q), _p(k), _p(v), _p(lp) if lp is not None else None, _p(o))
    return o
