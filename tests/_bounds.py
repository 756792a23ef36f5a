"""Per-element error bounds of the bf16 projections, derived from the arithmetic.

The kernels form every stored value (Q, K, V, H, y) as an fp32 sum of exact
bf16 x bf16 products and round that sum once to bf16, nearest even; the oracle
computes the same sum exactly (fp64) and rounds it once.  The two stored
values can differ only where the exact sum lies closer to a bf16 rounding
boundary than the fp32 sum's error.  So a stored value is checked against the
interval [RNE(v - A), RNE(v + A)], where v is the oracle's unrounded value and
A bounds the kernel's error before rounding: outside that narrow band the
kernel must be bit-exact, inside it one bf16 step either way is allowed.

The fp32 error bound A of a dot product (how it is derived):
  * products of two bf16 values are exact in fp32, so all error comes from
    the additions: each rounds its result S_i by a relative amount of at
    most u = 2^-24, and the total error is sum_i delta_i S_i;
  * every partial sum the kernels form adds aligned blocks of 16 consecutive
    k (the k width of one MFMA), in one of these orders: sequentially in
    increasing k, possibly cut into contiguous chunks (prefill tiles and
    their k-split tails); by eight waves each taking every eighth 64-wide
    step (decode), then combined; or per group, the group sums then added
    in any order (the atomic K-axis schedule).  R, the largest magnitude any
    of these partial sums can take, is computed from the data: twice the
    largest prefix sum (a chunk is a difference of two prefixes), twice the
    largest prefix of each of the eight step classes, the sum of the
    classes' magnitudes, and, on the K axis, the sum of the group sums'
    magnitudes;
  * inside one MFMA the 16 products may themselves be summed in fp32 before
    the block joins the accumulator; those partial sums are at most the
    block's sum of |products|;
  * treating the delta_i as independent and zero-mean, Hoeffding's
    inequality bounds sum_i delta_i S_i by LAMBDA u sqrt(n) max|S_i| except
    with probability 2 exp(-LAMBDA^2 / 2) (about 2.5e-14 for LAMBDA = 8).
FFN intermediate h = silu(a) b adds the error of silu (hardware exp and
reciprocal: a relative (|a| + 8) u at most) and propagates the errors of a
and b; the down projection's output y adds, for every h the kernel may have
rounded to the neighbouring bf16 value, that step times |w_down|.
"""
from __future__ import annotations

import math

import numpy as np
import torch

from paper_2607_28418_amd import synth

U32 = 2.0 ** -24
LAMBDA = 8.0
BLOCK = 16        # k width of one MFMA step
STEP = 64         # k width of one decode wave step
WAVES = 8         # decode waves interleaving the steps


def rne_bf16(v: np.ndarray) -> np.ndarray:
    """Nearest bf16 value to every float64 in v (ties to even), one rounding."""
    v = np.asarray(v, np.float64)
    m, e = np.frexp(v)                 # v = m 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.round(m * 256.0) / 256.0, e)   # 8 significant bits; numpy rounds half to even


def f64(a: np.ndarray) -> np.ndarray:
    return synth.as_f32(a).astype(np.float64)


def _partial_sum_bound(bs: torch.Tensor, ba: torch.Tensor, group_blocks: int = 0) -> torch.Tensor:
    """bs, ba [nb][...]: block sums and block sums of |products|, in k order.
    Returns the bound on the fp32 error of the full sum, per element of [...]."""
    nb = bs.shape[0]
    P = bs.cumsum(0)
    R = 2.0 * P.abs().amax(0)
    steps_blk = STEP // BLOCK
    pad = (-nb) % (steps_blk * WAVES)
    if pad:
        bs_p = torch.cat([bs, bs.new_zeros((pad,) + bs.shape[1:])])
    else:
        bs_p = bs
    q = bs_p.shape[0] // (steps_blk * WAVES)
    cls = bs_p.reshape((q, WAVES, steps_blk) + bs.shape[1:]).transpose(0, 1)
    cls = cls.reshape((WAVES, q * steps_blk) + bs.shape[1:])
    Pc = cls.cumsum(1)
    R = torch.maximum(R, 2.0 * Pc.abs().amax(1).amax(0))
    R = torch.maximum(R, Pc[:, -1].abs().sum(0))
    if group_blocks:
        gs = bs.reshape((nb // group_blocks, group_blocks) + bs.shape[1:]).sum(1)
        R = torch.maximum(R, gs.abs().sum(0))
    Bm = ba.amax(0)
    K = nb * BLOCK
    n_nodes = nb + 64          # one rounding per MFMA step, plus combinations
    return LAMBDA * U32 * (math.sqrt(n_nodes) * R + math.sqrt(K) * Bm)


def dot_error_bound(x: np.ndarray, w: np.ndarray, group: int = 0, rows_per_chunk: int = 0) -> np.ndarray:
    """Bound on |fp32 sum - exact sum| of out[t, n] = sum_k x[t, k] w[n, k].

    x [M][K] and w [N][K] are float64 (zeros where a masked input block is
    left out).  group > 0 (a multiple of 16) adds the K-axis scatter order."""
    M, K = x.shape
    N = w.shape[0]
    assert w.shape[1] == K and K % BLOCK == 0
    nb = K // BLOCK
    Wt = torch.from_numpy(np.ascontiguousarray(w))
    Wb = Wt.reshape(N, nb, BLOCK).permute(1, 2, 0).contiguous()        # [nb][16][N]
    Wa = Wb.abs()
    if not rows_per_chunk:
        rows_per_chunk = max(1, int(2e7 // (nb * N)))
    out = np.empty((M, N), np.float64)
    for r0 in range(0, M, rows_per_chunk):
        X = torch.from_numpy(np.ascontiguousarray(x[r0:r0 + rows_per_chunk]))
        m = X.shape[0]
        Xb = X.reshape(m, nb, BLOCK).permute(1, 0, 2).contiguous()      # [nb][m][16]
        bs = torch.bmm(Xb, Wb)                                           # [nb][m][N]
        ba = torch.bmm(Xb.abs(), Wa)
        out[r0:r0 + m] = _partial_sum_bound(bs, ba, group // BLOCK if group else 0).numpy()
    return out


def in_rounding_band(got: np.ndarray, v: np.ndarray, A: np.ndarray):
    """Elements of got outside [RNE(v - A), RNE(v + A)] (boolean array)."""
    lo, hi = rne_bf16(v - A), rne_bf16(v + A)
    return (got < lo) | (got > hi)


def check_band(got: np.ndarray, v: np.ndarray, A: np.ndarray, what: str, zero=None):
    """Every element of got (bf16 values as float64) lies in its rounding band;
    elements flagged by `zero` must be exactly +0."""
    assert got.shape == v.shape, (what, got.shape, v.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    if zero is not None:
        z = got[zero]
        assert not z.any() and not np.signbit(z).any(), f"{what}: skipped outputs not +0"
    bad = in_rounding_band(got, v, A)
    if zero is not None:
        bad &= ~zero
    n = int(bad.sum())
    if n:
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {n} of {bad.size} elements outside the rounding band, first at "
                             f"{tuple(i)}: got {got[tuple(i)]!r}, exact {v[tuple(i)]!r}, bound {A[tuple(i)]:.3g}")


# ---- the projections ------------------------------------------------------------

def expand(mask: np.ndarray, G: int) -> np.ndarray:
    return np.repeat(mask.astype(bool), G, axis=1)


def nproj_band(x, w, mask, G):
    """Bound for an N-axis output (Q; K/V with mask None): exact value is the
    oracle's; A per element (active outputs only)."""
    return dot_error_bound(f64(x), f64(w))


def kproj_band(a, w, mask, G):
    """Bound for a K-axis output (O): the inactive input blocks are exact zeros."""
    am = f64(a) * expand(mask, G)
    return dot_error_bound(am, f64(w), group=G)


def silu64(a):
    return a / (1.0 + np.exp(-a))


def ffn_bands(x, w_gate, w_up, w_down, mask, G, h_exact, h_ref):
    """(A_h, A_y_flip, A_y) for the FFN on the bf16 path.

    h_exact: the oracle's unrounded H; h_ref: its bf16 H (both [M][Dff] fp64).
    A_h bounds the kernel's fp32 h before rounding; A_y_flip is the part of
    y's bound due to h values the kernel may round the other way; A_y adds
    the down projection's own fp32 error."""
    X = f64(x)
    Wg, Wu, Wd = f64(w_gate), f64(w_up), f64(w_down)
    act = expand(mask, G)
    a = X @ Wg.T
    b = X @ Wu.T
    ea = dot_error_bound(X, Wg)
    eb = dot_error_bound(X, Wu)
    s = 1.0 / (1.0 + np.exp(-a))
    dsilu = np.abs(s * (1.0 + a * (1.0 - s)))
    A_h = dsilu * np.abs(b) * ea + np.abs(a * s) * eb + 1.1 * ea * eb + (np.abs(a) + 8.0) * U32 * np.abs(h_exact)
    A_h = np.where(act, A_h, 0.0)
    step = np.where(act, rne_bf16(h_exact + A_h) - rne_bf16(h_exact - A_h), 0.0)
    A_flip = step @ np.abs(Wd).T
    hm = np.where(act, h_ref, 0.0)
    A_y = A_flip + dot_error_bound(hm, Wd, group=G)
    return A_h, A_flip, A_y
