"""Shared test helpers: device transfer and the parity tolerance."""
import numpy as np
import torch

from paper_2607_28418_amd import synth

# Parity bar for the bf16 path against the storage-matched fp64 oracle
# (bf16 rounding of H and of every output, as the kernels store them):
#   mean |got - ref| <= 1e-3  and  max |got - ref| / max(|ref|, 0.1 rms(ref)) <= 2e-2.
# A kernel that is exact except for fp32 accumulation order scores about
# 1e-5 / 8e-3 (one bf16 ulp where a rounding flips); dropping a single
# (token, group) contribution scores about 4 on the second measure.
BF16_MAE, BF16_REL = 1e-3, 2e-2
# fp32 path against the unrounded fp64 oracle.
F32_MAE, F32_REL = 1e-6, 1e-4


def dev():
    return torch.device("cuda", 0)


def to_dev(a: np.ndarray, device=None):
    device = device or dev()
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def to_np64(t) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def parity_stats(got: np.ndarray, ref: np.ndarray, abs_allow=0.0):
    """(mean abs error, max relative error); the relative error of an element
    is (|got-ref| - abs_allow)+ / max(|ref|, 0.1 rms(ref)).  abs_allow is a
    scalar or an array of ref's shape (a per-element allowance)."""
    mae_err = np.abs(got - ref)
    err = np.maximum(mae_err - abs_allow, 0.0)
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0
    floor = np.maximum(np.abs(ref), 0.1 * rms)
    with np.errstate(divide="ignore", invalid="ignore"):
        rel = np.where(floor > 0, err / floor, np.where(err > 0, np.inf, 0.0))
    return float(mae_err.mean()) if err.size else 0.0, float(rel.max()) if rel.size else 0.0


def assert_close(got, ref: np.ndarray, kind: str = "bf16", what: str = "", abs_allow=0.0):
    g = to_np64(got) if isinstance(got, torch.Tensor) else got
    assert g.shape == ref.shape, (what, g.shape, ref.shape)
    assert np.isfinite(g).all(), f"{what}: non-finite output"
    mae, rel = parity_stats(g, ref, abs_allow)
    mae_tol, rel_tol = (BF16_MAE, BF16_REL) if kind == "bf16" else (F32_MAE, F32_REL)
    assert mae <= mae_tol and rel <= rel_tol, f"{what}: mae={mae:.3g} (<= {mae_tol}) maxrel={rel:.3g} (<= {rel_tol})"
    return mae, rel


# ---- masked attention -------------------------------------------------------------

def bf16_ulp_arr(x):
    a = np.abs(x)
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a > 0, 2.0 ** (e - 7), 0.0)


def attention_bound(orc, q, k, v, mask, n_seq, n_q, n_kv, hd, causal, T_k, leftpad=None):
    """Per-element error bound of the bf16 attention path (probabilities
    rounded to bf16 for P.V: unit roundoff 2^-8 times attention applied to
    |V|; fp32 scores, exponentials and sums: (2^-12 + T_k 2^-24) of the
    same); the stored output's own bf16 rounding is added by the check."""
    vabs = np.abs(synth.as_f32(v)).astype(np.float32)
    a_abs = orc.attention(synth.as_f32(q), synth.as_f32(k), vabs, mask, n_seq, n_q, n_kv, hd, causal,
                          leftpad=leftpad)
    return (2.0 ** -8 + 2.0 ** -12 + T_k * 2.0 ** -24) * a_abs


def check_attention_rows(got, ref, bound, mask_rows, hpg_feat, what):
    """got/ref/bound [rows][n_q*hd] float64; inactive (row, group) blocks must be +0."""
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    inactive = ~np.repeat(mask_rows.astype(bool), hpg_feat, axis=1)
    assert not got[inactive].any() and not np.signbit(got[inactive]).any(), f"{what}: inactive rows not +0"
    err = np.abs(got - ref)
    allow = bound + bf16_ulp_arr(got)
    worst = float(np.max(err - allow)) if err.size else 0.0
    assert worst <= 0.0, f"{what}: {int((err > allow).sum())} elements over the bound (worst excess {worst:.3g})"
    mae = float(err.mean()) if err.size else 0.0
    assert mae <= 1e-3, f"{what}: mae {mae:.3g}"
    return mae


# ---- bf16 projections: rounding bands (tests/_bounds) plus the parity bar -----------

def _rows_np(t, rows):
    if isinstance(t, np.ndarray):
        return np.asarray(t if rows is None else t[rows], np.float64)
    if rows is None:
        return to_np64(t)
    return to_np64(t[torch.as_tensor(rows, device=t.device)])


def _sel(a, rows):
    return a if rows is None else a[rows]


def check_ffn(orc, c, y, h=None, rows=None, what="ffn"):
    """bf16 masked FFN against the oracle on token rows `rows` (all if None).

    H and y must lie in their rounding bands (bit-exact outside a narrow band
    around bf16 rounding boundaries, one bf16 step inside it; skipped H
    blocks and all-inactive rows exactly +0), and y must meet the parity bar
    (mean |err| <= 1e-3, max relative error <= 2e-2 with the 0.1 rms floor)
    after the per-element allowance for H values the kernel may round to the
    neighbouring bf16 value."""
    from tests import _bounds as B
    x, mask = _sel(c.x, rows), _sel(c.mask, rows)
    rh, ry = orc.ffn(x, c.w_gate, c.w_up, c.w_down, mask, c.G, round_bf16=True)
    h64, _ = orc.ffn(x, c.w_gate, c.w_up, c.w_down, mask, c.G)
    y64 = orc.kproj(synth.f32_to_bf16_bits(rh.astype(np.float32)), c.w_down, mask, c.G)
    A_h, A_flip, A_y = B.ffn_bands(x, c.w_gate, c.w_up, c.w_down, mask, c.G, h64, rh)
    if h is not None:
        B.check_band(_rows_np(h, rows), h64, A_h, f"{what} h", zero=~B.expand(mask, c.G))
    yg = _rows_np(y, rows)
    B.check_band(yg, y64, A_y, f"{what} y", zero=np.broadcast_to(~mask.any(1)[:, None], yg.shape))
    return assert_close(yg, ry, what=f"{what} y", abs_allow=A_flip)


def check_nproj(orc, x, w, mask, G, got, rows=None, what="q"):
    """bf16 N-axis projection (mask None: dense) against the oracle: rounding
    band, +0 at inactive blocks, and the parity bar."""
    from tests import _bounds as B
    x = _sel(x, rows)
    if mask is None:
        v, ref, zero = orc.linear(x, w), orc.linear(x, w, round_bf16=True), None
    else:
        mask = _sel(mask, rows)
        v, ref = orc.nproj(x, w, mask, G), orc.nproj(x, w, mask, G, round_bf16=True)
        zero = ~B.expand(mask, G)
    g = _rows_np(got, rows)
    B.check_band(g, v, B.nproj_band(x, w, mask, G), what, zero=zero)
    return assert_close(g, ref, what=what)


def check_kproj(orc, a, w, mask, G, got, rows=None, what="o"):
    """bf16 K-axis projection against the oracle: rounding band, +0 rows for
    tokens with no active group, and the parity bar."""
    from tests import _bounds as B
    a, mask = _sel(a, rows), _sel(mask, rows)
    v, ref = orc.kproj(a, w, mask, G), orc.kproj(a, w, mask, G, round_bf16=True)
    g = _rows_np(got, rows)
    B.check_band(g, v, B.kproj_band(a, w, mask, G), what,
                 zero=np.broadcast_to(~mask.any(1)[:, None], g.shape))
    return assert_close(g, ref, what=what)
