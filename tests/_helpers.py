"""Shared test helpers: device transfer and the parity tolerance."""
import numpy as np
import torch

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


def parity_stats(got: np.ndarray, ref: np.ndarray, abs_allow: float = 0.0):
    """(mean abs error, max relative error); the relative error of an element
    is (|got-ref| - abs_allow)+ / max(|ref|, 0.1 rms(ref))."""
    err = np.maximum(np.abs(got - ref) - abs_allow, 0.0) if abs_allow else np.abs(got - ref)
    mae_err = np.abs(got - ref)
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0
    floor = np.maximum(np.abs(ref), 0.1 * rms)
    with np.errstate(divide="ignore", invalid="ignore"):
        rel = np.where(floor > 0, err / floor, np.where(err > 0, np.inf, 0.0))
    return float(mae_err.mean()) if err.size else 0.0, float(rel.max()) if rel.size else 0.0


def bf16_ulp(v: float) -> float:
    """Spacing of bf16 values at magnitude v (8 significant bits)."""
    return 2.0 ** (np.floor(np.log2(v)) - 7) if v > 0 else 0.0


def ffn_flip_allowance(h_ref: np.ndarray, w_down: np.ndarray) -> float:
    """Absolute allowance for the FFN output on the bf16 path.

    H is stored in bf16, so a kernel whose fp32 sums differ from fp64 in the
    last bits rounds a few H entries to the neighbouring bf16 value (a one-ulp
    flip; about 1e-4 of the entries).  Each flip moves one output by
    ulp(h) * |w_down|, whatever the size of that output, so near-zero outputs
    need an absolute allowance: two flips of the largest |h| times the largest
    |w_down|.  Computed from oracle values and inputs only."""
    return 2.0 * bf16_ulp(float(np.abs(h_ref).max())) * float(np.abs(w_down).max())


def assert_close(got, ref: np.ndarray, kind: str = "bf16", what: str = "", abs_allow: float = 0.0):
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


def attention_bound(orc, q, k, v, mask, n_seq, n_q, n_kv, hd, causal, T_k):
    """Per-element error bound of the bf16 attention path (probabilities
    rounded to bf16 for P.V: unit roundoff 2^-8 times attention applied to
    |V|; fp32 scores, exponentials and sums: (2^-12 + T_k 2^-24) of the
    same); the stored output's own bf16 rounding is added by the check."""
    from paper_2607_28418_amd import synth
    vabs = np.abs(synth.as_f32(v)).astype(np.float32)
    a_abs = orc.attention(synth.as_f32(q), synth.as_f32(k), vabs, mask, n_seq, n_q, n_kv, hd, causal)
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
