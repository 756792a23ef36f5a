"""The bf16 projection checks accept correct fp32 kernels and reject plausible
mistakes (CPU only).

The checks (tests/_helpers: check_ffn, check_nproj, check_kproj, built on the
rounding bands of tests/_bounds) compare a kernel's stored bf16 values with
the oracle, Section 3.1 equations (1)-(3).  Here the "kernels" are fp32
emulations on the CPU, in the summation orders the HIP kernels use
(sequential over 16-wide k blocks, eight interleaved 64-wide step classes,
torch's own blocked order), each rounding to bf16 where the kernels store.
They must pass.  Each mistake is planted in such an emulation (never in a
kernel): a (token, group) pair left out, a group computed with the
neighbouring group's weights, the last 16 k of a group left out of the K-axis
sum, and y computed from fp32 H instead of the stored bf16 H.  The checks
must reject every one, at the sizes of the GPU tests and at the full
Llama-3-8B widths.
"""
import numpy as np
import pytest
import torch

from paper_2607_28418_amd import synth
from tests._helpers import check_ffn, check_kproj, check_nproj


def _bf16(v32: np.ndarray) -> np.ndarray:
    """fp32 -> stored bf16 value (as float64), round to nearest even."""
    return synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(v32.astype(np.float32))).astype(np.float64)


def _dot32(x, w, order):
    """fp32 x [M][K] @ w [N][K]^T in one of the kernels' summation orders."""
    X, Wt = torch.from_numpy(np.ascontiguousarray(x, np.float32)), torch.from_numpy(np.ascontiguousarray(w, np.float32))
    K = X.shape[1]
    if order == "torch":
        return (X @ Wt.T).numpy()
    if order == "seq16":
        acc = torch.zeros(X.shape[0], Wt.shape[0], dtype=torch.float32)
        for b in range(0, K, 16):
            acc += X[:, b:b + 16] @ Wt[:, b:b + 16].T
        return acc.numpy()
    assert order == "waves8"
    part = [torch.zeros(X.shape[0], Wt.shape[0], dtype=torch.float32) for _ in range(8)]
    for s in range(K // 64):
        for h in (0, 32):
            k0 = s * 64 + h
            part[s % 8] += X[:, k0:k0 + 32] @ Wt[:, k0:k0 + 32].T
    tot = [part[i] + part[i + 4] for i in range(4)]
    return (((tot[0] + tot[1]) + tot[2]) + tot[3]).numpy()


def _silu32(a):
    a = a.astype(np.float32)
    return a * (np.float32(1.0) / (np.float32(1.0) + np.exp(-a)))


def _emu_ffn(c, order="seq16", mask=None, shift=None, skip_tail=None, unrounded_h=False):
    """An fp32 emulation of the bf16 FFN kernels, optionally with a mistake."""
    mask = c.mask if mask is None else mask
    X = synth.as_f32(c.x)
    Wg, Wu, Wd = (synth.as_f32(w) for w in (c.w_gate, c.w_up, c.w_down))
    if shift is not None:   # token t computes group g with group g+1's gate/up rows
        t, g = shift
        G = c.G
        Wg2, Wu2 = Wg.copy(), Wu.copy()
        Wg2[g * G:(g + 1) * G], Wu2[g * G:(g + 1) * G] = Wg[(g + 1) * G:(g + 2) * G], Wu[(g + 1) * G:(g + 2) * G]
        a2, b2 = _dot32(X[t:t + 1], Wg2, order), _dot32(X[t:t + 1], Wu2, order)
    a, b = _dot32(X, Wg, order), _dot32(X, Wu, order)
    if shift is not None:
        a[shift[0]], b[shift[0]] = a2[0], b2[0]
    h32 = _silu32(a) * b
    act = np.repeat(mask.astype(bool), c.G, axis=1)
    h32 = np.where(act, h32, np.float32(0))
    h = _bf16(h32)
    hin = h32 if unrounded_h else h.astype(np.float32)
    if skip_tail is not None:   # the K-axis sum leaves out the last 16 k of group g
        hin = hin.copy()
        g = skip_tail
        hin[:, (g + 1) * c.G - 16:(g + 1) * c.G] = 0
    y = _bf16(_dot32(hin, Wd, order))
    return h, y


def _rejects(fn):
    try:
        fn()
    except AssertionError:
        return True
    return False


SMALL = dict(seed=41, M=96, D=256, Dff=1024, G=128)
FULL = dict(seed=42, M=3, D=4096, Dff=14336, G=128)


@pytest.fixture(scope="module", params=["small", "full"])
def ffn_c(request):
    p = SMALL if request.param == "small" else FULL
    c = synth.ffn_case(p["seed"], p["M"], p["D"], p["Dff"], p["G"], mask="topk")
    c.mask[0, :] = 0   # one token with no active group: y row +0
    return c


@pytest.mark.parametrize("order", ["seq16", "waves8", "torch"])
def test_ffn_check_accepts_fp32_kernels(orc, ffn_c, order):
    h, y = _emu_ffn(ffn_c, order)
    check_ffn(orc, ffn_c, y, h)


def _first_active(c, t=1):
    return t, int(np.flatnonzero(c.mask[t])[0])


def test_ffn_check_rejects_a_dropped_pair(orc, ffn_c):
    m = ffn_c.mask.copy()
    t, g = _first_active(ffn_c)
    m[t, g] = 0
    h, y = _emu_ffn(ffn_c, mask=m)
    assert _rejects(lambda: check_ffn(orc, ffn_c, y, h))
    assert _rejects(lambda: check_ffn(orc, ffn_c, y))       # y alone catches it


def test_ffn_check_rejects_a_shifted_group(orc, ffn_c):
    t, g = _first_active(ffn_c)
    g = min(g, ffn_c.mask.shape[1] - 2)
    h, y = _emu_ffn(ffn_c, shift=(t, g))
    assert _rejects(lambda: check_ffn(orc, ffn_c, y, h))
    assert _rejects(lambda: check_ffn(orc, ffn_c, y))


def test_ffn_check_rejects_a_short_k_range(orc, ffn_c):
    g = int(np.flatnonzero(ffn_c.mask[1:].any(0))[0])
    h, y = _emu_ffn(ffn_c, skip_tail=g)
    assert _rejects(lambda: check_ffn(orc, ffn_c, y, h))


def test_ffn_check_rejects_unrounded_h(orc, ffn_c):
    h, y = _emu_ffn(ffn_c, unrounded_h=True)
    assert _rejects(lambda: check_ffn(orc, ffn_c, y, h))


# ---- Q (N axis) and O (K axis) --------------------------------------------------------

@pytest.fixture(scope="module", params=["small", "full"])
def attn_c(request):
    if request.param == "small":
        c = synth.attn_case(43, 96, 256, 8, 2, 128, 512, mask="topk")
    else:
        c = synth.attn_case(44, 3, 4096, 32, 8, 128, 512, mask="topk")
    c.mask[0, :] = 0
    return c


def _emu_q(c, order="seq16", mask=None, shift=None):
    mask = c.mask if mask is None else mask
    X, Wq = synth.as_f32(c.x), synth.as_f32(c.w_q)
    if shift is not None:
        t, g = shift
        Wq = Wq.copy()
        Wq[g * c.G:(g + 1) * c.G] = Wq[(g + 1) * c.G:(g + 2) * c.G].copy()
    q = _dot32(X, Wq, order)
    if shift is not None:
        q0 = _dot32(X, synth.as_f32(c.w_q), order)
        keep = np.ones(q.shape[0], bool)
        keep[shift[0]] = False
        q[keep] = q0[keep]
    return _bf16(np.where(np.repeat(mask.astype(bool), c.G, axis=1), q, np.float32(0)))


def _emu_o(c, order="seq16", mask=None, shift=None, skip_tail=None):
    mask = c.mask if mask is None else mask
    A = synth.as_f32(c.a) * np.repeat(mask.astype(bool), c.G, axis=1)
    Wo = synth.as_f32(c.w_o)
    if shift is not None:   # token t reads group g's inputs against group g+1's weight columns
        t, g = shift
        A = A.copy()
        A[t, (g + 1) * c.G:(g + 2) * c.G] = A[t, g * c.G:(g + 1) * c.G]
        A[t, g * c.G:(g + 1) * c.G] = 0
    if skip_tail is not None:
        A = A.copy()
        A[:, (skip_tail + 1) * c.G - 16:(skip_tail + 1) * c.G] = 0
    return _bf16(_dot32(A.astype(np.float32), Wo, order))


@pytest.mark.parametrize("order", ["seq16", "waves8", "torch"])
def test_q_k_o_checks_accept_fp32_kernels(orc, attn_c, order):
    c = attn_c
    check_nproj(orc, c.x, c.w_q, c.mask, c.G, _emu_q(c, order), what="q")
    check_nproj(orc, c.x, c.w_k, None, 0, _bf16(_dot32(synth.as_f32(c.x), synth.as_f32(c.w_k), order)), what="k")
    check_kproj(orc, c.a, c.w_o, c.mask, c.G, _emu_o(c, order), what="o")


def test_q_and_o_checks_reject_a_dropped_pair(orc, attn_c):
    c = attn_c
    m = c.mask.copy()
    t, g = _first_active(c)
    m[t, g] = 0
    assert _rejects(lambda: check_nproj(orc, c.x, c.w_q, c.mask, c.G, _emu_q(c, mask=m)))
    assert _rejects(lambda: check_kproj(orc, c.a, c.w_o, c.mask, c.G, _emu_o(c, mask=m)))


def test_q_and_o_checks_reject_a_shifted_group(orc, attn_c):
    c = attn_c
    t = 1
    g = int(np.flatnonzero(c.mask[t, :-1])[0])
    assert _rejects(lambda: check_nproj(orc, c.x, c.w_q, c.mask, c.G, _emu_q(c, shift=(t, g))))
    assert _rejects(lambda: check_kproj(orc, c.a, c.w_o, c.mask, c.G, _emu_o(c, shift=(t, g))))


def test_o_check_rejects_a_short_k_range(orc, attn_c):
    c = attn_c
    g = int(np.flatnonzero(c.mask[1:].any(0))[0])
    assert _rejects(lambda: check_kproj(orc, c.a, c.w_o, c.mask, c.G, _emu_o(c, skip_tail=g)))
