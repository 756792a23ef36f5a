"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Every case prints its name before it runs so that a failing GPU run names it.
Sizes: small cases span several tiles with ragged tails and are checked
element by element; full-size cases run the whole problem on the GPU and
check sampled token rows against the oracle (rows are independent).
"""
import dataclasses
import sys

import numpy as np
import pytest
import torch

import paper_2607_28418_amd as W
from paper_2607_28418_amd import synth
from tests._helpers import assert_close, check_ffn, check_kproj, check_nproj, dev, to_dev, to_np64

pytestmark = pytest.mark.gpu


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


@pytest.fixture(autouse=True)
def _options():
    W.lib()
    yield
    W.wide_set_option("decode_max_m", 64)
    W.wide_set_option("k_path", 0)
    W.wide_set_option("big_tiles", 1)
    W.wide_set_option("kd_pattern", 1)
    W.wide_set_option("mn_order", 7)
    W.wide_set_option("mn_tail", 1)
    for key in ("gemv_n_ncb", "gemv_n_split", "gemv_k_ncb", "gemv_k_split"):
        W.wide_set_option(key, 0)


def ffn_dev(c):
    return [to_dev(a) for a in (c.x, c.w_gate, c.w_up, c.w_down)] + [to_dev(c.mask)]


# ------------------------------------------------------------------ reorder

@pytest.mark.parametrize("M,ng,kind", [
    (1, 1, "bernoulli"), (7, 3, "bernoulli"), (255, 24, "bernoulli"), (256, 86, "beta"),
    (257, 86, "bernoulli"), (300, 4096, "bernoulli"), (2048, 8, "bernoulli"),
    (4096, 86, "topk"), (8192, 112, "topk"), (1000, 5, "zeros"), (1000, 5, "ones"),
    # single-kernel path up to 32768 tokens (1024-token chunks, ragged tails), three-kernel beyond
    (1024, 7, "bernoulli"), (1025, 3, "bernoulli"), (32768, 24, "bernoulli"), (32769, 24, "bernoulli"),
    (65573, 112, "topk"),
    # single-kernel path at its largest sizes and group counts of 32..128
    (64, 32, "ones"), (65, 48, "zeros"), (1000, 64, "bernoulli"), (32767, 128, "bernoulli"),
    (32768, 112, "topk")])
def test_reorder_bit_exact(orc, M, ng, kind):
    say("reorder", M, ng, kind)
    g = synth.rng(M + ng)
    if kind == "topk":
        x = g.standard_normal((M, 64), dtype=np.float32)
        mask = synth.mask_topk(synth.router_logits(g, x, ng), synth.keep_count(ng, 0.5))
    else:
        mask = synth.make_mask(g, kind, M, ng, 0.5)
    mask = mask * g.integers(1, 256, mask.shape).astype(np.uint8)   # any nonzero byte is active
    idx, cnt = W.wide_mask_reorder(to_dev(mask))
    torch.cuda.synchronize()
    ridx, rcnt = orc.mask_reorder(mask)
    assert np.array_equal(cnt.cpu().numpy(), rcnt)
    assert np.array_equal(idx.cpu().numpy(), ridx)


def test_reorder_empty():
    say("reorder M=0")
    idx, cnt = W.wide_mask_reorder(torch.zeros((0, 9), dtype=torch.uint8, device=dev()))
    torch.cuda.synchronize()
    assert idx.shape == (9, 0) and not cnt.cpu().numpy().any()


# ------------------------------------------------------------------ FFN bf16

@pytest.mark.parametrize("big", [1, 0])
@pytest.mark.parametrize("M,D,Dff,G,kind,kpath", [
    (300, 256, 512, 64, "bernoulli", 1), (300, 256, 512, 64, "bernoulli", 2),
    (129, 512, 1024, 128, "beta", 1), (129, 512, 1024, 128, "beta", 2),
    (1000, 256, 1024, 256, "topk", 0), (65, 256, 256, 128, "bernoulli", 1),
    (700, 512, 768, 128, "bernoulli", 2), (513, 256, 1024, 512, "topk", 1)])
def test_ffn_bf16_prefill_small(orc, M, D, Dff, G, kind, kpath, big):
    say("ffn prefill", M, D, Dff, G, kind, kpath, "big", big)
    W.wide_set_option("decode_max_m", 0)
    W.wide_set_option("k_path", kpath)
    W.wide_set_option("big_tiles", big)
    c = synth.ffn_case(M * 7 + G, M, D, Dff, G, mask=kind)
    x, wg, wu, wd, m = ffn_dev(c)
    h = torch.empty((M, Dff), dtype=torch.bfloat16, device=dev())
    y = W.wide_ffn_masked(x, wg, wu, wd, m, G, h_out=h)
    torch.cuda.synchronize()
    check_ffn(orc, c, y, h)


@pytest.mark.parametrize("B", [1, 4, 16, 33, 48, 64])
def test_ffn_bf16_decode_small(orc, B):
    say("ffn decode small", B)
    c = synth.ffn_case(B, B, 512, 1024, 128, mask="beta")
    x, wg, wu, wd, m = ffn_dev(c)
    h = torch.empty((B, 1024), dtype=torch.bfloat16, device=dev())
    y = W.wide_ffn_masked(x, wg, wu, wd, m, 128, h_out=h)
    torch.cuda.synchronize()
    check_ffn(orc, c, y, h)


# every decode variant the tuning options can select: column or row blocks
# per workgroup (1..8) and the split of the k steps over workgroups (with
# its finishing kernel)
DECODE_FORCED = [(1, 1, 1, 1), (2, 2, 2, 2), (4, 4, 4, 4), (8, 1, 8, 8), (8, 4, 8, 4), (2, 8, 4, 2)]


@pytest.mark.parametrize("B", [3, 24, 32, 64])
@pytest.mark.parametrize("n_ncb,n_split,k_ncb,k_split", DECODE_FORCED)
def test_decode_forced_variants(orc, B, n_ncb, n_split, k_ncb, k_split):
    say("decode forced variants B", B, "n", n_ncb, n_split, "k", k_ncb, k_split)
    W.wide_set_option("gemv_n_ncb", n_ncb)
    W.wide_set_option("gemv_n_split", n_split)
    W.wide_set_option("gemv_k_ncb", k_ncb)
    W.wide_set_option("gemv_k_split", k_split)
    c = synth.ffn_case(40 + B, B, 1024, 2048, 128, mask="beta")
    x, wg, wu, wd, m = ffn_dev(c)
    h = torch.empty((B, 2048), dtype=torch.bfloat16, device=dev())
    y = W.wide_ffn_masked(x, wg, wu, wd, m, 128, h_out=h)
    torch.cuda.synchronize()
    check_ffn(orc, c, y, h, what="ffn")
    check_qkvo(orc, synth.attn_case(50 + B, B, 1024, 8, 2, 128, 256, mask="topk"))


def test_ffn_decode_equals_prefill_rows(orc):
    """Rows are independent: a decode call on rows [0,16) and a prefill call on
    all 200 rows agree with the oracle and with each other on those rows."""
    say("ffn decode vs prefill rows")
    c = synth.ffn_case(11, 200, 512, 1024, 128, mask="bernoulli")
    x, wg, wu, wd, m = ffn_dev(c)
    y_pre = W.wide_ffn_masked(x, wg, wu, wd, m, 128)
    y_dec = W.wide_ffn_masked(x[:16].contiguous(), wg, wu, wd, m[:16].contiguous(), 128)
    torch.cuda.synchronize()
    check_ffn(orc, c, y_pre, rows=np.arange(16), what="prefill rows")
    check_ffn(orc, dataclasses.replace(c, x=c.x[:16], mask=c.mask[:16]), y_dec, what="decode rows")


@pytest.mark.parametrize("kind", ["zeros", "ones"])
@pytest.mark.parametrize("M", [5, 300])
def test_ffn_degenerate_masks(orc, kind, M):
    say("ffn degenerate", kind, M)
    c = synth.ffn_case(3, M, 256, 512, 64 if M > 64 else 128, mask=kind)
    G = c.G
    x, wg, wu, wd, m = ffn_dev(c)
    h = torch.full((M, 512), float("nan"), dtype=torch.bfloat16, device=dev())
    y = torch.full((M, 256), float("nan"), dtype=torch.bfloat16, device=dev())
    W.wide_ffn_masked(x, wg, wu, wd, m, G, h_out=h, y=y)
    torch.cuda.synchronize()
    if kind == "zeros":
        assert not to_np64(y).any() and not to_np64(h).any()
        assert not torch.signbit(y.float()).any()
    else:
        check_ffn(orc, c, y, h)


def test_ffn_m_zero_is_noop():
    say("ffn M=0")
    e = torch.empty((0, 256), dtype=torch.bfloat16, device=dev())
    w = torch.zeros((512, 256), dtype=torch.bfloat16, device=dev())
    wd = torch.zeros((256, 512), dtype=torch.bfloat16, device=dev())
    y = W.wide_ffn_masked(e, w, w, wd, torch.empty((0, 4), dtype=torch.uint8, device=dev()), 128)
    assert y.shape == (0, 256)


@pytest.mark.parametrize("M,kpath", [(40, 0), (300, 1), (300, 2)])
def test_ffn_poisoned_unused_groups(orc, M, kpath):
    """Weights of groups no token uses are never read: NaN there changes nothing."""
    say("ffn poison", M, kpath)
    W.wide_set_option("k_path", kpath)
    c = synth.ffn_case(21, M, 256, 1024, 128, mask="bernoulli")
    c.mask[:, [1, 5]] = 0
    x, wg, wu, wd, m = ffn_dev(c)
    y0 = W.wide_ffn_masked(x, wg, wu, wd, m, 128).clone()
    nan = float("nan")
    for gi in (1, 5):
        wg[gi * 128:(gi + 1) * 128] = nan
        wu[gi * 128:(gi + 1) * 128] = nan
        wd[:, gi * 128:(gi + 1) * 128] = nan
    y1 = W.wide_ffn_masked(x, wg, wu, wd, m, 128)
    torch.cuda.synchronize()
    assert torch.isfinite(y1.float()).all()
    check_ffn(orc, c, y0, what="clean")
    check_ffn(orc, c, y1, what="poisoned")


@pytest.mark.parametrize("pack", [3, 8])
def test_ffn_scatter_packs_groups_per_workgroup(orc, pack):
    """The atomic K-axis schedule with several K-groups run in turn by one
    workgroup (Appendix B, Algorithm 3's outer loop); 11 groups, so the last
    workgroup of a column tile gets fewer."""
    say("ffn scatter pack", pack)
    W.wide_set_option("decode_max_m", 0)
    W.wide_set_option("k_path", 2)
    W.wide_set_option("ks_pack", pack)
    try:
        c = synth.ffn_case(17 + pack, 700, 512, 11 * 128, 128, mask="topk")
        x, wg, wu, wd, m = ffn_dev(c)
        y = W.wide_ffn_masked(x, wg, wu, wd, m, 128)
        torch.cuda.synchronize()
        check_ffn(orc, c, y, what=f"pack {pack}")
    finally:
        W.wide_set_option("ks_pack", 1)


def test_ffn_reuses_given_reorder(orc):
    say("ffn given idx")
    c = synth.ffn_case(5, 400, 256, 512, 128, mask="bernoulli")
    x, wg, wu, wd, m = ffn_dev(c)
    idx, cnt = W.wide_mask_reorder(m)
    W.wide_set_option("k_path", 1)
    y_a = W.wide_ffn_masked(x, wg, wu, wd, m, 128, idx=idx, counts=cnt)
    y_b = W.wide_ffn_masked(x, wg, wu, wd, m, 128)
    torch.cuda.synchronize()
    assert torch.equal(y_a, y_b)   # dense-masked K path: no atomics, deterministic


@pytest.mark.parametrize("keep", [0.5, 0.25])
def test_ffn_bf16_prefill_full_llama7b_sampled(orc, keep):
    say("ffn prefill llama7b T=4096 keep", keep)
    c = synth.ffn_case(3, 4096, 4096, 11008, 128, mask="topk", keep=keep)
    x, wg, wu, wd, m = ffn_dev(c)
    y = W.wide_ffn_masked(x, wg, wu, wd, m, 128)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, 4095], synth.rng(0).integers(0, 4096, 14)]))
    check_ffn(orc, c, y, rows=rows, what="sampled rows")


@pytest.mark.parametrize("B", [1, 4, 16, 64])
def test_ffn_bf16_decode_full_llama7b(orc, B):
    say("ffn decode llama7b B", B)
    c = synth.ffn_case(2, B, 4096, 11008, 128, mask="beta")
    x, wg, wu, wd, m = ffn_dev(c)
    y = W.wide_ffn_masked(x, wg, wu, wd, m, 128)
    torch.cuda.synchronize()
    check_ffn(orc, c, y, what="decode rows")


# ------------------------------------------------------------------ FFN fp32

def test_ffn_fp32_small_full(orc):
    say("ffn fp32 D=512 Dff=1536 G=64 T=128")
    c = synth.ffn_case(1, 128, 512, 1536, 64, dtype="f32", mask="bernoulli")
    x, wg, wu, wd, m = ffn_dev(c)
    h = torch.empty((128, 1536), dtype=torch.float32, device=dev())
    y = W.wide_ffn_masked(x, wg, wu, wd, m, 64, h_out=h)
    torch.cuda.synchronize()
    rh, ry = orc.ffn(c.x, c.w_gate, c.w_up, c.w_down, c.mask, 64)
    assert_close(h, rh, kind="f32", what="h")
    assert_close(y, ry, kind="f32", what="y")


# ------------------------------------------------------------------ attention

def attn_dev(c):
    return {k: to_dev(getattr(c, k)) for k in ("x", "w_q", "w_k", "w_v", "w_o", "a", "mask")}


def check_qkvo(orc, c, kind="bf16", kpath=0):
    d = attn_dev(c)
    W.wide_set_option("k_path", kpath)
    q, k, v = W.wide_qkvo_masked(W.PHASE_QKV, d["x"], d["mask"], c.G, c.n_q, c.n_kv, c.hd,
                                 w_q=d["w_q"], w_k=d["w_k"], w_v=d["w_v"])
    y = W.wide_qkvo_masked(W.PHASE_O, d["a"], d["mask"], c.G, c.n_q, c.n_kv, c.hd, w_o=d["w_o"])
    torch.cuda.synchronize()
    if kind == "bf16":
        check_nproj(orc, c.x, c.w_q, c.mask, c.G, q, what="q")
        check_nproj(orc, c.x, c.w_k, None, 0, k, what="k")
        check_nproj(orc, c.x, c.w_v, None, 0, v, what="v")
        check_kproj(orc, c.a, c.w_o, c.mask, c.G, y, what="o")
        return
    assert_close(q, orc.nproj(c.x, c.w_q, c.mask, c.G), kind, "q")
    assert_close(k, orc.linear(c.x, c.w_k), kind, "k")
    assert_close(v, orc.linear(c.x, c.w_v), kind, "v")
    assert_close(y, orc.kproj(c.a, c.w_o, c.mask, c.G), kind, "o")


@pytest.mark.parametrize("big", [1, 0])
@pytest.mark.parametrize("M,n_q,n_kv,G,kpath", [
    (300, 8, 2, 512, 1), (300, 8, 2, 512, 2), (130, 8, 4, 256, 0), (40, 8, 2, 512, 0),
    (1, 8, 8, 128, 0), (64, 16, 4, 512, 0), (600, 16, 4, 512, 2), (257, 8, 2, 128, 1)])
def test_qkvo_bf16_small(orc, M, n_q, n_kv, G, kpath, big):
    say("qkvo bf16", M, n_q, n_kv, G, kpath, "big", big)
    W.wide_set_option("big_tiles", big)
    c = synth.attn_case(M + G, M, 256, n_q, n_kv, 128, G, mask="topk")
    check_qkvo(orc, c, kpath=kpath)


def test_qkvo_fp32_small(orc):
    say("qkvo fp32")
    c = synth.attn_case(4, 70, 128, 8, 2, 32, 64, dtype="f32", mask="bernoulli")
    check_qkvo(orc, c, kind="f32")


@pytest.mark.parametrize("n_q,n_kv,hd,G", [(8, 2, 128, 256), (64, 8, 128, 128), (136, 8, 64, 64)])
def test_o_poisoned_inactive_blocks(orc, n_q, n_kv, hd, G):
    """Inactive blocks of the attention output are never read: 4, 64 and 136
    groups cover the dense-masked K axis with its rows' mask words in
    registers (up to 32 and up to 128 groups) and in LDS (beyond)."""
    for M, kpath in ((300, 1), (300, 2), (20, 0)):
        say("o poison", n_q, hd, G, M, kpath)
        W.wide_set_option("k_path", kpath)
        c = synth.attn_case(9, M, 256, n_q, n_kv, hd, G, mask="bernoulli")
        d = attn_dev(c)
        a = d["a"].clone()
        inactive = torch.from_numpy(np.repeat(c.mask == 0, c.G, axis=1)).to(dev())
        a[inactive] = float("nan")
        y = W.wide_qkvo_masked(W.PHASE_O, a, d["mask"], c.G, n_q, n_kv, hd, w_o=d["w_o"])
        torch.cuda.synchronize()
        check_kproj(orc, c.a, c.w_o, c.mask, c.G, y, what="o poisoned")


@pytest.mark.parametrize("name", ["attn_proj_mha", "layer_llama3_8b"])
def test_qkvo_bf16_full_sampled(orc, name):
    p = synth.WORKLOADS[name].params
    say("qkvo full", name)
    M = 2048
    c = synth.attn_case(4, M, p["D"], p["n_q"], p["n_kv"], p["hd"], p.get("G_attn", p.get("G")),
                        mask="topk")
    d = attn_dev(c)
    q, k, v = W.wide_qkvo_masked(W.PHASE_QKV, d["x"], d["mask"], c.G, c.n_q, c.n_kv, c.hd,
                                 w_q=d["w_q"], w_k=d["w_k"], w_v=d["w_v"])
    y = W.wide_qkvo_masked(W.PHASE_O, d["a"], d["mask"], c.G, c.n_q, c.n_kv, c.hd, w_o=d["w_o"])
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, M - 1], synth.rng(2).integers(0, M, 10)]))
    check_nproj(orc, c.x, c.w_q, c.mask, c.G, q, rows=rows, what="q")
    check_nproj(orc, c.x, c.w_k, None, 0, k, rows=rows, what="k")
    check_nproj(orc, c.x, c.w_v, None, 0, v, rows=rows, what="v")
    check_kproj(orc, c.a, c.w_o, c.mask, c.G, y, rows=rows, what="o")


# ------------------------------------------------------------------ graphs

@pytest.mark.parametrize("M", [24, 600])
def test_calls_replay_in_hip_graph(orc, M):
    """Decode and prefill calls captured in one HIP graph: every replay (with
    eager work and syncs in between) equals the eager result."""
    say("graph replay", M)
    W.wide_set_option("k_path", 1)   # deterministic K path: replays compare bitwise
    c = synth.ffn_case(M + 1, M, 512, 1024, 128, mask="topk")
    x, wg, wu, wd, m = ffn_dev(c)
    ca = synth.attn_case(M + 2, M, 512, 8, 2, 128, 512, mask="topk")
    d = attn_dev(ca)
    y = torch.empty((M, 512), dtype=torch.bfloat16, device=dev())
    q = torch.empty((M, 1024), dtype=torch.bfloat16, device=dev())
    kk = torch.empty((M, 256), dtype=torch.bfloat16, device=dev())
    vv = torch.empty((M, 256), dtype=torch.bfloat16, device=dev())
    yo = torch.empty((M, 512), dtype=torch.bfloat16, device=dev())
    ws = torch.empty(max(W.wide_workspace_size(W.OP_FFN, W.BF16, M, 512, 1024, 128),
                         W.wide_workspace_size(W.OP_QKV, W.BF16, M, 512, 1024, 512),
                         W.wide_workspace_size(W.OP_O, W.BF16, M, 512, 1024, 512)),
                     dtype=torch.uint8, device=dev())

    def step():
        W.wide_ffn_masked(x, wg, wu, wd, m, 128, y=y, ws=ws)
        W.wide_qkvo_masked(W.PHASE_QKV, d["x"], d["mask"], 512, 8, 2, 128, w_q=d["w_q"], w_k=d["w_k"],
                           w_v=d["w_v"], q=q, k=kk, v=vv, ws=ws)
        W.wide_qkvo_masked(W.PHASE_O, d["a"], d["mask"], 512, 8, 2, 128, w_o=d["w_o"], y=yo, ws=ws)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (y, q, kk, vv, yo)]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for _ in range(3):
        for t in (y, q, kk, vv, yo):
            t.fill_(7.0)          # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for got, want in zip((y, q, kk, vv, yo), ref):
            assert torch.equal(got, want)
    check_ffn(orc, c, y)


# ------------------------------------------------------------------ errors, timing

def test_errors_leave_outputs_untouched():
    say("errors")
    x = torch.zeros((8, 256), dtype=torch.bfloat16, device=dev())
    w = torch.zeros((480, 256), dtype=torch.bfloat16, device=dev())
    wd = torch.zeros((256, 480), dtype=torch.bfloat16, device=dev())
    y = torch.full((8, 256), 3.0, dtype=torch.bfloat16, device=dev())
    with pytest.raises(W.WideError) as ei:
        W.wide_ffn_masked(x, w, w, wd, torch.ones((8, 10), dtype=torch.uint8, device=dev()), 48, y=y,
                          ws=torch.empty(1 << 20, dtype=torch.uint8, device=dev()))
    assert ei.value.status == 1 and "power of two" in str(ei.value)
    torch.cuda.synchronize()
    assert (y.float() == 3.0).all()


def test_timing_records_kernels():
    say("timing")
    c = synth.ffn_case(1, 256, 256, 512, 128, mask="bernoulli")
    x, wg, wu, wd, m = ffn_dev(c)
    W.wide_timing_enable(True)
    W.wide_timing_reset()
    W.wide_ffn_masked(x, wg, wu, wd, m, 128)
    ms, n = W.wide_timing_query("wide_mn256<true>")
    W.wide_timing_enable(False)
    assert n == 1 and ms > 0


def test_timing_filter_times_only_matching_launches():
    say("timing filter")
    c = synth.ffn_case(1, 256, 256, 512, 128, mask="bernoulli")
    x, wg, wu, wd, m = ffn_dev(c)
    W.wide_timing_enable(True)
    W.wide_timing_reset()
    try:
        W.wide_timing_filter("wide_mn256<true>")
        W.wide_ffn_masked(x, wg, wu, wd, m, 128)
        W.wide_timing_filter(None)
        W.wide_ffn_masked(x, wg, wu, wd, m, 128)
        n_up = W.wide_timing_query("wide_mn256<true>")[1]
        n_down = W.wide_timing_query("wide_kd256")[1]
    finally:
        W.wide_timing_filter(None)
        W.wide_timing_enable(False)
    assert n_up == 2 and n_down == 1


# ------------------------------------------------------------------ router

def _router_case(M, D, r, ng, seed):
    g = synth.rng(seed)
    x = synth.normal(g, (M, D), 1.0, "bf16")
    w1 = synth.normal(g, (r, D), 0.02, "bf16")
    w2 = synth.normal(g, (2 * ng, r), 0.3, "bf16")
    return x, w1, w2


def _router_bound(x, w1, w2):
    """Bound on |fp32 logit - fp64 logit| from the kernel's arithmetic: X W1 is
    a sum of D exact bf16 products in fp32 (any order), then r fp32 FMAs with
    W2.  gamma_n = n u / (1 - n u), u = 2^-24."""
    u = 2.0 ** -24
    X, W1, W2 = (synth.as_f32(a).astype(np.float64) for a in (x, w1, w2))
    D, r = X.shape[1], W1.shape[0]
    gD, gr = D * u / (1 - D * u), (r + 1) * u / (1 - (r + 1) * u)
    dh = gD * (np.abs(X) @ np.abs(W1).T)
    h = np.abs(X @ W1.T)
    return dh @ np.abs(W2).T + gr * ((h + dh) @ np.abs(W2).T)


@pytest.mark.parametrize("M,D,r,ng", [
    (1, 64, 16, 3), (33, 128, 32, 24), (300, 4096, 32, 112), (257, 4096, 7, 300),
    (64, 4096, 16, 8), (2048, 4096, 32, 8), (8192, 4096, 32, 112)])
def test_router_matches_oracle(orc, M, D, r, ng):
    say("router", M, D, r, ng)
    x, w1, w2 = _router_case(M, D, r, ng, M + D + r + ng)
    mask, lg, idx, cnt = W.wide_router(to_dev(x), to_dev(w1), to_dev(w2), logits=True, reorder=True)
    torch.cuda.synchronize()
    ref_lg, ref_mask = orc.router(x, w1, w2)
    bound = _router_bound(x, w1, w2)
    got_lg = lg.cpu().numpy().astype(np.float64)
    assert (np.abs(got_lg - ref_lg) <= bound).all(), float(np.max(np.abs(got_lg - ref_lg) - bound))
    # the decision is fixed wherever the pair's gap exceeds both logits' bounds
    gap = np.abs(ref_lg[:, 0::2] - ref_lg[:, 1::2])
    amb = gap <= bound[:, 0::2] + bound[:, 1::2]
    got_mask = mask.cpu().numpy()
    assert np.array_equal(got_mask[~amb], ref_mask[~amb])
    # inside the band either class is correct; the kernel must still follow its own logits
    assert np.array_equal(got_mask, (got_lg[:, 0::2] >= got_lg[:, 1::2]).astype(np.uint8))
    assert amb.mean() < 0.1   # the bound is a worst case (about 5% of pairs at d_model 4096)
    # the reorder returned with it is that of the returned mask
    ridx, rcnt = orc.mask_reorder(got_mask)
    assert np.array_equal(cnt.cpu().numpy(), rcnt) and np.array_equal(idx.cpu().numpy(), ridx)


def test_router_ties_execute():
    say("router ties")
    g = synth.rng(5)
    x = synth.normal(g, (40, 128), 1.0, "bf16")
    w1 = synth.normal(g, (16, 128), 0.02, "bf16")
    half = synth.normal(g, (5, 16), 0.3, "bf16")
    w2 = np.repeat(half, 2, axis=0)            # both classes of each group identical
    mask = W.wide_router(to_dev(x), to_dev(w1), to_dev(w2))
    torch.cuda.synchronize()
    assert mask.cpu().numpy().all()


def test_router_empty_batch():
    say("router M=0")
    mask, idx, cnt = W.wide_router(torch.zeros((0, 64), dtype=torch.bfloat16, device=dev()),
                                   torch.zeros((16, 64), dtype=torch.bfloat16, device=dev()),
                                   torch.zeros((6, 16), dtype=torch.bfloat16, device=dev()), reorder=True)
    torch.cuda.synchronize()
    assert mask.shape == (0, 3) and idx.shape == (3, 0) and not cnt.cpu().numpy().any()


# ------------------------------------------------------------------ M axis (one group)

@pytest.mark.parametrize("M,big,decode", [(300, 1, 0), (300, 0, 0), (8, 1, 1), (513, 1, 0)])
def test_ffn_single_group_m_axis(orc, M, big, decode):
    """group_size = d_ff: each token runs the whole FFN or skips it (App. A's
    M-axis case); d_ff = 1152 is no power of two."""
    say("ffn single group", M, "big", big, "decode", decode)
    W.wide_set_option("decode_max_m", 64 if decode else 0)
    W.wide_set_option("big_tiles", big)
    D, Dff = 256, 1152
    c = synth.ffn_case(M + 3, M, D, Dff, Dff, mask="bernoulli")
    x, wg, wu, wd, m = ffn_dev(c)
    h = torch.empty((M, Dff), dtype=torch.bfloat16, device=dev())
    y = W.wide_ffn_masked(x, wg, wu, wd, m, Dff, h_out=h)
    torch.cuda.synchronize()
    assert 0 < c.mask.mean() < 1
    check_ffn(orc, c, y, h)
    yn = to_np64(y)
    assert not yn[c.mask[:, 0] == 0].any()


def test_ffn_single_group_fp32(orc):
    say("ffn single group fp32")
    c = synth.ffn_case(9, 100, 128, 240, 240, dtype="f32", mask="bernoulli")
    x, wg, wu, wd, m = ffn_dev(c)
    y = W.wide_ffn_masked(x, wg, wu, wd, m, 240)
    torch.cuda.synchronize()
    _, ry = orc.ffn(c.x, c.w_gate, c.w_up, c.w_down, c.mask, 240)
    assert_close(y, ry, kind="f32", what="y")


@pytest.mark.parametrize("M", [300, 24])
def test_qkvo_single_group_m_axis(orc, M):
    """group_size = n_q*head_dim: all heads form one group."""
    say("qkvo single group", M)
    c = synth.attn_case(M + 1, M, 512, 8, 2, 128, 1024, mask="bernoulli")
    check_qkvo(orc, c)


@pytest.mark.parametrize("M,n_q,n_kv,G,kind", [(600, 16, 4, 256, "topk"), (777, 32, 8, 512, "bernoulli"),
                                               (40000, 8, 2, 256, "bernoulli"),  # three-kernel sort
                                               (300, 8, 2, 512, "topk")])
def test_o_pattern_order_is_bitwise_same(orc, M, n_q, n_kv, G, kind):
    """Reading the rows of the dense-masked K axis in mask-pattern order only
    skips k steps whose contributions are exact zeros: outputs are bitwise
    equal with and without it (and match the oracle)."""
    say("o pattern order", M, n_q, n_kv, G, kind)
    c = synth.attn_case(M + G, M, 512, n_q, n_kv, 128, G, mask=kind)
    d = attn_dev(c)
    outs = []
    for on in (1, 0):
        W.wide_set_option("kd_pattern", on)
        outs.append(W.wide_qkvo_masked(W.PHASE_O, d["a"], d["mask"], G, n_q, n_kv, 128, w_o=d["w_o"]))
    W.wide_set_option("kd_pattern", 1)
    torch.cuda.synchronize()
    assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16))
    rows = np.arange(M) if M <= 1000 else np.sort(synth.rng(M).choice(M, 64, replace=False))
    check_kproj(orc, c.a, c.w_o, c.mask, G, outs[0], rows=rows, what="o")


def _edge_count_mask(g, M, ng):
    """Per-group active counts that hit every tile-order case: none, all,
    whole 256-row tiles, one row more or less than a tile, random."""
    mask = synth.mask_bernoulli(g, M, ng, 0.5)
    forced = [0, M, 512, 256, 257, 255, 1, min(M, 768)]
    for j, c in enumerate(forced[:ng]):
        col = np.zeros(M, np.uint8)
        col[g.permutation(M)[:c]] = 1
        mask[:, j] = col
    return mask


@pytest.mark.parametrize("order", [6, 2, 0])
@pytest.mark.parametrize("M,ng", [(1000, 16), (700, 24), (1300, 8), (256, 8)])
def test_ffn_tile_order_edge_counts(orc, M, ng, order):
    """Each XCD's share of gate/up tiles runs m-tile by m-tile over its
    groups (6), or its full tiles, then partial, then empty ones (2), or
    group by group (0); every (group, m-tile) must still be written once."""
    say("ffn tile order", M, ng, order)
    W.wide_set_option("decode_max_m", 0)
    W.wide_set_option("mn_order", order)
    G = 128
    c = synth.ffn_case(M + ng, M, 256, ng * G, G)
    c.mask[:] = _edge_count_mask(synth.rng(M * 3 + ng), M, ng)
    x, wg, wu, wd, m = ffn_dev(c)
    h = torch.full((M, ng * G), 7.0, dtype=torch.bfloat16, device=dev())
    y = W.wide_ffn_masked(x, wg, wu, wd, m, G, h_out=h)
    y2 = W.wide_ffn_masked(x, wg, wu, wd, m, G)  # H kept in the workspace
    torch.cuda.synchronize()
    check_ffn(orc, c, y, h)
    assert torch.equal(y.view(torch.int16), y2.view(torch.int16))


@pytest.mark.parametrize("order", [0, 1, 2, 3])
@pytest.mark.parametrize("M", [1000, 300])
def test_qkv_tile_order_edge_counts(orc, M, order):
    """Q (8 masked groups) before or after the dense K and V regions, with or
    without the per-XCD full/partial/empty order inside Q."""
    say("qkv tile order", M, order)
    W.wide_set_option("mn_order", order)
    c = synth.attn_case(M + 11, M, 256, 16, 4, 128, 256, mask="bernoulli")
    c.mask[:] = _edge_count_mask(synth.rng(M * 5), M, 8)
    check_qkvo(orc, c, kpath=0)


@pytest.mark.parametrize("Dff", [2048, 2112, 6144, 8192, 8704])
def test_ffn_kd256_group_counts(orc, Dff):
    """The dense-masked K-axis kernel keeps the tile rows' mask words in
    registers for up to 32 and up to 128 groups and reads them from LDS
    beyond; 32, 33, 96, 128 and 136 groups of 64 cover each form and edge."""
    M, D, G = 300, 256, 64
    say("ffn kd256 groups", Dff // G)
    W.wide_set_option("decode_max_m", 0)
    W.wide_set_option("k_path", 1)
    c = synth.ffn_case(Dff + 5, M, D, Dff, G, mask="bernoulli")
    x, wg, wu, wd, m = ffn_dev(c)
    y = W.wide_ffn_masked(x, wg, wu, wd, m, G)
    torch.cuda.synchronize()
    check_ffn(orc, c, y)


@pytest.mark.parametrize("M,D,Dff", [(1000, 256, 2048), (3000, 512, 4096), (300, 256, 1024)])
def test_ffn_tail_split_matches(orc, M, D, Dff):
    """The tail split (each XCD's last partial round cut along k) serves
    Q/K/V only; gate/up runs its last round whole, so the FFN matches the
    oracle with the option on or off."""
    say("ffn tail split", M, D, Dff)
    W.wide_set_option("decode_max_m", 0)
    G = 128
    c = synth.ffn_case(M + D, M, D, Dff, G, mask="topk")
    x, wg, wu, wd, m = ffn_dev(c)
    for tail in (1, 0):
        W.wide_set_option("mn_tail", tail)
        h = torch.full((M, Dff), 7.0, dtype=torch.bfloat16, device=dev())
        y = W.wide_ffn_masked(x, wg, wu, wd, m, G, h_out=h)
        torch.cuda.synchronize()
        check_ffn(orc, c, y, h, what=f"tail={tail}")
    W.wide_set_option("mn_tail", 1)


@pytest.mark.parametrize("order", [2, 3])
@pytest.mark.parametrize("M", [1000, 2600])
def test_qkv_tail_split_matches(orc, M, order):
    say("qkv tail split", M, order)
    W.wide_set_option("mn_order", order)
    c = synth.attn_case(M + 13, M, 512, 16, 4, 128, 256, mask="topk")
    for tail in (1, 0):
        W.wide_set_option("mn_tail", tail)
        check_qkvo(orc, c, kpath=0)
    W.wide_set_option("mn_tail", 1)
