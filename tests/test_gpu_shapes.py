"""GPU parity at the benchmark's own shapes, and at the groups narrower than a tile.

Part 1 runs the Llama-3-8B layer exactly as the benchmark times it (d_model
4096, 32 q / 8 kv heads of 128 in 8 head groups of 512, d_ff 14336 in 112
groups of 128): prefill at T = 8192 and decode at 17, 24 and 32 tokens, and
the Llama-7B prefill FFN (config of Section 4 style kernel benchmarks) at
keep 0.75.  Prefill checks sampled token rows (rows are independent): the
first and last token, and for a few groups the tokens at the edges of that
group's boundary m-tile in the reorder (the last full tile's last row, the
partial tile's first row, the group's last active token and first inactive
one).  Decode checks every row and asserts through the timing labels which
kernel variants ran.

Part 2 covers group sizes 16 and 32 (Section 3.1: channel groups of 2^k,
k >= 4; Table 1 uses 32) and attention groups of one 64-wide head: prefill,
decode, degenerate masks, and weights of unused groups poisoned with NaN.

Part 3 runs prefill with token-row operands larger than 2 GiB, past what
the tile kernels' 32-bit buffer offsets reach, so the same kernels load
through 64-bit addresses: sampled rows on both sides of the 2 GiB line.
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


# ---------------------------------------------------------------- Llama-3-8B layer

P = synth.WORKLOADS["layer_llama3_8b"].params
D, DFF, G, NQ, NKV, HD, GA = P["D"], P["Dff"], P["G"], P["n_q"], P["n_kv"], P["hd"], P["G_attn"]


@pytest.fixture(scope="module")
def layer():
    say("layer weights (Llama-3-8B shapes)")
    g = synth.rng(2024)
    n = synth.normal
    w = dict(w_q=n(g, (NQ * HD, D), 0.02, "bf16"), w_k=n(g, (NKV * HD, D), 0.02, "bf16"),
             w_v=n(g, (NKV * HD, D), 0.02, "bf16"), w_o=n(g, (D, NQ * HD), 0.02, "bf16"),
             w_gate=n(g, (DFF, D), 0.02, "bf16"), w_up=n(g, (DFF, D), 0.02, "bf16"),
             w_down=n(g, (D, DFF), 0.02, "bf16"))
    dv = {k: to_dev(v) for k, v in w.items()}
    return w, dv


def _tokens(seed, M, keep):
    g = synth.rng(seed)
    x = synth.normal(g, (M, D), 1.0, "bf16")
    a = synth.normal(g, (M, NQ * HD), 1.0, "bf16")
    mf = synth.mask_topk(synth.router_logits(g, x, DFF // G), synth.keep_count(DFF // G, keep))
    ma = synth.mask_topk(synth.router_logits(g, x, NQ * HD // GA), synth.keep_count(NQ * HD // GA, keep))
    return x, a, mf, ma


def boundary_rows(orc, mask, groups, M, extra_seed, n_random=8):
    """Token rows at the edges of each listed group's boundary m-tile (256
    sorted positions per tile), the first and last token, and a few random."""
    idx, cnt = orc.mask_reorder(mask)
    rows = [0, M - 1]
    for g in groups:
        c = int(cnt[g])
        j = c // 256
        for p in (256 * j - 1, 256 * j, c - 1, c):
            if 0 <= p < M:
                rows.append(int(idx[g][p]))
    rows += list(synth.rng(extra_seed).integers(0, M, n_random))
    return np.unique(np.array(rows))


def test_layer_ffn_prefill_t8192(orc, layer):
    w, dv = layer
    M = 8192
    say("layer FFN prefill T=8192 d_ff 14336 G=128 keep 0.5")
    x, _, mf, _ = _tokens(11, M, 0.5)
    c = synth.FFNCase(x, w["w_gate"], w["w_up"], w["w_down"], mf, G, "bf16")
    h = torch.empty((M, DFF), dtype=torch.bfloat16, device=dev())
    y = W.wide_ffn_masked(to_dev(x), dv["w_gate"], dv["w_up"], dv["w_down"], to_dev(mf), G, h_out=h)
    torch.cuda.synchronize()
    rows = boundary_rows(orc, mf, (0, 55, 111), M, 5)
    check_ffn(orc, c, y, h, rows=rows, what="layer ffn")


def test_layer_qkvo_prefill_t8192(orc, layer):
    w, dv = layer
    M = 8192
    say("layer Q/K/V/O prefill T=8192 32q/8kv G=512 keep 0.5")
    x, a, _, ma = _tokens(12, M, 0.5)
    m = to_dev(ma)
    q, k, v = W.wide_qkvo_masked(W.PHASE_QKV, to_dev(x), m, GA, NQ, NKV, HD, w_q=dv["w_q"], w_k=dv["w_k"],
                                 w_v=dv["w_v"])
    y = W.wide_qkvo_masked(W.PHASE_O, to_dev(a), m, GA, NQ, NKV, HD, w_o=dv["w_o"])
    torch.cuda.synchronize()
    rows = boundary_rows(orc, ma, range(8), M, 6)
    check_nproj(orc, x, w["w_q"], ma, GA, q, rows=rows, what="q")
    check_nproj(orc, x, w["w_k"], None, 0, k, rows=rows, what="k")
    check_nproj(orc, x, w["w_v"], None, 0, v, rows=rows, what="v")
    check_kproj(orc, a, w["w_o"], ma, GA, y, rows=rows, what="o")


# decode: the variant every call must run (token blocks of 16, column or row
# blocks of 16 per workgroup), from the dispatch rules of the decode kernels:
# gate/up, Q/K/V, down (64 rows per workgroup, 4-way split of its 224 k
# steps) and O (16 rows, no split)
DECODE_VARIANTS = {
    B: ("wide_gemv_n<true>/ntb2_ncb4", "wide_gemv_n<false>/ntb2_ncb2", "wide_gemv_k/ntb2_ncb4",
        "wide_gemv_k/ntb2_ncb1") for B in (17, 24, 32)
}


@pytest.mark.parametrize("B", [17, 24, 32])
def test_layer_decode(orc, layer, B):
    w, dv = layer
    say("layer decode B", B)
    x, a, mf, ma = _tokens(100 + B, B, 0.5)
    W.wide_timing_enable(True)
    W.wide_timing_reset()
    h = torch.empty((B, DFF), dtype=torch.bfloat16, device=dev())
    y = W.wide_ffn_masked(to_dev(x), dv["w_gate"], dv["w_up"], dv["w_down"], to_dev(mf), G, h_out=h)
    m = to_dev(ma)
    q, k, v = W.wide_qkvo_masked(W.PHASE_QKV, to_dev(x), m, GA, NQ, NKV, HD, w_q=dv["w_q"], w_k=dv["w_k"],
                                 w_v=dv["w_v"])
    yo = W.wide_qkvo_masked(W.PHASE_O, to_dev(a), m, GA, NQ, NKV, HD, w_o=dv["w_o"])
    torch.cuda.synchronize()
    ran = {lbl: W.wide_timing_query(lbl)[1] for lbl in DECODE_VARIANTS[B]}
    W.wide_timing_enable(False)
    assert all(n == 1 for n in ran.values()), ran
    c = synth.FFNCase(x, w["w_gate"], w["w_up"], w["w_down"], mf, G, "bf16")
    check_ffn(orc, c, y, h, what=f"decode ffn B={B}")
    check_nproj(orc, x, w["w_q"], ma, GA, q, what="q")
    check_nproj(orc, x, w["w_k"], None, 0, k, what="k")
    check_nproj(orc, x, w["w_v"], None, 0, v, what="v")
    check_kproj(orc, a, w["w_o"], ma, GA, yo, what="o")


def test_prefill_ffn_llama7b_keep075(orc):
    say("ffn prefill llama7b T=4096 keep 0.75")
    c = synth.ffn_case(3, 4096, 4096, 11008, 128, mask="topk", keep=0.75)
    y = W.wide_ffn_masked(*(to_dev(t) for t in (c.x, c.w_gate, c.w_up, c.w_down, c.mask)), 128)
    torch.cuda.synchronize()
    rows = boundary_rows(orc, c.mask, (0, 40, 85), 4096, 7)
    check_ffn(orc, c, y, rows=rows, what="keep 0.75")


# ---------------------------------------------------------------- narrow groups

def ffn_dev(c):
    return [to_dev(a) for a in (c.x, c.w_gate, c.w_up, c.w_down)] + [to_dev(c.mask)]


@pytest.mark.parametrize("M,Dd,Dff,Gs,kind", [
    (300, 256, 1024, 16, "bernoulli"), (300, 256, 1024, 32, "bernoulli"), (1000, 512, 2048, 32, "topk"),
    (513, 256, 1152, 16, "beta"), (65, 256, 896, 32, "bernoulli"), (2100, 256, 512, 16, "topk")])
def test_ffn_small_groups_prefill(orc, M, Dd, Dff, Gs, kind):
    say("ffn small groups prefill", M, Dd, Dff, Gs, kind)
    W.wide_set_option("decode_max_m", 0)
    c = synth.ffn_case(M + Gs, M, Dd, Dff, Gs, mask=kind)
    x, wg, wu, wd, m = ffn_dev(c)
    h = torch.full((M, Dff), float("nan"), dtype=torch.bfloat16, device=dev())
    y = W.wide_ffn_masked(x, wg, wu, wd, m, Gs, h_out=h)
    y2 = W.wide_ffn_masked(x, wg, wu, wd, m, Gs)   # H kept in the workspace
    torch.cuda.synchronize()
    check_ffn(orc, c, y, h, what=f"G={Gs}")
    assert torch.equal(y.view(torch.int16), y2.view(torch.int16))


def test_ffn_small_groups_big_tiles_off(orc):
    """The narrow-group path ignores the tile-size option (its N axis needs
    the 256-row token-order tiles); the K axis runs on the 128 tiles."""
    say("ffn small groups big_tiles 0")
    W.wide_set_option("decode_max_m", 0)
    W.wide_set_option("big_tiles", 0)
    c = synth.ffn_case(77, 400, 256, 1024, 32, mask="bernoulli")
    x, wg, wu, wd, m = ffn_dev(c)
    h = torch.empty((400, 1024), dtype=torch.bfloat16, device=dev())
    y = W.wide_ffn_masked(x, wg, wu, wd, m, 32, h_out=h)
    torch.cuda.synchronize()
    check_ffn(orc, c, y, h, what="G=32 small tiles")


@pytest.mark.parametrize("B", [1, 4, 17, 32, 64])
@pytest.mark.parametrize("Gs", [16, 32])
def test_ffn_small_groups_decode(orc, B, Gs):
    say("ffn small groups decode", B, Gs)
    c = synth.ffn_case(B * 3 + Gs, B, 512, 1024, Gs, mask="beta")
    x, wg, wu, wd, m = ffn_dev(c)
    h = torch.full((B, 1024), float("nan"), dtype=torch.bfloat16, device=dev())
    y = W.wide_ffn_masked(x, wg, wu, wd, m, Gs, h_out=h)
    torch.cuda.synchronize()
    check_ffn(orc, c, y, h, what=f"decode G={Gs}")


@pytest.mark.parametrize("kind", ["zeros", "ones"])
@pytest.mark.parametrize("M", [8, 300])
@pytest.mark.parametrize("Gs", [16, 32])
def test_ffn_small_groups_degenerate(orc, kind, M, Gs):
    say("ffn small groups degenerate", kind, M, Gs)
    c = synth.ffn_case(5, M, 256, 512, Gs, mask=kind)
    x, wg, wu, wd, m = ffn_dev(c)
    h = torch.full((M, 512), float("nan"), dtype=torch.bfloat16, device=dev())
    y = torch.full((M, 256), float("nan"), dtype=torch.bfloat16, device=dev())
    W.wide_ffn_masked(x, wg, wu, wd, m, Gs, h_out=h, y=y)
    torch.cuda.synchronize()
    if kind == "zeros":
        assert not to_np64(y).any() and not to_np64(h).any()
        assert not torch.signbit(y.float()).any() and not torch.signbit(h.float()).any()
    else:
        check_ffn(orc, c, y, h)


@pytest.mark.parametrize("M", [40, 300])
@pytest.mark.parametrize("Gs", [16, 32])
def test_ffn_small_groups_poisoned_unused_blocks(orc, M, Gs):
    """Weights of a 64-wide block of groups that no token uses are never read
    (groups narrower than 64 are skipped 64 columns at a time on the K axis
    and per group on the N axis): NaN there changes nothing."""
    say("ffn small groups poison", M, Gs)
    c = synth.ffn_case(31 + Gs, M, 256, 1024, Gs, mask="bernoulli")
    per = 64 // Gs
    unused = [1, 5]                       # 64-wide blocks
    for b in unused:
        c.mask[:, b * per:(b + 1) * per] = 0
    # and single narrow groups inside otherwise used blocks: unused on the N axis
    c.mask[:, 9 * per] = 0
    x, wg, wu, wd, m = ffn_dev(c)
    y0 = W.wide_ffn_masked(x, wg, wu, wd, m, Gs).clone()
    nan = float("nan")
    for b in unused:
        wg[b * 64:(b + 1) * 64] = nan
        wu[b * 64:(b + 1) * 64] = nan
        wd[:, b * 64:(b + 1) * 64] = nan
    g9 = 9 * per
    wg[g9 * Gs:(g9 + 1) * Gs] = nan     # gate/up rows of the single unused group
    wu[g9 * Gs:(g9 + 1) * Gs] = nan
    y1 = W.wide_ffn_masked(x, wg, wu, wd, m, Gs)
    torch.cuda.synchronize()
    assert torch.isfinite(y1.float()).all()
    check_ffn(orc, c, y0, what="clean")
    check_ffn(orc, c, y1, what="poisoned")


def test_ffn_small_groups_fp32(orc):
    say("ffn fp32 G=16")
    c = synth.ffn_case(8, 100, 128, 256, 16, dtype="f32", mask="bernoulli")
    x, wg, wu, wd, m = ffn_dev(c)
    h = torch.empty((100, 256), dtype=torch.float32, device=dev())
    y = W.wide_ffn_masked(x, wg, wu, wd, m, 16, h_out=h)
    torch.cuda.synchronize()
    rh, ry = orc.ffn(c.x, c.w_gate, c.w_up, c.w_down, c.mask, 16)
    assert_close(h, rh, kind="f32", what="h")
    assert_close(y, ry, kind="f32", what="y")


def test_ffn_small_groups_full_width_sampled(orc, layer):
    """G = 32 at the Llama-3-8B widths (448 groups), T = 2048, sampled rows."""
    w, dv = layer
    M, Gs = 2048, 32
    say("ffn G=32 d_ff 14336 T=2048")
    g = synth.rng(91)
    x = synth.normal(g, (M, D), 1.0, "bf16")
    mf = synth.mask_topk(synth.router_logits(g, x, DFF // Gs), synth.keep_count(DFF // Gs, 0.5))
    c = synth.FFNCase(x, w["w_gate"], w["w_up"], w["w_down"], mf, Gs, "bf16")
    y = W.wide_ffn_masked(to_dev(x), dv["w_gate"], dv["w_up"], dv["w_down"], to_dev(mf), Gs)
    yd = W.wide_ffn_masked(to_dev(x[:32]), dv["w_gate"], dv["w_up"], dv["w_down"], to_dev(mf[:32]), Gs)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, 1, M - 1], synth.rng(92).integers(0, M, 8)]))
    check_ffn(orc, c, y, rows=rows, what="prefill G=32")
    check_ffn(orc, dataclasses.replace(c, x=x[:32], mask=mf[:32]), yd, what="decode G=32")


@pytest.mark.parametrize("M", [300, 24])
def test_qkvo_head_dim_64_groups_of_one_head(orc, M):
    """head_dim 64 with one head per group (G = 64): Q runs on token-order
    tiles, O on the K-axis kernels."""
    say("qkvo G=64 hd=64", M)
    c = synth.attn_case(M + 64, M, 256, 8, 4, 64, 64, mask="bernoulli")
    d = {k: to_dev(getattr(c, k)) for k in ("x", "w_q", "w_k", "w_v", "w_o", "a", "mask")}
    q, k, v = W.wide_qkvo_masked(W.PHASE_QKV, d["x"], d["mask"], 64, 8, 4, 64, w_q=d["w_q"], w_k=d["w_k"],
                                 w_v=d["w_v"])
    y = W.wide_qkvo_masked(W.PHASE_O, d["a"], d["mask"], 64, 8, 4, 64, w_o=d["w_o"])
    torch.cuda.synchronize()
    check_nproj(orc, c.x, c.w_q, c.mask, 64, q, what="q")
    check_nproj(orc, c.x, c.w_k, None, 0, k, what="k")
    check_nproj(orc, c.x, c.w_v, None, 0, v, what="v")
    check_kproj(orc, c.a, c.w_o, c.mask, 64, y, what="o")


def test_misaligned_mask_is_copied_by_the_binding(orc):
    """The library needs a 16-byte aligned mask; the binding copies a row
    slice that is not (8 groups: row 1 starts 8 bytes in)."""
    say("misaligned mask slice")
    c = synth.attn_case(3, 65, 256, 8, 2, 128, 128, mask="bernoulli")
    d = {k: to_dev(getattr(c, k)) for k in ("a", "w_o", "mask")}
    m1 = d["mask"][1:]
    assert m1.data_ptr() % 16 != 0
    y = W.wide_qkvo_masked(W.PHASE_O, d["a"][1:].contiguous(), m1, 128, 8, 2, 128, w_o=d["w_o"])
    torch.cuda.synchronize()
    check_kproj(orc, c.a[1:], c.w_o, c.mask[1:], 128, y, what="o")


# ------------------------------------------------------------------ part 3

class _Periodic:
    """Rows of an [M][D] matrix that repeats a block of P rows.  P is odd,
    so a row address off by any power of two lands on a different row."""

    def __init__(self, block):
        self.block = block

    def __getitem__(self, rows):
        return self.block[np.asarray(rows) % len(self.block)]


def _periodic_dev(block, M):
    b = to_dev(block)
    return b.repeat(-(-M // len(block)), 1)[:M].contiguous()


def _rows_across(M, edge, seed):
    return np.unique(np.concatenate([[0, edge - 1, edge, edge + 1, M - 1],
                                     synth.rng(seed).integers(0, M, 8)]))


def test_ffn_token_operands_past_2gib(orc):
    D, Dff, G, P = 4096, 4096, 128, 4099
    edge = (1 << 31) // (2 * D)  # first token row past 2 GiB of x (and of H: Dff = D)
    M = edge + 1500
    say("ffn prefill, x and H past 2 GiB: M", M)
    g = synth.rng(41)
    block = synth.normal(g, (P, D), 1.0, "bf16")
    wg = synth.normal(g, (Dff, D), 0.02, "bf16")
    wu = synth.normal(g, (Dff, D), 0.02, "bf16")
    wd = synth.normal(g, (D, Dff), 0.02, "bf16")
    mask = synth.make_mask(g, "bernoulli", M, Dff // G, 0.5)
    x = _periodic_dev(block, M)
    y = W.wide_ffn_masked(x, to_dev(wg), to_dev(wu), to_dev(wd), to_dev(mask), G)
    torch.cuda.synchronize()
    del x
    c = synth.FFNCase(_Periodic(block), wg, wu, wd, mask, G, "bf16")
    check_ffn(orc, c, y, rows=_rows_across(M, edge, 3), what="past 2 GiB")


def test_qkv_token_operand_past_2gib(orc):
    D, n_q, n_kv, hd, G, P = 4096, 4, 2, 128, 256, 4099
    edge = (1 << 31) // (2 * D)
    M = edge + 700
    say("q/k/v prefill, x past 2 GiB: M", M)
    g = synth.rng(43)
    block = synth.normal(g, (P, D), 1.0, "bf16")
    wq = synth.normal(g, (n_q * hd, D), 0.02, "bf16")
    wk = synth.normal(g, (n_kv * hd, D), 0.02, "bf16")
    wv = synth.normal(g, (n_kv * hd, D), 0.02, "bf16")
    mask = synth.make_mask(g, "bernoulli", M, n_q * hd // G, 0.5)
    x = _periodic_dev(block, M)
    q, k, v = W.wide_qkvo_masked(W.PHASE_QKV, x, to_dev(mask), G, n_q, n_kv, hd,
                                 w_q=to_dev(wq), w_k=to_dev(wk), w_v=to_dev(wv))
    torch.cuda.synchronize()
    del x
    rows = _rows_across(M, edge, 5)
    xs = _Periodic(block)
    check_nproj(orc, xs, wq, mask, G, q, rows=rows, what="q past 2 GiB")
    check_nproj(orc, xs, wk, None, 0, k, rows=rows, what="k past 2 GiB")
    check_nproj(orc, xs, wv, None, 0, v, rows=rows, what="v past 2 GiB")
