"""GPU parity of the head-group masked attention (prefill) against the fp64
oracle, through the C ABI.

Tolerance, derived from the kernel's arithmetic (it rounds the softmax
probabilities P to bf16 for the P.V product and stores o in bf16): with unit
roundoff u = 2^-8, the rounded P moves an output by at most
u * sum_j w_j |v_j|, i.e. u times attention applied to |V| (w = the softmax
weights), which the oracle computes; fp32 scores, exponentials and sums add
at most (2^-12 + T_k 2^-24) of the same quantity; storing o in bf16 adds at
most one bf16 ulp of the stored value.  Every element must satisfy the bound
(inactive rows: exactly +0), and the mean error must stay under 1e-3.
"""
import sys

import numpy as np
import pytest
import torch

import paper_2607_28418_amd as W
from paper_2607_28418_amd import synth
from tests._helpers import attention_bound, check_attention_rows as check_rows, dev, to_dev, to_np64

pytestmark = pytest.mark.gpu


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def run_case(orc, n_seq, T_q, T_k, n_q, n_kv, G, causal, mask="topk", keep=0.5, qk_std=1.0, seed=0,
             given_reorder=False, leftpad=None):
    hd = 128
    ng = n_q * hd // G
    c = synth.attn_prefill_case(seed, n_seq, T_q, T_k, n_q, n_kv, hd, ng, mask=mask, keep=keep,
                                qk_std=qk_std)
    q, k, v, m = (to_dev(a) for a in (c.q, c.k, c.v, c.mask))
    o = torch.full_like(q, float("nan"))   # every element must be written
    idx = cnt = None
    if given_reorder:
        idx, cnt = W.wide_mask_reorder(m)
    lp = None if leftpad is None else to_dev(np.asarray(leftpad, np.int32))
    W.wide_attention_masked(q, k, v, m, n_seq, n_q, n_kv, hd, G, causal, idx=idx, counts=cnt, o=o, leftpad=lp)
    torch.cuda.synchronize()
    got = to_np64(o)
    ref = orc.attention(c.q, c.k, c.v, c.mask, n_seq, n_q, n_kv, hd, causal, leftpad=leftpad)
    bound = attention_bound(orc, c.q, c.k, c.v, c.mask, n_seq, n_q, n_kv, hd, causal, T_k, leftpad=leftpad)
    check_rows(got, ref, bound, c.mask, G, f"attention {n_seq}x{T_q}/{T_k} {n_q}/{n_kv} G={G}")
    return c, got


@pytest.mark.parametrize("n_seq,T_q,T_k,n_q,n_kv,G,causal,mask,qk_std", [
    (1, 200, 200, 8, 2, 256, True, "topk", 1.0),      # two heads per workgroup
    (2, 150, 150, 4, 4, 128, True, "bernoulli", 1.0),  # one head, 128 rows per workgroup
    (1, 300, 300, 8, 2, 512, True, "topk", 1.0),      # four heads of one KV head per workgroup
    (3, 70, 130, 8, 2, 512, True, "topk", 1.0),       # queries after a 60-key prefix, 3 sequences
    (2, 100, 37, 4, 1, 256, False, "bernoulli", 1.0),  # non-causal, ragged key tile, T_k < T_q
    (1, 64, 64, 2, 2, 128, True, "bernoulli", 2.5),   # peaked softmax
    (5, 1, 77, 8, 2, 512, True, "bernoulli", 1.0),    # one query per sequence
    (2, 257, 257, 32, 8, 512, True, "topk", 1.5),     # Llama-3-8B heads
    (1, 129, 129, 8, 8, 1024, False, "bernoulli", 1.0),
])
def test_attention_matches_oracle(orc, n_seq, T_q, T_k, n_q, n_kv, G, causal, mask, qk_std):
    say("attention", n_seq, T_q, T_k, n_q, n_kv, G, causal, mask, qk_std)
    run_case(orc, n_seq, T_q, T_k, n_q, n_kv, G, causal, mask=mask, qk_std=qk_std, seed=T_q + n_q)


@pytest.mark.parametrize("n_seq,T_q,T_k,n_q,n_kv,G,causal,leftpad", [
    (3, 200, 200, 8, 2, 512, True, [0, 37, 130]),       # padding queries see no key: +0
    (2, 70, 130, 8, 2, 256, True, [60, 129]),           # after a prefix; the tile of key 129 only
    (2, 100, 100, 4, 4, 128, False, [5, 99]),
    (2, 257, 257, 32, 8, 512, True, [64, 200]),         # a tile-aligned first key; Llama-3-8B heads
    (2, 64, 64, 8, 2, 512, True, [64, 0]),              # every key hidden in one sequence
    (1, 1000, 1000, 8, 2, 512, True, [300]),            # one sequence: the key-range split is off
])
def test_attention_left_padding(orc, n_seq, T_q, T_k, n_q, n_kv, G, causal, leftpad):
    """Algorithm 4's first key leftpad(b): keys before it are hidden."""
    say("attention leftpad", n_seq, T_q, T_k, n_q, n_kv, G, causal, leftpad)
    c, got = run_case(orc, n_seq, T_q, T_k, n_q, n_kv, G, causal, mask="bernoulli", keep=0.7,
                      seed=T_q + sum(leftpad), leftpad=leftpad)
    if causal:   # queries before the padding's end see nothing: exactly +0
        for b, lp in enumerate(leftpad):
            first = max(0, lp - (T_k - T_q))
            assert not got[b * T_q:b * T_q + first].any()


@pytest.mark.parametrize("kind", ["zeros", "ones"])
def test_attention_degenerate_masks(orc, kind):
    say("attention mask", kind)
    run_case(orc, 2, 96, 96, 8, 2, 512, True, mask=kind)


def test_attention_given_reorder_is_bitwise_same(orc):
    say("attention given reorder")
    c, got = run_case(orc, 2, 180, 180, 8, 2, 256, True, seed=3)
    _, got2 = run_case(orc, 2, 180, 180, 8, 2, 256, True, seed=3, given_reorder=True)
    assert np.array_equal(got, got2)


def test_attention_never_reads_inactive_queries(orc):
    say("attention poisoned inactive q")
    n_seq, T, n_q, n_kv, G, hd = 1, 160, 8, 2, 256, 128
    c = synth.attn_prefill_case(11, n_seq, T, T, n_q, n_kv, hd, n_q * hd // G)
    q, k, v, m = (to_dev(a) for a in (c.q, c.k, c.v, c.mask))
    o1 = W.wide_attention_masked(q, k, v, m, n_seq, n_q, n_kv, hd, G, True)
    inactive = ~np.repeat(c.mask.astype(bool), G, axis=1)
    qp = q.clone()
    qp[torch.from_numpy(inactive).to(dev())] = float("nan")
    o2 = W.wide_attention_masked(qp, k, v, m, n_seq, n_q, n_kv, hd, G, True)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))


def test_attention_empty():
    say("attention empty")
    z = torch.zeros((0, 256), dtype=torch.bfloat16, device=dev())
    zk = torch.zeros((0, 128), dtype=torch.bfloat16, device=dev())
    o = W.wide_attention_masked(z, zk, zk, torch.zeros((0, 2), dtype=torch.uint8, device=dev()),
                                1, 2, 1, 128, 128, True)
    torch.cuda.synchronize()
    assert o.shape == (0, 256)


@pytest.mark.parametrize("keep", [0.5, 0.25, 0.125])
def test_attention_llama3_8b_full_sampled(orc, keep):
    """Full size (one sequence of 8192 tokens, 32/8 heads, 8 groups), checked
    on sampled rows: the oracle computes a row at position p from keys 0..p."""
    say("attention full llama3-8b T=8192 keep", keep)
    T, n_q, n_kv, G, hd = 8192, 32, 8, 512, 128
    c = synth.attn_prefill_case(21, 1, T, T, n_q, n_kv, hd, n_q * hd // G, keep=keep)
    q, k, v, m = (to_dev(a) for a in (c.q, c.k, c.v, c.mask))
    o = torch.full_like(q, float("nan"))
    W.wide_attention_masked(q, k, v, m, 1, n_q, n_kv, hd, G, True, o=o)
    torch.cuda.synchronize()
    got = to_np64(o)
    assert np.isfinite(got).all()
    g = synth.rng(5)
    rows = np.unique(np.concatenate([[0, 1, 63, 64, 4095, T - 2, T - 1], g.integers(0, T, 17)]))
    for p in rows:
        sl = slice(p, p + 1)
        args = (c.q[sl], c.k[:p + 1], c.v[:p + 1], c.mask[sl], 1, n_q, n_kv, hd, True)
        ref = orc.attention(*args)
        bound = attention_bound(orc, *args, T_k=p + 1)
        check_rows(got[sl], ref, bound, c.mask[sl], G, f"row {p}")


@pytest.fixture
def attn_split_on():
    yield
    W.wide_set_option("attn_split", 1024)
    W.wide_set_option("attn_split_rounds", 1)


@pytest.mark.parametrize("T_q,T_k,n_q,n_kv,G,mask,keep", [
    (1000, 1000, 8, 2, 512, "topk", 0.5),       # four heads per workgroup, 32-row tiles
    (777, 1200, 32, 8, 512, "bernoulli", 0.3),  # queries after a 423-key prefix, ragged last key tile
    (640, 640, 8, 2, 256, "topk", 0.25),        # two heads per workgroup, 64-row tiles
    (700, 700, 4, 4, 128, "bernoulli", 0.5),    # one head per workgroup, 128-row tiles
    (512, 512, 8, 2, 512, "ones", 1.0),         # every row active
])
def test_attention_key_split_matches_oracle(orc, attn_split_on, T_q, T_k, n_q, n_kv, G, mask, keep):
    """One causal sequence with few query tiles: the key ranges are cut into
    chunks whose partial results a merge kernel combines.  Both the split and
    the unsplit run meet the bound, and the split really ran (its merge
    kernel was launched)."""
    for split, rounds in ((1024, 1), (1024, 8), (0, 1)):
        say("attention key split", split, rounds, T_q, T_k, n_q, n_kv, G, mask, keep)
        W.wide_set_option("attn_split", split)
        W.wide_set_option("attn_split_rounds", rounds)
        W.wide_timing_enable(True)
        W.wide_timing_reset()
        run_case(orc, 1, T_q, T_k, n_q, n_kv, G, True, mask=mask, keep=keep, seed=T_q + split)
        _, n_merge = W.wide_timing_query("wide_attn_merge")
        W.wide_timing_enable(False)
        assert (n_merge > 0) == (split > 0)


def test_attention_key_split_replays_in_hip_graph(attn_split_on):
    say("attention key split graph replay")
    hd, n_q, n_kv, G, T = 128, 8, 2, 512, 900
    cp = synth.attn_prefill_case(8, 1, T, T, n_q, n_kv, hd, n_q * hd // G, mask="topk", keep=0.25)
    q, k, v, m = (to_dev(a) for a in (cp.q, cp.k, cp.v, cp.mask))
    o = torch.empty_like(q)
    ws = torch.empty(W.wide_attention_workspace_size(1, T, T, n_q, n_kv, hd, G, True),
                     dtype=torch.uint8, device=dev())
    step = lambda: W.wide_attention_masked(q, k, v, m, 1, n_q, n_kv, hd, G, True, o=o, ws=ws)
    step()
    torch.cuda.synchronize()
    ref = o.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for _ in range(3):
        o.fill_(7.0)
        ws.fill_(0x5A)   # stale schedule and partials must not matter
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16), ref.view(torch.int16))


def test_attention_key_split_long_keys_sampled(orc):
    """3360 queries after a 56640-key prefix (T_k = 60000, 938 key tiles):
    with 840 active query tiles the work term alone asks for chunks longer
    than any tile's range; the schedule caps the chunk at the key tiles of
    the whole range (no split) and every row is still right.  Sampled rows
    against the oracle."""
    T_q, T_k, n_q, n_kv, G, hd = 3360, 60000, 32, 8, 512, 128
    say("attention long keys", T_q, T_k)
    c = synth.attn_prefill_case(31, 1, T_q, T_k, n_q, n_kv, hd, n_q * hd // G, mask="ones")
    q, k, v, m = (to_dev(a) for a in (c.q, c.k, c.v, c.mask))
    o = torch.full_like(q, float("nan"))
    W.wide_attention_masked(q, k, v, m, 1, n_q, n_kv, hd, G, True, o=o)
    torch.cuda.synchronize()
    got = to_np64(o)
    assert np.isfinite(got).all()
    delta = T_k - T_q
    for p in (0, 1777, T_q - 1):
        sl = slice(p, p + 1)
        args = (c.q[sl], c.k[:delta + p + 1], c.v[:delta + p + 1], c.mask[sl], 1, n_q, n_kv, hd, True)
        ref = orc.attention(*args)
        bound = attention_bound(orc, *args, T_k=delta + p + 1)
        check_rows(got[sl], ref, bound, c.mask[sl], G, f"row {p}")


@pytest.mark.parametrize("n_seq,T_q,T_k,n_q,n_kv,G,causal", [
    (2, 300, 300, 8, 2, 512, True), (3, 70, 133, 8, 2, 256, True), (1, 200, 90, 4, 4, 128, False)])
def test_attention_zero_queries_are_exact_means(orc, n_seq, T_q, T_k, n_q, n_kv, G, causal):
    """q = 0 makes every score 0, so every probability is exactly 1 (no bf16
    rounding of P): each active output is the mean of the visible value rows
    up to fp32 summation, which pins key ranges, causal limits and sequence
    boundaries far more tightly than the general bound."""
    say("attention zero queries", n_seq, T_q, T_k, n_q, n_kv, G, causal)
    hd = 128
    c = synth.attn_prefill_case(7 + T_q, n_seq, T_q, T_k, n_q, n_kv, hd, n_q * hd // G, mask="bernoulli")
    qz = np.zeros_like(c.q)
    q, k, v, m = (to_dev(a) for a in (qz, c.k, c.v, c.mask))
    o = W.wide_attention_masked(q, k, v, m, n_seq, n_q, n_kv, hd, G, causal)
    torch.cuda.synchronize()
    got = to_np64(o)
    ref = orc.attention(qz, c.k, c.v, c.mask, n_seq, n_q, n_kv, hd, causal)
    a_abs = orc.attention(synth.as_f32(qz), synth.as_f32(c.k), np.abs(synth.as_f32(c.v)), c.mask,
                          n_seq, n_q, n_kv, hd, causal)
    check_rows(got, ref, (2.0 ** -16 + T_k * 2.0 ** -24) * a_abs, c.mask, G, "zero queries")


# ------------------------------------------------------------------ decode

def decode_bound(orc, q, k, v, mask, n_q, n_kv, hd):
    """Decode keeps the probabilities in fp32 (no bf16 rounding of P): fp32
    scores (128 bf16 products, error well under 2^-10 relative in p for
    |q|,|k| ~ N(0, 1.5^2)), exponentials, sums and the merge of chunks; plus
    the stored output's bf16 rounding (added by the check)."""
    from paper_2607_28418_amd import synth as s
    vabs = np.abs(s.as_f32(v)).astype(np.float32)
    a_abs = orc.attention(s.as_f32(q), s.as_f32(k), vabs, mask, 1, n_q, n_kv, hd, False)
    return (2.0 ** -10 + k.shape[0] * 2.0 ** -24) * a_abs


def head_major(a, n_kv, hd):
    """[B][L][n_kv*hd] -> [B][n_kv][L][hd] (contiguous)."""
    B, L = a.shape[:2]
    return np.ascontiguousarray(a.reshape(B, L, n_kv, hd).transpose(0, 2, 1, 3))


def run_decode(orc, B, L, n_q, n_kv, G, mask="bernoulli", keep=0.5, qk_std=1.0, ragged=False, seed=0,
               poison_unused=False, hm=False):
    hd = 128
    c = synth.attn_decode_case(seed, B, L, n_q, n_kv, hd, n_q * hd // G, mask=mask, keep=keep,
                               qk_std=qk_std, ragged=ragged)
    k_host, v_host = c.k.copy(), c.v.copy()
    if poison_unused:
        # rows past each kv_len, and the whole cache of KV heads no active head reads
        nan = np.uint16(0x7FC0)
        hpg, qpk = G // hd, n_q // n_kv
        for b in range(B):
            k_host[b, c.kv_len[b]:] = nan
            v_host[b, c.kv_len[b]:] = nan
            for hk in range(n_kv):
                if not any(c.mask[b, (hk * qpk + i) // hpg] for i in range(qpk)):
                    k_host[b, :, hk * hd:(hk + 1) * hd] = nan
                    v_host[b, :, hk * hd:(hk + 1) * hd] = nan
    if hm:
        k_host, v_host = head_major(k_host, n_kv, hd), head_major(v_host, n_kv, hd)
    q, k, v, m = (to_dev(a) for a in (c.q, k_host, v_host, c.mask))
    kl = to_dev(c.kv_len) if ragged else None
    o = torch.full_like(q, float("nan"))
    W.wide_attention_decode(q, k, v, m, n_q, n_kv, hd, G, kv_len=kl, o=o, head_major=hm)
    torch.cuda.synchronize()
    got = to_np64(o)
    for b in range(B):
        n = int(c.kv_len[b])
        args = (c.q[b:b + 1], c.k[b, :n], c.v[b, :n], c.mask[b:b + 1])
        ref = orc.attention(*args, 1, n_q, n_kv, hd, False)
        bound = decode_bound(orc, *args, n_q, n_kv, hd)
        check_rows(got[b:b + 1], ref, bound, c.mask[b:b + 1], G, f"decode b={b} len={n}")
    return c, got


@pytest.mark.parametrize("B,L,n_q,n_kv,G,ragged", [
    (5, 300, 8, 2, 256, False),      # ragged last 64-key step, two heads per group
    (3, 3000, 8, 2, 512, True),      # many chunks, per-sequence lengths
    (4, 200, 4, 4, 128, False),      # one head per KV head
    (6, 500, 8, 4, 256, True),       # two query heads per KV head
    (2, 777, 16, 2, 512, True),      # eight query heads per KV head
    (2, 130, 16, 1, 1024, False),    # 16 query heads on one KV head
    (32, 2048, 32, 8, 512, False),   # Llama-3-8B heads, 32 sequences
])
@pytest.mark.parametrize("hm", [False, True])
def test_attention_decode_matches_oracle(orc, B, L, n_q, n_kv, G, ragged, hm):
    say("attention decode", B, L, n_q, n_kv, G, ragged, "head-major" if hm else "token-major")
    run_decode(orc, B, L, n_q, n_kv, G, ragged=ragged, qk_std=1.5, seed=B + L, hm=hm)


@pytest.mark.parametrize("kind", ["zeros", "ones"])
def test_attention_decode_degenerate_masks(orc, kind):
    say("attention decode mask", kind)
    run_decode(orc, 6, 500, 8, 2, 512, mask=kind)


@pytest.mark.parametrize("hm", [False, True])
def test_attention_decode_never_reads_unused_cache(orc, hm):
    say("attention decode poisoned cache", hm)
    run_decode(orc, 8, 700, 8, 2, 512, ragged=True, poison_unused=True, seed=4, hm=hm)


def test_attention_decode_empty():
    say("attention decode empty")
    o = W.wide_attention_decode(torch.zeros((0, 256), dtype=torch.bfloat16, device=dev()),
                                torch.zeros((0, 64, 128), dtype=torch.bfloat16, device=dev()),
                                torch.zeros((0, 64, 128), dtype=torch.bfloat16, device=dev()),
                                torch.zeros((0, 2), dtype=torch.uint8, device=dev()), 2, 1, 128, 128)
    torch.cuda.synchronize()
    assert o.shape == (0, 256)


def test_attention_decode_timing_labels_are_distinct():
    say("attention decode timing labels")
    c = synth.attn_decode_case(2, 4, 256, 8, 2, 128, 2)
    q, k, v, m = (to_dev(a) for a in (c.q, c.k, c.v, c.mask))
    W.wide_timing_enable(True)
    W.wide_timing_reset()
    W.wide_attention_decode(q, k, v, m, 8, 2, 128, 512)
    n_dec, n_merge = W.wide_timing_query("wide_attn_decode")[1], W.wide_timing_query("wide_attn_decode_merge")[1]
    W.wide_timing_enable(False)
    assert n_dec == 1 and n_merge == 1


def test_attention_calls_replay_in_hip_graph():
    """Prefill and decode attention captured in one HIP graph: every replay
    (with eager work and syncs in between) equals the eager result bitwise."""
    say("attention graph replay")
    hd, n_q, n_kv, G = 128, 8, 2, 512
    cp = synth.attn_prefill_case(3, 2, 150, 150, n_q, n_kv, hd, n_q * hd // G, mask="topk")
    q, k, v, m = (to_dev(a) for a in (cp.q, cp.k, cp.v, cp.mask))
    cd = synth.attn_decode_case(4, 6, 300, n_q, n_kv, hd, n_q * hd // G, ragged=True)
    dq, dk, dv, dm, dl = (to_dev(a) for a in (cd.q, cd.k, cd.v, cd.mask, cd.kv_len))
    o = torch.empty_like(q)
    do = torch.empty_like(dq)
    ws = torch.empty(W.wide_attention_workspace_size(2, 150, 150, n_q, n_kv, hd, G, True),
                     dtype=torch.uint8, device=dev())
    dws = torch.empty(W.wide_attention_decode_workspace_size(6, 300, n_q, n_kv, hd, G),
                      dtype=torch.uint8, device=dev())

    def step():
        W.wide_attention_masked(q, k, v, m, 2, n_q, n_kv, hd, G, True, o=o, ws=ws)
        W.wide_attention_decode(dq, dk, dv, dm, n_q, n_kv, hd, G, kv_len=dl, o=do, ws=dws)

    step()
    torch.cuda.synchronize()
    ref = [o.clone(), do.clone()]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for _ in range(3):
        o.fill_(7.0)
        do.fill_(7.0)
        ws.fill_(0x5A)   # stale workspace contents must not matter
        dws.fill_(0x5A)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16), ref[0].view(torch.int16))
        assert torch.equal(do.view(torch.int16), ref[1].view(torch.int16))
