"""The speedup bound 1/(1-s) is a FLOP identity (CPU only).

For every prunable projection (Q, O, gate/up, down) the executed FLOPs are
those of the active (token, group) pairs, so active / dense FLOPs equals the
mask's mean, 1 - s; for a top-k mask that is exactly k / n_groups.  The
benchmark's FLOP accounting (bench.Layer) must reproduce that, and its ideal
speedup of the whole layer (K and V stay dense, Section 3.1) must follow.
"""
import numpy as np
import pytest

from bench import Layer
from paper_2607_28418_amd import synth


@pytest.mark.parametrize("keep", [0.25, 0.5, 0.75])
def test_topk_masks_keep_exactly_k_groups(keep):
    g = synth.rng(3)
    x = synth.normal(g, (500, 64), 1.0, "bf16")
    for ng in (8, 86, 112):
        k = synth.keep_count(ng, keep)
        m = synth.mask_topk(synth.router_logits(g, x, ng), k)
        assert (m.sum(1) == k).all()
        assert m.mean() == k / ng


@pytest.mark.parametrize("keep", [0.25, 0.5, 0.75])
def test_bench_flops_give_the_ideal_speedup(keep):
    L = Layer(7, 512, 32, keep, weights=False)
    for name in ("prefill", "decode"):
        act, dense = L.active_flops(name), L.dense_flops_per_op(name)
        ma, mf = L.batches[name]["mask_attn"], L.batches[name]["mask_ffn"]
        for op, m in (("q", ma), ("o", ma), ("gate_up", mf), ("down", mf)):
            s = 1.0 - m.mean()
            assert act[op] / dense[op] == pytest.approx(1.0 - s, rel=1e-12)
            assert dense[op] / act[op] == pytest.approx(1.0 / (1.0 - s), rel=1e-12)
        assert act["kv"] == dense["kv"]               # K and V are never pruned
        assert sum(dense.values()) == pytest.approx(L.dense_flops(name), rel=1e-12)
        # whole layer: dense / active with K, V dense
        ka, kf = synth.keep_count(L.nga, keep) / L.nga, synth.keep_count(L.ng, keep) / L.ng
        D = L.D
        expect = (2 * L.Nq + 2 * L.Nkv + 3 * L.Dff) / (2 * L.Nq * ka + 2 * L.Nkv + 3 * L.Dff * kf)
        assert L.dense_flops(name) / act["total"] == pytest.approx(expect, rel=1e-12)
        del D


def test_bernoulli_mask_flops():
    g = synth.rng(9)
    m = synth.mask_bernoulli(g, 4000, 24, 0.5)
    G, D = 64, 512
    active = sum(2.0 * D * G * int(m[t].sum()) for t in range(m.shape[0]))
    dense = 2.0 * D * G * m.size
    assert active / dense == pytest.approx(m.mean(), rel=1e-12)
    assert abs(m.mean() - 0.5) < 0.01
