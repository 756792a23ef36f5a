"""The allocation-free FFN entry point against the one with a workspace.

wide_ffn_masked_noalloc runs the same kernels as wide_ffn_masked with its
scratch in the library's static per-GPU array.  Two calls in a row (the
second smaller, so it reuses scratch the first one left behind) must give
outputs bitwise equal to wide_ffn_masked's (the dense-masked K axis has no
atomics), which meet the oracle bar; a call needing more scratch than the
array holds is refused before anything runs; and the call replays from a
HIP graph.
"""
import sys

import numpy as np
import pytest
import torch

import paper_2607_28418_amd as W
from paper_2607_28418_amd import synth
from tests._helpers import check_ffn, dev, to_dev

pytestmark = pytest.mark.gpu


def say(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


@pytest.fixture(autouse=True)
def _options():
    W.lib()
    W.wide_set_option("k_path", 1)
    yield
    W.wide_set_option("k_path", 0)


def _dev(c):
    return [to_dev(a) for a in (c.x, c.w_gate, c.w_up, c.w_down, c.mask)]


@pytest.mark.parametrize("sizes,G,with_h", [
    ((1000, 300), 128, False),    # prefill (reorder, H and K-axis scratch in the array), then smaller
    ((1000, 300), 128, True),
    ((48, 5), 128, False),        # decode, then a smaller batch
    ((700, 33), 32, False),       # narrow groups: merged mask in the array; then decode
    ((2048, 1024), 64, True),
])
def test_noalloc_matches_workspace_entry_point(orc, sizes, G, with_h):
    D, Dff = 512, 2048
    for M in sizes:
        say("noalloc", M, G, with_h)
        c = synth.ffn_case(M + G, M, D, Dff, G, mask="topk")
        x, wg, wu, wd, m = _dev(c)
        h_ref = torch.empty((M, Dff), dtype=torch.bfloat16, device=dev()) if with_h else None
        h_got = torch.full((M, Dff), 5.0, dtype=torch.bfloat16, device=dev()) if with_h else None
        y_ref = W.wide_ffn_masked(x, wg, wu, wd, m, G, h_out=h_ref)
        y_got = torch.full((M, D), 5.0, dtype=torch.bfloat16, device=dev())
        W.wide_ffn_masked_noalloc(x, wg, wu, wd, m, G, h_out=h_got, y=y_got)
        torch.cuda.synchronize()
        assert torch.equal(y_got.view(torch.int16), y_ref.view(torch.int16)), f"M={M}: y differs"
        if with_h:
            assert torch.equal(h_got.view(torch.int16), h_ref.view(torch.int16)), f"M={M}: h differs"
        check_ffn(orc, c, y_got, h_got, rows=np.unique(np.r_[0, M - 1, np.arange(0, M, max(1, M // 16))]),
                  what=f"noalloc M={M}")


def test_noalloc_refuses_more_than_its_scratch():
    say("noalloc too big")
    cap = W.wide_static_scratch_bytes()
    M, D, Dff, G = 8192, 256, 4096, 128          # H alone: 64 MiB > the scratch
    assert M * Dff * 2 > cap
    x = torch.zeros((M, D), dtype=torch.bfloat16, device=dev())
    w = torch.zeros((Dff, D), dtype=torch.bfloat16, device=dev())
    wd = torch.zeros((D, Dff), dtype=torch.bfloat16, device=dev())
    m = torch.ones((M, Dff // G), dtype=torch.uint8, device=dev())
    y = torch.full((M, D), 3.0, dtype=torch.bfloat16, device=dev())
    with pytest.raises(W.WideError) as ei:
        W.wide_ffn_masked_noalloc(x, w, w, wd, m, G, y=y)
    assert ei.value.status == W.ERR_WORKSPACE and "static scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert (y.float() == 3.0).all()
    # with H given by the caller the same call fits
    h = torch.empty((M, Dff), dtype=torch.bfloat16, device=dev())
    W.wide_ffn_masked_noalloc(x, w, w, wd, m, G, h_out=h, y=y)
    torch.cuda.synchronize()
    assert not y.float().any()


def test_noalloc_replays_in_hip_graph(orc):
    say("noalloc graph")
    M, D, Dff, G = 600, 512, 1024, 128
    c = synth.ffn_case(9, M, D, Dff, G, mask="topk")
    x, wg, wu, wd, m = _dev(c)
    y = torch.empty((M, D), dtype=torch.bfloat16, device=dev())
    W.wide_ffn_masked_noalloc(x, wg, wu, wd, m, G, y=y)      # first call on the device: outside capture
    torch.cuda.synchronize()
    ref = y.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        W.wide_ffn_masked_noalloc(x, wg, wu, wd, m, G, y=y)
    for _ in range(3):
        y.fill_(7.0)
        W.wide_ffn_masked_noalloc(x[:40].contiguous(), wg, wu, wd, m[:40].contiguous(), G)  # eager use in between
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), ref.view(torch.int16))
    check_ffn(orc, c, y, what="graph replay")
