"""The prefill attention key-range split sizes its chunk length so that the
units it lists fit the workspace: at most kAttnMaxChunks chunks per query
tile, at most kAttnMaxUnits units in all, and a chunk length within the
schedule's size histogram.  This restates the rule (the chunk length is the
largest of ceil(nkt / 8), ceil(W / (rounds * 512)) and
ceil(W / (2048 - tiles)), W the key tiles of all active query tiles, but
at most nkt) and
checks those bounds over random and extreme tile sets (no GPU)."""
import re
from pathlib import Path

import numpy as np

HDR = Path(__file__).resolve().parents[1] / "paper_2607_28418_amd" / "csrc" / "kernels.h"


def _const(name):
    text = HDR.read_text()
    m = re.search(r"constexpr int %s = ([^;]+);" % name, text)
    expr = m.group(1)
    for k in re.findall(r"kAttn\w+", expr):
        expr = expr.replace(k, str(_const(k)))
    return int(eval(expr))


MAX_CHUNKS, MAX_UNITS = _const("kAttnMaxChunks"), _const("kAttnMaxUnits")
MAX_TILES, SLOTS, MAX_CH = _const("kAttnMaxSplitTiles"), _const("kAttnSlots"), _const("kAttnMaxChunkTiles")


def chunk_len(nt, nkt, rounds):
    work, total = int(nt.sum()), len(nt)
    per_round = rounds * SLOTS
    ch = -(-nkt // MAX_CHUNKS)
    ch = max(ch, -(-work // per_round))
    ch = max(ch, -(-work // (MAX_UNITS - total)))
    return min(ch, nkt)


def test_constants_leave_room_for_the_chunks():
    assert MAX_TILES * 2 <= MAX_UNITS and MAX_CH >= 1 and MAX_CHUNKS <= 8


def test_schedule_bounds_hold():
    g = np.random.default_rng(0)
    cases = []
    for _ in range(3000):
        nkt = int(g.integers(8, MAX_CH + 1))   # key tiles of 64 (the split needs 8..1024)
        total = int(g.integers(1, MAX_TILES + 1))
        kind = g.integers(0, 3)
        if kind == 0:
            nt = g.integers(1, nkt + 1, total)
        elif kind == 1:                        # every tile spans all keys
            nt = np.full(total, nkt)
        else:                                  # causal ramp
            nt = np.maximum(1, (np.arange(1, total + 1) * nkt) // total)
        cases.append((nt, nkt, int(g.integers(1, 9))))
    cases.append((np.full(MAX_TILES, MAX_CH), MAX_CH, 1))
    cases.append((np.ones(1, dtype=np.int64), 8, 8))
    for nt, nkt, rounds in cases:
        ch = chunk_len(nt, nkt, rounds)
        nc = -(-nt // ch)
        assert 1 <= ch <= MAX_CH
        assert nc.max() <= MAX_CHUNKS
        assert int(nc.sum()) <= MAX_UNITS
        assert (np.minimum(ch, nt - (nc - 1) * ch) >= 1).all()  # every chunk has a key tile
