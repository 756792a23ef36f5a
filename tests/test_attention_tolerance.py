"""The attention parity bound rejects plausible kernel mistakes (CPU only).

Each mistake is planted in a reference computed by the oracle (never in a
kernel): an off-by-one causal limit, a key left out of a row, grouped-query
heads reading the wrong KV head, and P rounded to bf16 twice.  The bound of
tests/_helpers must reject the first three at the sizes the GPU tests use
and accept the last, which stays inside the rounding the bound allows for.
"""
import numpy as np

from paper_2607_28418_amd import synth
from tests._helpers import attention_bound, check_attention_rows


def _rejects(got, ref, bound, mask, G):
    try:
        check_attention_rows(got, ref, bound, mask, G, "planted")
    except AssertionError:
        return True
    return False


def _case(seed=3, T=200, n_q=8, n_kv=2, G=256):
    c = synth.attn_prefill_case(seed, 1, T, T, n_q, n_kv, 128, n_q * 128 // G, keep=0.5)
    return c, G


def test_bound_accepts_the_oracle_itself(orc):
    c, G = _case()
    ref = orc.attention(c.q, c.k, c.v, c.mask, 1, 8, 2, 128, True)
    got = orc.attention(c.q, c.k, c.v, c.mask, 1, 8, 2, 128, True, round_bf16=True)
    bound = attention_bound(orc, c.q, c.k, c.v, c.mask, 1, 8, 2, 128, True, c.T_k)
    assert not _rejects(got, ref, bound, c.mask, G)


def test_bound_rejects_an_off_by_one_causal_limit(orc):
    c, G = _case()
    ref = orc.attention(c.q, c.k, c.v, c.mask, 1, 8, 2, 128, True)
    # every query also sees the next key: one extra key row and T_k = T + 1
    # put the causal limit of query p at key p + 1
    k1 = np.concatenate([c.k, c.k[-1:]])
    v1 = np.concatenate([c.v, c.v[-1:]])
    wrong = orc.attention(c.q, k1, v1, c.mask, 1, 8, 2, 128, True, round_bf16=True)
    bound = attention_bound(orc, c.q, c.k, c.v, c.mask, 1, 8, 2, 128, True, c.T_k)
    assert _rejects(wrong, ref, bound, c.mask, G)


def test_bound_rejects_a_dropped_key(orc):
    c, G = _case()
    ref = orc.attention(c.q, c.k, c.v, c.mask, 1, 8, 2, 128, True)
    wrong = orc.attention(c.q, c.k, c.v, c.mask, 1, 8, 2, 128, True, round_bf16=True)
    # rows that see key 70 recomputed without it (numerator and denominator):
    # one query against the other visible keys, all of which it sees
    drop = 70
    for p in range(drop, c.T_q):
        keep = np.r_[0:drop, drop + 1:p + 1]
        if keep.size == 0:
            continue
        wrong[p] = orc.attention(c.q[p:p + 1], c.k[keep], c.v[keep], c.mask[p:p + 1], 1, 8, 2, 128, True,
                                 round_bf16=True)[0]
    bound = attention_bound(orc, c.q, c.k, c.v, c.mask, 1, 8, 2, 128, True, c.T_k)
    assert _rejects(wrong, ref, bound, c.mask, G)


def test_bound_rejects_the_wrong_kv_head(orc):
    c, G = _case()
    ref = orc.attention(c.q, c.k, c.v, c.mask, 1, 8, 2, 128, True)
    # the two KV heads swapped (a head-to-KV-head map mistake)
    ks = np.ascontiguousarray(c.k.reshape(-1, 2, 128)[:, ::-1].reshape(-1, 256))
    vs = np.ascontiguousarray(c.v.reshape(-1, 2, 128)[:, ::-1].reshape(-1, 256))
    wrong = orc.attention(c.q, ks, vs, c.mask, 1, 8, 2, 128, True, round_bf16=True)
    bound = attention_bound(orc, c.q, c.k, c.v, c.mask, 1, 8, 2, 128, True, c.T_k)
    assert _rejects(wrong, ref, bound, c.mask, G)
