"""CPU-only checks of the C ABI: every declared symbol is exported, and the
host-side validation rejects bad arguments before touching the device (no
compute call is made here; the fake pointers below are never dereferenced)."""
import ctypes
import os
import re

import pytest

import paper_2607_28418_amd as W

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "wide.h")

A = ctypes.c_void_p(0x10000)      # aligned, never dereferenced
MIS = ctypes.c_void_p(0x10008)    # 8-byte aligned only


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wide_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert {"wide_mask_reorder", "wide_ffn_masked", "wide_qkvo_masked",
            "wide_workspace_size", "wide_last_error"} <= set(names)
    lib = ctypes.CDLL(W.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def ffn(dt=W.BF16, M=128, D=4096, Dff=11008, G=128, mask=A, idx=None, cnt=None, x=A, wg=A, wu=A,
        wd=A, h=None, y=A, ws=A, ws_bytes=1 << 40):
    return W.lib().wide_ffn_masked(dt, M, D, Dff, G, mask, idx, cnt, x, wg, wu, wd, h, y, ws,
                                   ws_bytes, None)


def err():
    return W.lib().wide_last_error().decode()


@pytest.mark.parametrize("kw,status,msg", [
    (dict(G=48), W.ERR_INVALID_ARG, "power of two"),
    (dict(G=8), W.ERR_INVALID_ARG, "power of two"),
    (dict(Dff=11000), W.ERR_INVALID_ARG, "does not divide"),
    (dict(G=32, Dff=1056), W.ERR_UNSUPPORTED, "group_size < 64"),
    (dict(mask=MIS), W.ERR_INVALID_ARG, "mask is not 16-byte aligned"),
    (dict(D=4000), W.ERR_UNSUPPORTED, "256"),
    (dict(M=-1), W.ERR_INVALID_ARG, "out of range"),
    (dict(dt=7), W.ERR_INVALID_ARG, "dtype"),
    (dict(x=None), W.ERR_INVALID_ARG, "x is NULL"),
    (dict(wd=MIS), W.ERR_INVALID_ARG, "aligned"),
    (dict(idx=A), W.ERR_INVALID_ARG, "both"),
    (dict(ws=None), W.ERR_WORKSPACE, "NULL"),
    (dict(ws_bytes=1000), W.ERR_WORKSPACE, "needed"),
    (dict(ws=ctypes.c_void_p(0x10010)), W.ERR_INVALID_ARG, "256-byte"),
])
def test_ffn_validation(kw, status, msg):
    assert ffn(**kw) == status
    assert msg in err()


def test_m_zero_is_ok_without_touching_anything():
    assert ffn(M=0, x=None, y=None, mask=None, ws=None) == W.OK


def test_qkvo_validation():
    L = W.lib()
    def call(phase=W.PHASE_QKV, dt=W.BF16, M=16, D=4096, nq=32, nkv=8, hd=128, G=512, **p):
        args = dict(mask=A, idx=None, cnt=None, inp=A, wq=A, wk=A, wv=A, wo=A, q=A, k=A, v=A, y=A,
                    ws=A, wsb=1 << 40)
        args.update(p)
        return L.wide_qkvo_masked(phase, dt, M, D, nq, nkv, hd, G, args["mask"], args["idx"],
                                  args["cnt"], args["inp"], args["wq"], args["wk"], args["wv"],
                                  args["wo"], args["q"], args["k"], args["v"], args["y"],
                                  args["ws"], args["wsb"], None)
    assert call(nq=30, nkv=8) == W.ERR_INVALID_ARG and "multiple of n_kv" in err()
    assert call(G=500) == W.ERR_INVALID_ARG and "head_dim" in err()
    assert call(G=384) == W.ERR_INVALID_ARG and "divide" in err()
    assert call(phase=5) == W.ERR_INVALID_ARG
    assert call(wq=None) == W.ERR_INVALID_ARG and "w_q" in err()
    assert call(phase=W.PHASE_O, wo=None) == W.ERR_INVALID_ARG and "w_o" in err()
    assert call(hd=64, G=64, nkv=2) == W.ERR_UNSUPPORTED and "group_size 64" in err()
    assert call(mask=MIS) == W.ERR_INVALID_ARG and "mask is not 16-byte aligned" in err()
    assert call(phase=W.PHASE_O, mask=MIS) == W.ERR_INVALID_ARG
    assert call(M=0, inp=None, mask=None, q=None, k=None, v=None) == W.OK


def test_workspace_sizes():
    s = W.wide_workspace_size
    assert s(W.OP_FFN, W.BF16, 4096, 4096, 11008, 48) == W.SIZE_MAX
    # groups of 16 and 32 (Section 3.1: {2^k, k >= 4}): a merged mask instead of a reorder
    for G in (16, 32):
        small = s(W.OP_FFN, W.BF16, 8192, 4096, 14336, G)
        assert small != W.SIZE_MAX and small >= 8192 * 14336 * 2 + 8192 * (14336 // 64)
        assert s(W.OP_FFN, W.BF16, 16, 4096, 14336, G) != W.SIZE_MAX
    assert s(W.OP_FFN, W.BF16, 8192, 4096, 1056, 32) == W.SIZE_MAX
    pre = s(W.OP_FFN, W.BF16, 4096, 4096, 11008, 128)
    # H (bf16) + fp32 K-axis buffer + reorder index at least
    assert pre >= 4096 * 11008 * 2 + 4096 * 4096 * 4 + 86 * 4096 * 4
    dec = s(W.OP_FFN, W.BF16, 16, 4096, 11008, 128)
    assert 16 * 11008 * 2 <= dec < pre
    assert s(W.OP_REORDER, W.BF16, 8192, 0, 112, 1) >= 2 * 32 * 112 * 4
    # decode QKV: fp32 partial sums of the k split, bounded without n_kv
    assert 0 < s(W.OP_QKV, W.BF16, 16, 4096, 4096, 512) <= 8 * 16 * 3 * 4096 * 4 + 256
    assert s(W.OP_O, W.BF16, 8192, 4096, 4096, 512) >= 8192 * 4096 * 4
    assert s(W.OP_FFN, W.F32, 128, 512, 1536, 64) >= 128 * 1536 * 4


def test_options():
    W.wide_set_option("decode_max_m", 8)
    assert W.wide_get_option("decode_max_m") == 8
    W.wide_set_option("decode_max_m", 64)
    with pytest.raises(W.WideError):
        W.wide_set_option("k_path", 9)
    for gone in ("nope", "ring_bk", "attn_qb"):  # (the measured-slower variants are not built)
        with pytest.raises(W.WideError):
            W.wide_set_option(gone, 1)
    for key, default, bad in (("mn_order", 7, 8), ("kd_pattern", 1, 2), ("mn_tail", 1, 2),
                               ("attn_split", 1024, 1025), ("attn_split_rounds", 1, 9), ("ks_pack", 1, 0),
                               ("gemv_n_ncb", 0, 3), ("gemv_k_split", 0, 16)):
        assert W.wide_get_option(key) == default
        W.wide_set_option(key, {"attn_split_rounds": 3, "ks_pack": 4, "gemv_n_ncb": 8, "gemv_k_split": 8}.get(key, 0))
        with pytest.raises(W.WideError):
            W.wide_set_option(key, bad)
        W.wide_set_option(key, default)
        assert W.wide_get_option(key) == default


def router(dt=W.BF16, M=64, D=4096, r=32, ng=112, x=A, w1=A, w2=A, mask=A, logits=None, idx=None,
           cnt=None, ws=A, ws_bytes=1 << 40):
    return W.lib().wide_router(dt, M, D, r, ng, x, w1, w2, mask, logits, idx, cnt, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(dt=W.F32), W.ERR_UNSUPPORTED, "bf16"),
    (dict(D=4000), W.ERR_INVALID_ARG, "multiple of 64"),
    (dict(r=0), W.ERR_INVALID_ARG, "rank"),
    (dict(r=33), W.ERR_INVALID_ARG, "rank"),
    (dict(ng=0), W.ERR_INVALID_ARG, "n_groups"),
    (dict(ng=4097), W.ERR_INVALID_ARG, "n_groups"),
    (dict(idx=A), W.ERR_INVALID_ARG, "both"),
    (dict(x=MIS), W.ERR_INVALID_ARG, "x is not 16-byte aligned"),
    (dict(w1=None), W.ERR_INVALID_ARG, "w1 is NULL"),
    (dict(mask=None), W.ERR_INVALID_ARG, "mask is NULL"),
    (dict(idx=A, cnt=A, ws_bytes=0), W.ERR_WORKSPACE, "workspace"),
    (dict(M=-1), W.ERR_INVALID_ARG, "M"),
])
def test_router_validation(kw, status, msg):
    assert router(**kw) == status
    assert msg in err()


def test_router_m_zero_without_reorder_is_ok():
    assert router(M=0, x=None, mask=None) == W.OK


def test_router_workspace_size():
    assert W.wide_workspace_size(W.OP_ROUTER, W.BF16, 8192, 4096, 112, 32) > 0
    assert W.wide_workspace_size(W.OP_ROUTER, W.F32, 8192, 4096, 112, 32) == W.SIZE_MAX
    assert W.wide_workspace_size(W.OP_ROUTER, W.BF16, 8192, 4000, 112, 32) == W.SIZE_MAX
    assert W.wide_workspace_size(W.OP_ROUTER, W.BF16, 8192, 4096, 112, 33) == W.SIZE_MAX


def attention(dt=W.BF16, n_seq=1, T_q=256, T_k=256, nq=32, nkv=8, hd=128, G=512, causal=1, mask=A, idx=None,
              cnt=None, q=A, k=A, v=A, o=A, ws=A, ws_bytes=1 << 40):
    return W.lib().wide_attention_masked(dt, n_seq, T_q, T_k, nq, nkv, hd, G, causal, None, mask, idx, cnt, q, k, v,
                                         o, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(dt=W.F32), W.ERR_UNSUPPORTED, "bf16"),
    (dict(dt=7), W.ERR_INVALID_ARG, "dtype"),
    (dict(hd=64, G=256), W.ERR_UNSUPPORTED, "head_dim 128"),
    (dict(nq=30), W.ERR_INVALID_ARG, "multiple of n_kv_heads"),
    (dict(G=192), W.ERR_INVALID_ARG, "multiple of head_dim"),
    (dict(G=128 * 3), W.ERR_INVALID_ARG, "does not divide"),
    (dict(T_k=100), W.ERR_INVALID_ARG, "T_k >= T_q"),
    (dict(T_k=0, causal=0), W.ERR_INVALID_ARG, "no keys"),
    (dict(causal=2), W.ERR_INVALID_ARG, "causal"),
    (dict(n_seq=-1), W.ERR_INVALID_ARG, ">= 0"),
    (dict(n_seq=1 << 20, T_q=1 << 12), W.ERR_INVALID_ARG, "2^31"),
    (dict(idx=A), W.ERR_INVALID_ARG, "both"),
    (dict(q=MIS), W.ERR_INVALID_ARG, "q is not 16-byte aligned"),
    (dict(v=None), W.ERR_INVALID_ARG, "v is NULL"),
    (dict(mask=None), W.ERR_INVALID_ARG, "mask is NULL"),
    (dict(ws_bytes=0), W.ERR_WORKSPACE, "workspace"),
    (dict(ws=None), W.ERR_WORKSPACE, "workspace"),
])
def test_attention_validation(kw, status, msg):
    assert attention(**kw) == status
    assert msg in err()


def test_attention_empty_is_ok_and_non_causal_allows_short_keys():
    assert attention(n_seq=0, mask=None, q=None, k=None, v=None, o=None, ws=None, ws_bytes=0) == W.OK
    assert attention(T_q=0, T_k=0, mask=None, q=None, k=None, v=None, o=None, ws=None, ws_bytes=0) == W.OK


def test_attention_workspace_size():
    n = W.wide_attention_workspace_size(1, 8192, 8192, 32, 8, 128, 512, True)
    n0 = W.wide_attention_workspace_size(1, 8192, 8192, 32, 8, 128, 512, False)
    # the transposed V (8 KV heads x 128 x 8192 bf16) is always there; the reorder only on request
    assert n0 >= 8 * 128 * 8192 * 2 and n > n0 + 8 * 8192 * 4
    assert W.wide_attention_workspace_size(2, 100, 130, 8, 2, 128, 256, False) >= 2 * 2 * 128 * 192 * 2
    assert W.wide_attention_workspace_size(1, 0, 0, 32, 8, 128, 512, True) == 0
    assert W.wide_attention_workspace_size(1, 64, 64, 32, 8, 64, 512, True) == W.SIZE_MAX


def attention_decode(dt=W.BF16, B=32, L=8192, nq=32, nkv=8, hd=128, G=512, mask=A, kv_len=None, layout=0, q=A,
                     k=A, v=A, o=A, ws=A, ws_bytes=1 << 40):
    return W.lib().wide_attention_decode(dt, B, L, nq, nkv, hd, G, mask, kv_len, layout, q, k, v, o, ws, ws_bytes,
                                         None)


@pytest.mark.parametrize("kw,status,msg", [
    (dict(dt=W.F32), W.ERR_UNSUPPORTED, "bf16"),
    (dict(hd=64, G=256), W.ERR_UNSUPPORTED, "head_dim 128"),
    (dict(nq=34, nkv=2, G=128), W.ERR_UNSUPPORTED, "16 query heads"),
    (dict(nq=30), W.ERR_INVALID_ARG, "multiple of n_kv_heads"),
    (dict(G=192), W.ERR_INVALID_ARG, "multiple of head_dim"),
    (dict(L=0), W.ERR_INVALID_ARG, "length 0"),
    (dict(B=-1), W.ERR_INVALID_ARG, ">= 0"),
    (dict(B=1 << 20, L=1 << 12), W.ERR_INVALID_ARG, "2^31"),
    (dict(k=MIS), W.ERR_INVALID_ARG, "k_cache is not 16-byte aligned"),
    (dict(o=None), W.ERR_INVALID_ARG, "o is NULL"),
    (dict(mask=None), W.ERR_INVALID_ARG, "mask is NULL"),
    (dict(ws_bytes=0), W.ERR_WORKSPACE, "workspace"),
    (dict(layout=2), W.ERR_INVALID_ARG, "kv_layout"),
])
def test_attention_decode_validation(kw, status, msg):
    assert attention_decode(**kw) == status
    assert msg in err()


def test_attention_decode_empty_and_workspace():
    assert attention_decode(B=0, mask=None, q=None, k=None, v=None, o=None, ws=None, ws_bytes=0) == W.OK
    n = W.wide_attention_decode_workspace_size(32, 8192, 32, 8, 128, 512)
    assert n >= 32 * 32 * 130 * 4   # at least one chunk of (max, sum, o[128]) per (token, head)
    assert W.wide_attention_decode_workspace_size(0, 8192, 32, 8, 128, 512) == 0
    assert W.wide_attention_decode_workspace_size(32, 8192, 32, 8, 64, 512) == W.SIZE_MAX


def test_single_group_is_accepted():
    # group_size = d_ff (one group, the M-axis case) need not be a power of two
    # (a valid call would launch; stop it at the workspace check instead)
    assert ffn(Dff=14336, G=14336, ws_bytes=0) == W.ERR_WORKSPACE
    assert ffn(Dff=14336, G=7168) == W.ERR_INVALID_ARG and "power of two" in err()
    assert ffn(Dff=1000, G=1000, D=256) == W.ERR_UNSUPPORTED and "128" in err()
    assert W.wide_workspace_size(W.OP_FFN, W.BF16, 8192, 4096, 14336, 14336) != W.SIZE_MAX


def test_attention_workspace_holds_the_key_split_only_where_it_can_run():
    """The key-range split's schedule and partials are carved only for one
    causal-capable sequence with enough key tiles; switching the option off
    shrinks the workspace back."""
    T, n_q, n_kv, hd, G = 8192, 32, 8, 128, 512
    with_split = W.wide_attention_workspace_size(1, T, T, n_q, n_kv, hd, G, False)
    two_seq = W.wide_attention_workspace_size(2, T, T, n_q, n_kv, hd, G, False)
    W.wide_set_option("attn_split", 0)
    try:
        without = W.wide_attention_workspace_size(1, T, T, n_q, n_kv, hd, G, False)
    finally:
        W.wide_set_option("attn_split", 1024)
    # 2048 units x (16384 + 512) floats of partials, plus the schedule's ints
    assert with_split - without >= 2048 * (16384 + 512) * 4
    assert with_split - without < 2048 * (16384 + 512) * 4 + 64 * 1024
    assert two_seq < 2 * with_split  # no split for two sequences: only V^T grows
    short = W.wide_attention_workspace_size(1, 256, 256, n_q, n_kv, hd, G, False)
    W.wide_set_option("attn_split", 0)
    try:
        assert W.wide_attention_workspace_size(1, 256, 256, n_q, n_kv, hd, G, False) == short
    finally:
        W.wide_set_option("attn_split", 1024)


def test_noalloc_refuses_sizes_beyond_its_scratch_before_any_device_call():
    """The allocation-free FFN checks its scratch need on the host first: a
    prefill whose H would have to sit in the 32 MiB array is refused."""
    L = W.lib()
    assert L.wide_static_scratch_bytes() == 32 << 20
    st = L.wide_ffn_masked_noalloc(W.BF16, 8192, 4096, 14336, 128, A, None, None, A, A, A, A, None, A, None)
    assert st == W.ERR_WORKSPACE and "static scratch" in err()
    st = L.wide_ffn_masked_noalloc(W.BF16, 8, 4096, 14336, 48, A, None, None, A, A, A, A, None, A, None)
    assert st == W.ERR_INVALID_ARG and "power of two" in err()
