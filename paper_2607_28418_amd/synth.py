"""Seeded synthetic inputs shared by the tests, the smoke check and the bench.

This module holds no arithmetic of the masked projections: it only draws
activations, weights and routing masks with the shapes and distributions of
WIDE's workloads (Llama-style FFN and attention projections at 25/50/75%
sparsity) and quantises them once to bf16.  Both the HIP path and the oracle
receive the same bytes from here.

Draw order per case is fixed: x, then the weights in argument order, then the
extra attention operand (if any), then the router/probability draws, then the
mask.  The generator is numpy's PCG64 seeded with the case seed.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


# ---- bf16 quantisation of inputs (round to nearest even from fp32) --------

def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 array -> bf16 bit patterns (uint16), round to nearest even.
    Inputs are finite draws; NaN/Inf are not expected here."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal(g: np.random.Generator, shape, std: float, dtype: str) -> np.ndarray:
    """N(0, std^2) draw as float32 (dtype 'f32') or bf16 bits (dtype 'bf16')."""
    a = g.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return a if dtype == "f32" else f32_to_bf16_bits(a)


def as_f32(a: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(a) if a.dtype == np.uint16 else a


# ---- routing masks ---------------------------------------------------------

def keep_count(n_groups: int, keep: float) -> int:
    """Groups kept per token for a keep fraction, rounded half up."""
    return int(np.floor(n_groups * keep + 0.5))


def mask_bernoulli(g, M: int, n_groups: int, p: float) -> np.ndarray:
    return (g.random((M, n_groups)) < p).astype(np.uint8)


def mask_beta_groups(g, M: int, n_groups: int, mean: float = 0.5) -> np.ndarray:
    """Per-group activation probability p_g ~ Beta(2,2), rescaled so that the
    mean over groups is `mean` (clipped to [0,1]); mask[t,g] ~ Bernoulli(p_g)."""
    p = g.beta(2.0, 2.0, size=n_groups)
    p = np.clip(p * (mean / p.mean()), 0.0, 1.0)
    return (g.random((M, n_groups)) < p[None, :]).astype(np.uint8)


def mask_topk(logits: np.ndarray, k: int) -> np.ndarray:
    """Keep the k largest logits of each row; ties go to the lower index."""
    M, n = logits.shape
    order = np.argsort(-logits, axis=1, kind="stable")[:, :k]
    m = np.zeros((M, n), np.uint8)
    np.put_along_axis(m, order, 1, axis=1)
    return m


def router_logits(g, x: np.ndarray, n_groups: int) -> np.ndarray:
    """Random-projection router logits (x R)/sqrt(D), R ~ N(0,1) [D][n_groups]."""
    D = x.shape[1]
    R = g.standard_normal(size=(D, n_groups), dtype=np.float32)
    return (as_f32(x) @ R) / np.float32(np.sqrt(D))


def make_mask(g, kind: str, M: int, n_groups: int, keep: float, x=None) -> np.ndarray:
    if kind == "bernoulli":
        return mask_bernoulli(g, M, n_groups, keep)
    if kind == "beta":
        return mask_beta_groups(g, M, n_groups, keep)
    if kind == "topk":
        return mask_topk(router_logits(g, x, n_groups), keep_count(n_groups, keep))
    if kind == "ones":
        return np.ones((M, n_groups), np.uint8)
    if kind == "zeros":
        return np.zeros((M, n_groups), np.uint8)
    raise ValueError(kind)


# ---- cases -----------------------------------------------------------------

@dataclass
class FFNCase:
    x: np.ndarray
    w_gate: np.ndarray
    w_up: np.ndarray
    w_down: np.ndarray
    mask: np.ndarray
    G: int
    dtype: str

    @property
    def M(self):
        return self.x.shape[0]


def ffn_case(seed: int, M: int, D: int, Dff: int, G: int, dtype: str = "bf16",
             mask: str = "bernoulli", keep: float = 0.5, w_std: float = 0.02) -> FFNCase:
    g = rng(seed)
    x = normal(g, (M, D), 1.0, dtype)
    wg = normal(g, (Dff, D), w_std, dtype)
    wu = normal(g, (Dff, D), w_std, dtype)
    wd = normal(g, (D, Dff), w_std, dtype)
    m = make_mask(g, mask, M, Dff // G, keep, x)
    return FFNCase(x, wg, wu, wd, m, G, dtype)


@dataclass
class AttnCase:
    x: np.ndarray          # [M][D]
    w_q: np.ndarray        # [n_q*hd][D]
    w_k: np.ndarray        # [n_kv*hd][D]
    w_v: np.ndarray        # [n_kv*hd][D]
    w_o: np.ndarray        # [D][n_q*hd]
    a: np.ndarray          # attention output fed to W_o, [M][n_q*hd]
    mask: np.ndarray       # [M][n_q*hd/G]
    G: int
    n_q: int
    n_kv: int
    hd: int
    dtype: str


def attn_case(seed: int, M: int, D: int, n_q: int, n_kv: int, hd: int, G: int,
              dtype: str = "bf16", mask: str = "topk", keep: float = 0.5,
              w_std: float = 0.02) -> AttnCase:
    g = rng(seed)
    x = normal(g, (M, D), 1.0, dtype)
    wq = normal(g, (n_q * hd, D), w_std, dtype)
    wk = normal(g, (n_kv * hd, D), w_std, dtype)
    wv = normal(g, (n_kv * hd, D), w_std, dtype)
    wo = normal(g, (D, n_q * hd), w_std, dtype)
    a = normal(g, (M, n_q * hd), 1.0, dtype)
    m = make_mask(g, mask, M, n_q * hd // G, keep, x)
    return AttnCase(x, wq, wk, wv, wo, a, m, G, n_q, n_kv, hd, dtype)


@dataclass
class AttnPrefillCase:
    q: np.ndarray          # [n_seq*T_q][n_q*hd]
    k: np.ndarray          # [n_seq*T_k][n_kv*hd]
    v: np.ndarray          # [n_seq*T_k][n_kv*hd]
    mask: np.ndarray       # [n_seq*T_q][n_groups]
    n_seq: int
    n_q: int
    n_kv: int
    hd: int
    dtype: str

    @property
    def T_q(self):
        return self.q.shape[0] // self.n_seq

    @property
    def T_k(self):
        return self.k.shape[0] // self.n_seq


def attn_prefill_case(seed: int, n_seq: int, T_q: int, T_k: int, n_q: int, n_kv: int, hd: int,
                      n_groups: int, dtype: str = "bf16", mask: str = "topk", keep: float = 0.5,
                      qk_std: float = 1.0) -> AttnPrefillCase:
    """q, k ~ N(0, qk_std^2) (scores q.k/sqrt(hd) then have std qk_std^2),
    v ~ N(0,1); the mask is drawn from the q rows (top-k of a random
    projection, as for the projections' masks)."""
    g = rng(seed)
    q = normal(g, (n_seq * T_q, n_q * hd), qk_std, dtype)
    k = normal(g, (n_seq * T_k, n_kv * hd), qk_std, dtype)
    v = normal(g, (n_seq * T_k, n_kv * hd), 1.0, dtype)
    m = make_mask(g, mask, n_seq * T_q, n_groups, keep, q)
    return AttnPrefillCase(q, k, v, m, n_seq, n_q, n_kv, hd, dtype)


@dataclass
class AttnDecodeCase:
    q: np.ndarray          # [B][n_q*hd]
    k: np.ndarray          # [B][L][n_kv*hd] key cache
    v: np.ndarray          # [B][L][n_kv*hd] value cache
    mask: np.ndarray       # [B][n_groups]
    kv_len: np.ndarray     # int32 [B]
    n_q: int
    n_kv: int
    hd: int
    dtype: str


def attn_decode_case(seed: int, B: int, L: int, n_q: int, n_kv: int, hd: int, n_groups: int,
                     dtype: str = "bf16", mask: str = "bernoulli", keep: float = 0.5,
                     qk_std: float = 1.0, ragged: bool = False) -> AttnDecodeCase:
    """One query token per sequence against a KV cache of capacity L; with
    `ragged`, each sequence's length is uniform in [1, L] (else L)."""
    g = rng(seed)
    q = normal(g, (B, n_q * hd), qk_std, dtype)
    k = normal(g, (B, L, n_kv * hd), qk_std, dtype)
    v = normal(g, (B, L, n_kv * hd), 1.0, dtype)
    m = make_mask(g, mask, B, n_groups, keep, q)
    kv_len = (g.integers(1, L + 1, B) if ragged else np.full(B, L)).astype(np.int32)
    return AttnDecodeCase(q, k, v, m, kv_len, n_q, n_kv, hd, dtype)


# ---- the paper's workloads (synthetic stand-ins) ---------------------------

@dataclass
class Workload:
    name: str
    desc: str
    params: dict = field(default_factory=dict)


WORKLOADS = {
    "ffn_fp32_small": Workload(
        "ffn_fp32_small",
        "single SwiGLU FFN fp32: D=512, Dff=1536 in 24 groups of 64, T=128, "
        "x~N(0,1), W~N(0,0.02^2), mask Bernoulli(0.5)",
        dict(M=128, D=512, Dff=1536, G=64, dtype="f32", mask="bernoulli", keep=0.5)),
    "ffn_decode_llama7b": Workload(
        "ffn_decode_llama7b",
        "decode FFN bf16, Llama-7B shape: D=4096, Dff=11008 in 86 groups of 128, "
        "B in {1,4,16,64}, p_g~Beta(2,2) rescaled to mean 0.5",
        dict(D=4096, Dff=11008, G=128, dtype="bf16", mask="beta", keep=0.5,
             batches=(1, 4, 16, 64))),
    "ffn_prefill_llama7b": Workload(
        "ffn_prefill_llama7b",
        "prefill FFN bf16, Llama-7B shape, T=4096, top-k of random-projection "
        "router logits (keep 50%, also 25%/75%)",
        dict(M=4096, D=4096, Dff=11008, G=128, dtype="bf16", mask="topk", keep=0.5)),
    "attn_proj_mha": Workload(
        "attn_proj_mha",
        "attention projections bf16: D=4096, 32 heads x 128 in 8 groups of 4 "
        "heads (G=512), T=2048, top-4 of 8 groups",
        dict(M=2048, D=4096, n_q=32, n_kv=32, hd=128, G=512, dtype="bf16",
             mask="topk", keep=0.5)),
    "attn_prefill_llama3_8b": Workload(
        "attn_prefill_llama3_8b",
        "head-group masked causal attention bf16, Llama-3-8B heads: 32 q / 8 kv "
        "heads x 128 in 8 head groups (one KV head each), T=8192 (one sequence), "
        "q,k,v~N(0,1), top-4 of 8 groups per token",
        dict(n_seq=1, T=8192, n_q=32, n_kv=8, hd=128, n_groups=8, dtype="bf16",
             mask="topk", keep=0.5)),
    "attn_decode_llama3_8b": Workload(
        "attn_decode_llama3_8b",
        "head-group masked decode attention bf16, Llama-3-8B heads: 32 q / 8 kv "
        "heads x 128 in 8 head groups, B=32 sequences with 8192 cached keys each, "
        "q,k,v~N(0,1), Bernoulli(0.5) per (token, group)",
        dict(B=32, L=8192, n_q=32, n_kv=8, hd=128, n_groups=8, dtype="bf16", mask="bernoulli",
             keep=0.5)),
    "layer_llama3_8b": Workload(
        "layer_llama3_8b",
        "full decoder-layer projections bf16, Llama-3-8B shape: D=4096, 32 q / "
        "8 kv heads x 128 (8 head groups, G=512), Dff=14336 in 112 groups of "
        "128; prefill T=8192, decode B=32; top-k masks at 25/50/75% sparsity",
        dict(M=8192, M_decode=32, D=4096, n_q=32, n_kv=8, hd=128, G_attn=512,
             Dff=14336, G=128, dtype="bf16", mask="topk", keep=0.5)),
}
