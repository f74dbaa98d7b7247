"""Seeded synthetic inputs shaped like the paper's Transformer workloads.

The paper evaluates on Llama2/Llama3 inference (Sec. III) without shapes or
data; these generators stand in for it with the hidden sizes of BERT-base,
7B/8B-class and 70B-class models.  This module holds none of the method's
arithmetic: it draws random tensors, rounds them to their storage dtype and,
for attention, forms the scores S = Q K^T / sqrt(d) with the causal mask,
which is how that workload defines its input.  The GPU path and the oracle
both consume exactly the tensors produced here.

Recipe (every tensor has its own stream ``np.random.default_rng([seed,
workload_id, tensor_id])``; draws are fp32; bf16 storage is the
round-to-nearest-even cast of the fp32 draw; N(a, v) names mean a and
variance v):

- LayerNorm -> Linear: x ~ N(0, 1); gamma ~ U(0.5, 1.5); beta ~ N(0, 0.02);
  W[K, N] ~ N(0, 1/K); bias = 0 where a workload states it, else absent.
  RMSNorm -> Linear (Eq. (6), Llama shapes): the same draws without beta.
  RMSNorm -> SwiGLU: the same x and gamma, and two weights W_gate, W_up [K, N]
  ~ N(0, 1/K) from their own streams.
  Optional outlier channels: a fixed set of channel indices (drawn once,
  without replacement) is scaled by a factor in every token, before rounding.
- Softmax -> P.V: either S ~ N(0, s^2) directly (no mask), or S = Q K^T /
  sqrt(d) in fp32 from bf16-rounded Q, K ~ N(0, 1) with keys j > i set to
  -inf (causal); V ~ N(0, 1).
- Attention from Q, K, V: Q, K, V ~ N(0, 1) rounded to bf16, scale 1/sqrt(d);
  decode attention draws Q[Lq] and the cache K, V[Lk] the same way.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence

import numpy as np
import torch

DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16}


@dataclasses.dataclass(frozen=True)
class LNWorkload:
    name: str
    wid: int           # workload id, part of every stream's seed
    M: int             # tokens
    K: int             # hidden size (normalized dimension)
    N: int             # output features
    dtype: str         # "f32" | "bf16"
    eps: float = 1e-5
    outliers: int = 0  # number of fixed outlier channels
    outlier_scale: float = 20.0
    zero_bias: bool = False  # workload states "bias 0"
    norm: str = "layernorm"  # "layernorm" (Eq. (1)-(2)) | "rms" (Eq. (6))

    def flops(self, rows: Optional[int] = None) -> float:
        return 2.0 * (self.M if rows is None else rows) * self.K * self.N


@dataclasses.dataclass(frozen=True)
class SMWorkload:
    name: str
    wid: int
    BH: int            # batch x heads
    L: int             # query length == key length
    d: int             # head dim
    causal: bool
    s_std: float = 2.0        # for scores drawn directly
    from_qk: bool = False     # S = Q K^T / sqrt(d) instead of direct draws

    def pairs(self) -> float:
        """Unmasked (query, key) pairs."""
        if self.causal:
            return self.BH * self.L * (self.L + 1) / 2.0
        return float(self.BH) * self.L * self.L

    def flops(self) -> float:
        return 2.0 * self.pairs() * self.d


# The five workloads, each written as its sizes and distributions.
LN_F32_SMALL = LNWorkload("ln_linear_f32_128x768x3072", 1, 128, 768, 3072, "f32", zero_bias=True)
SM_BF16_SMALL = SMWorkload("softmax_pv_bf16_12x512x512_d64", 2, 12, 512, 64, causal=False, s_std=2.0)
LN_QKV = LNWorkload("ln_qkv_bf16_4096x4096x12288", 3, 4096, 4096, 12288, "bf16", outliers=8)
SM_CAUSAL = SMWorkload("causal_softmax_pv_bf16_32x8192x8192_d128", 4, 32, 8192, 128, causal=True,
                       from_qk=True)
LN_FFN_PREFILL = LNWorkload("ln_ffn_up_bf16_8192x8192x28672", 5, 8192, 8192, 28672, "bf16")


def ln_ffn_decode(t: int) -> LNWorkload:
    """Decode-sized LayerNorm -> FFN up-projection: x[t, 8192], W[8192, 28672]."""
    return LNWorkload(f"ln_ffn_up_bf16_decode_t{t}_8192x28672", 5, t, 8192, 28672, "bf16")


def ln_qkv_tokens(t: int) -> LNWorkload:
    """The QKV projection of LN_QKV over t tokens: batched decode (t <= 128) or a prefill chunk."""
    return LNWorkload(f"ln_qkv_bf16_t{t}_4096x12288", 3, t, 4096, 12288, "bf16", outliers=8)


# Attention from Q, K, V directly (the scores formed in the kernel): the causal
# workload's own tensors, 32 heads x 8192 tokens, d = 128.
ATTN_CAUSAL = SMWorkload("causal_attention_bf16_32x8192x8192_d128", 4, 32, 8192, 128, causal=True, from_qk=True)



@dataclasses.dataclass(frozen=True)
class DecodeAttnWorkload:
    """Attention of a few new query tokens against a cache of Lk keys (every key visible).

    ``group`` query heads share each key/value head (grouped-query attention; 1 = one
    query head per key/value head); query head h * group + r reads key/value head h.
    """
    name: str
    wid: int
    BH: int            # sequences x key/value heads
    Lq: int            # new tokens per sequence (group * Lq <= 16)
    Lk: int            # cached keys
    d: int             # head dim
    group: int = 1     # query heads per key/value head

    def pairs(self) -> float:
        return float(self.BH) * self.group * self.Lq * self.Lk

    def flops(self) -> float:
        return 4.0 * self.pairs() * self.d  # both products

    def bytes(self) -> float:
        """Algorithmic HBM bytes: K and V read once, Q read and the output written (bf16)."""
        return 2.0 * (2.0 * self.BH * self.Lk * self.d + 2.0 * self.BH * self.group * self.Lq * self.d)


# Decode attention: 8 sequences x 32 heads, one new token each against 8192 cached
# keys of d = 128 (1 GiB of K and V, larger than the last-level cache).
ATTN_DECODE = DecodeAttnWorkload("decode_attention_bf16_256x1x8192_d128", 10, 256, 1, 8192, 128)
# The same cache read by grouped queries, as in 8B-class Llama 3 models: 32 sequences x
# 8 key/value heads, each shared by 4 of the 32 query heads, one new token.
ATTN_DECODE_GQA = DecodeAttnWorkload("decode_attention_gqa4_bf16_256kv_x1x8192_d128", 11, 256, 1, 8192, 128,
                                     group=4)


# RMSNorm -> Linear with Llama shapes: the fused QKV projection of an 8B-class
# model with grouped-query attention (32 query + 2 x 8 key/value heads of 128
# over hidden 4096), and the 70B-class FFN up-projection at decode.
RMS_QKV = LNWorkload("rms_qkv_bf16_4096x4096x6144", 6, 4096, 4096, 6144, "bf16", outliers=8, norm="rms")


def rms_ffn_decode(t: int) -> LNWorkload:
    """Decode-sized RMSNorm -> FFN up-projection: x[t, 8192], W[8192, 28672]."""
    return LNWorkload(f"rms_ffn_up_bf16_decode_t{t}_8192x28672", 7, t, 8192, 28672, "bf16", norm="rms")


# RMSNorm -> SwiGLU (gate and up projections of the Llama MLP): an 8B-class
# prefill (hidden 4096, intermediate 14336) and a 70B-class decode token
# (hidden 8192, intermediate 28672).  N is the intermediate size; FLOP count
# both products.
SWIGLU_PREFILL = LNWorkload("rms_swiglu_bf16_4096x4096x14336", 8, 4096, 4096, 14336, "bf16", outliers=8,
                            norm="rms")


def swiglu_decode(t: int) -> LNWorkload:
    return LNWorkload(f"rms_swiglu_bf16_decode_t{t}_8192x28672", 9, t, 8192, 28672, "bf16", norm="rms")


WORKLOADS = {w.name: w for w in (LN_F32_SMALL, SM_BF16_SMALL, LN_QKV, SM_CAUSAL, LN_FFN_PREFILL,
                                 ln_ffn_decode(1), ln_ffn_decode(4), ln_ffn_decode(16),
                                 ln_qkv_tokens(32), ln_qkv_tokens(128), ln_qkv_tokens(1024),
                                 RMS_QKV, rms_ffn_decode(1), SWIGLU_PREFILL, swiglu_decode(1), ATTN_CAUSAL,
                                 ATTN_DECODE, ATTN_DECODE_GQA)}

# tensor ids inside a workload's seed
_X, _GAMMA, _BETA, _W, _OUTLIER_CH, _S, _Q, _KEY, _V, _W_UP = range(10)


def _rng(seed: int, wid: int, tid: int, extra: int = 0) -> np.random.Generator:
    return np.random.default_rng([seed, wid, tid, extra])


def to_storage(a: np.ndarray, dtype: str) -> torch.Tensor:
    """fp32 array -> torch CPU tensor in the storage dtype (bf16: round to nearest even)."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(DTYPES[dtype]) if dtype != "f32" else t.clone()


def _normal(rng, shape, std):
    a = rng.standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return a


def make_ln(w: LNWorkload, seed: int = 0, M: Optional[int] = None, x_extra: int = 0) -> dict:
    """Inputs of a LayerNorm -> Linear workload as CPU tensors in storage dtype.

    ``M`` overrides the token count (the weights do not depend on it); ``x_extra``
    selects an independent activation stream with the same weights.
    """
    M = w.M if M is None else M
    x = _normal(_rng(seed, w.wid, _X, x_extra), (M, w.K), 1.0)
    if w.outliers:
        ch = _rng(seed, w.wid, _OUTLIER_CH).choice(w.K, size=w.outliers, replace=False)
        x[:, ch] *= np.float32(w.outlier_scale)
    gamma = _rng(seed, w.wid, _GAMMA).uniform(0.5, 1.5, w.K).astype(np.float32)
    beta = _normal(_rng(seed, w.wid, _BETA), (w.K,), math.sqrt(0.02))
    W = _normal(_rng(seed, w.wid, _W), (w.K, w.N), 1.0 / math.sqrt(w.K))
    out = dict(x=to_storage(x, w.dtype), gamma=to_storage(gamma, w.dtype),
               beta=to_storage(beta, w.dtype) if w.norm == "layernorm" else None,
               W=to_storage(W, w.dtype), bias=None, eps=w.eps, norm=w.norm)
    if w.zero_bias:
        out["bias"] = torch.zeros(w.N, dtype=DTYPES[w.dtype])
    return out


def make_swiglu(w: LNWorkload, seed: int = 0, M: Optional[int] = None) -> dict:
    """Inputs of an RMSNorm -> SwiGLU workload: x, gamma, W_gate (the LN recipe's W) and W_up."""
    out = make_ln(w, seed, M)
    Wu = _normal(_rng(seed, w.wid, _W_UP), (w.K, w.N), 1.0 / math.sqrt(w.K))
    out.update(Wg=out.pop("W"), Wu=to_storage(Wu, w.dtype), beta=None)
    return out


def make_swiglu_case(M: int, K: int, N: int, dtype: str, seed: int = 0, outliers: int = 0,
                     eps: float = 1e-5) -> dict:
    """An RMSNorm -> SwiGLU case of any size with the same recipe (for parity tests)."""
    return make_swiglu(LNWorkload(f"swiglu_{M}x{K}x{N}_{dtype}", 101, M, K, N, dtype, eps=eps, outliers=outliers,
                                  norm="rms"), seed)


def make_ln_case(M: int, K: int, N: int, dtype: str, seed: int = 0, outliers: int = 0,
                 zero_bias: bool = False, mean_offset: float = 0.0, eps: float = 1e-5,
                 norm: str = "layernorm") -> dict:
    """A LayerNorm (or RMSNorm) -> Linear case of any size with the same recipe (for parity tests)."""
    w = LNWorkload(f"case_{M}x{K}x{N}_{dtype}", 100, M, K, N, dtype, eps=eps, outliers=outliers,
                   zero_bias=zero_bias, norm=norm)
    out = make_ln(w, seed)
    if mean_offset:
        x = out["x"].float() + mean_offset
        out["x"] = x.to(DTYPES[dtype])
    return out


def _scores_direct(rng, BH, L, std):
    return _normal(rng, (BH, L, L), std)


def make_sm(w: SMWorkload, seed: int = 0, heads: Optional[Sequence[int]] = None,
            L: Optional[int] = None) -> dict:
    """Inputs of a Softmax -> P.V workload: S[BH, L, L] and V[BH, L, d] (bf16 CPU tensors).

    ``heads`` restricts generation to a subset of heads (each head has its own
    streams, so a subset equals the corresponding slice of the full tensor).
    """
    L = w.L if L is None else L
    heads = list(range(w.BH)) if heads is None else list(heads)
    S = torch.empty((len(heads), L, L), dtype=torch.bfloat16)
    V = torch.empty((len(heads), L, w.d), dtype=torch.bfloat16)
    mask = torch.triu(torch.ones(L, L, dtype=torch.bool), diagonal=1) if w.causal else None
    for i, h in enumerate(heads):
        if w.from_qk:
            q = to_storage(_normal(_rng(seed, w.wid, _Q, h), (L, w.d), 1.0), "bf16").float()
            k = to_storage(_normal(_rng(seed, w.wid, _KEY, h), (L, w.d), 1.0), "bf16").float()
            s = torch.matmul(q, k.t()) * (1.0 / math.sqrt(w.d))
        else:
            s = torch.from_numpy(_normal(_rng(seed, w.wid, _S, h), (L, L), w.s_std))
        if mask is not None:
            s = s.masked_fill(mask, float("-inf"))
        S[i] = s.to(torch.bfloat16)
        V[i] = to_storage(_normal(_rng(seed, w.wid, _V, h), (L, w.d), 1.0), "bf16")
    return dict(S=S, V=V, causal=w.causal)


def make_qkv(w: SMWorkload, seed: int = 0, heads: Optional[Sequence[int]] = None,
             L: Optional[int] = None) -> dict:
    """Q, K, V[BH, L, d] (bf16 CPU tensors) of a workload whose scores come from Q K^T.

    The same streams as make_sm's, so S = Q K^T / sqrt(d) (fp32, then bf16) of
    make_sm is exactly the score matrix these tensors define.
    """
    assert w.from_qk, w
    L = w.L if L is None else L
    heads = list(range(w.BH)) if heads is None else list(heads)
    Q, K, V = (torch.empty((len(heads), L, w.d), dtype=torch.bfloat16) for _ in range(3))
    for i, h in enumerate(heads):
        Q[i] = to_storage(_normal(_rng(seed, w.wid, _Q, h), (L, w.d), 1.0), "bf16")
        K[i] = to_storage(_normal(_rng(seed, w.wid, _KEY, h), (L, w.d), 1.0), "bf16")
        V[i] = to_storage(_normal(_rng(seed, w.wid, _V, h), (L, w.d), 1.0), "bf16")
    return dict(Q=Q, K=K, V=V, causal=w.causal, scale=1.0 / math.sqrt(w.d))


def make_qkv_case(BH: int, L: int, d: int, causal: bool, seed: int = 0) -> dict:
    """Q, K, V of any size with the same recipe (for parity tests)."""
    return make_qkv(SMWorkload(f"attn_{BH}x{L}_d{d}", 201, BH, L, d, causal, from_qk=True), seed)


def make_decode(w: DecodeAttnWorkload, seed: int = 0, heads: Optional[Sequence[int]] = None) -> dict:
    """Q[n * group, Lq, d] and the cache K, V[n, Lk, d] (bf16 CPU tensors) of the listed
    key/value heads (query heads h * group .. h * group + group - 1 for head h)."""
    heads = list(range(w.BH)) if heads is None else list(heads)
    g = w.group
    Q = torch.empty((len(heads) * g, w.Lq, w.d), dtype=torch.bfloat16)
    K, V = (torch.empty((len(heads), w.Lk, w.d), dtype=torch.bfloat16) for _ in range(2))
    for i, h in enumerate(heads):
        for r in range(g):
            Q[i * g + r] = to_storage(_normal(_rng(seed, w.wid, _Q, h * g + r), (w.Lq, w.d), 1.0), "bf16")
        K[i] = to_storage(_normal(_rng(seed, w.wid, _KEY, h), (w.Lk, w.d), 1.0), "bf16")
        V[i] = to_storage(_normal(_rng(seed, w.wid, _V, h), (w.Lk, w.d), 1.0), "bf16")
    return dict(Q=Q, K=K, V=V, causal=False, scale=1.0 / math.sqrt(w.d))


def make_decode_case(BH: int, Lq: int, Lk: int, d: int, seed: int = 0, group: int = 1) -> dict:
    """A decode-attention case of any size with the same recipe (for parity tests)."""
    return make_decode(DecodeAttnWorkload(f"decode_{BH}x{Lq}x{Lk}_d{d}_g{group}", 203, BH, Lq, Lk, d, group), seed)


def make_sm_case(BH: int, L: int, d: int, causal: bool, seed: int = 0, s_std: float = 2.0,
                 from_qk: bool = False) -> dict:
    """A Softmax -> P.V case of any size with the same recipe (for parity tests)."""
    w = SMWorkload(f"case_{BH}x{L}_d{d}", 200, BH, L, d, causal, s_std=s_std, from_qk=from_qk)
    return make_sm(w, seed)


def sample_rows(n_rows: int, k: int, seed: int = 0) -> np.ndarray:
    """k distinct row indices in [0, n_rows): the first, the last and a seeded sample."""
    k = min(k, n_rows)
    rng = np.random.default_rng([seed, 999])
    picked = {0, n_rows - 1}
    rest = rng.choice(n_rows, size=min(n_rows, k + 2), replace=False)
    for r in rest:
        if len(picked) >= k:
            break
        picked.add(int(r))
    return np.array(sorted(picked)[:k], dtype=np.int64)
