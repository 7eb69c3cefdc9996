"""Seeded synthetic inputs for the decode path (shared by tests, bench and the oracle side).

This module draws random numbers and rounds them to their storage types; it
holds none of the method's arithmetic.  One numpy PCG64 stream per call, drawn
in a fixed order: ranks, outlier channels, B_k, B_v, q, ctx lengths, latents
(sequence by sequence), hidden states and down-projection weights, needles.

Distributions (stand-ins for LLaMA-shaped latent caches, whose trained ranks
and weights are not available):
  * latent channel i (1-based within its key head or the value block)
    ~ N(0, sigma_i^2), sigma_i = i^-1/2 (the latent is scaled by the singular
    values, so leading channels are larger);
  * optional outlier channels: a seeded 1 % of all latent channels get x8;
  * B_k,g ~ N(0,1)/sqrt(r_g), B_v ~ N(0,1)/sqrt(r_v), stored fp16;
  * q ~ N(0,1) (already rotated), fp16 or bf16;
  * hidden states x ~ N(0,1) bf16; down-projection column i ~ N(0,1)*sigma_i/sqrt(d_model);
  * absorbed output weights W'_out,i (``absorbed_weights``, own stream): entries
    ~ N(0, 1/(H_q r_v)), the variance of W_out,i U_V,i for an output projection
    W_out ~ N(0, 1/(H_q d)) and U_V as above; fp16;
  * peaked variant of strength k (peaked=True is k = 1): q x 4k and four needle
    tokens per sequence whose key latents are scaled x 8k (attention concentrates
    on a few tokens with large scores; outputs of order 0.5-1.5).
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import List, Optional

import numpy as np

Q_F16, Q_INT4, Q_MIX8_4, Q_MIX4_3 = 0, 1, 2, 3
DT_F16, DT_BF16, DT_F32 = 0, 1, 2


@dataclass
class Workload:
    name: str
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ctx: int                       # context length per sequence (max for ragged)
    key_rank: Optional[List[int]]  # None: drawn per `rank_draw`
    rank_draw: str                 # "fixed" | "choice:16,32,..." | "perm:16,16,32,..."
    value_rank: int
    qmode: int
    rope_theta: float
    q_dtype: int
    out_dtype: int
    outlier_frac: float = 0.0      # fraction of latent channels scaled x8
    ragged: Optional[tuple] = None  # (lo, hi) for uniform ragged context lengths
    d_model: int = 0               # hidden size of the append-from-hidden step
    append_tokens: int = 0         # tokens appended per sequence per step
    seed: int = 0
    extra: dict = field(default_factory=dict)

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# The five workloads; small variants for parity tests are derived with `shrink`.
WORKLOADS = {
    "c1": Workload("c1_mha4x1_d64_ctx1k_r16_f16", 1, 4, 1, 64, 1024, [16], "fixed", 16,
                   Q_F16, 1e4, DT_F16, DT_F16, seed=1001),
    "c2": Workload("c2_llama8b_b4_ctx32k_int4", 4, 32, 8, 128, 32768, None,
                   "choice:16,32,48,64,96", 256, Q_INT4, 5e5, DT_BF16, DT_BF16, seed=1002),
    "c3": Workload("c3_llama8b_b4_ctx128k_mix8_4", 4, 32, 8, 128, 131072, None,
                   "perm:16,16,32,32,32,32,48,48", 256, Q_MIX8_4, 5e5, DT_BF16, DT_BF16,
                   outlier_frac=0.01, d_model=4096, append_tokens=1, seed=1003),
    "c4": Workload("c4_llama8b_b32_ragged2k_16k_int4", 32, 32, 8, 128, 16384, None,
                   "perm:16,16,16,32,32,48,48,48", 256, Q_INT4, 5e5, DT_BF16, DT_BF16,
                   ragged=(2048, 16384), d_model=4096, append_tokens=1, seed=1004),
    "c5": Workload("c5_70b_b2_ctx64k_mix8_4", 2, 64, 8, 128, 65536, None,
                   "choice:32,48,64,80,96,112,128", 384, Q_MIX8_4, 5e5, DT_BF16, DT_BF16,
                   d_model=8192, append_tokens=4096, seed=1005),
    # C3's layer with the paper's own quantizer: about 20 % of the channels in
    # 4 bits, the rest in 3 bits
    "c3q": Workload("c3q_llama8b_b4_ctx128k_mix4_3", 4, 32, 8, 128, 131072, None,
                    "perm:16,16,32,32,32,32,48,48", 256, Q_MIX4_3, 5e5, DT_BF16, DT_BF16,
                    outlier_frac=0.01, d_model=4096, append_tokens=1, seed=1006),
    "c5q": Workload("c5q_70b_b2_ctx64k_mix4_3", 2, 64, 8, 128, 65536, None,
                    "choice:32,48,64,80,96,112,128", 384, Q_MIX4_3, 5e5, DT_BF16, DT_BF16,
                    d_model=8192, append_tokens=4096, seed=1007),
}


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def to_bits(a: np.ndarray, dtype: int) -> np.ndarray:
    if dtype == DT_BF16:
        return f32_to_bf16_bits(a.astype(np.float32))
    return np.ascontiguousarray(a.astype(np.float16)).view(np.uint16)


def draw_ranks(w: Workload, rng: np.random.Generator) -> List[int]:
    if w.key_rank is not None:
        return list(w.key_rank)
    kind, vals = w.rank_draw.split(":")
    vals = [int(v) for v in vals.split(",")]
    if kind == "choice":
        return [int(v) for v in rng.choice(vals, size=w.n_kv_heads)]
    if kind == "perm":
        assert len(vals) == w.n_kv_heads
        return [int(v) for v in rng.permutation(vals)]
    raise ValueError(w.rank_draw)


def sigmas(width_blocks: List[int]) -> np.ndarray:
    """Per-channel scale i^-1/2, restarting at i = 1 in every block."""
    return np.concatenate([np.arange(1, r + 1, dtype=np.float64) ** -0.5 for r in width_blocks])


@dataclass
class Inputs:
    w: Workload
    key_rank: List[int]
    value_rank: int
    Bk: np.ndarray          # fp16 bits [sum_r][d]
    Bv: np.ndarray          # fp16 bits [r_v][H_kv*d]
    q: np.ndarray           # q_dtype bits [B][H_q][d]
    ctx_len: np.ndarray     # int32 [B]
    latents: np.ndarray     # fp16 bits [B][L][sum_r + r_v]
    scale: np.ndarray       # per-channel std of the latents (incl. outliers)
    x: Optional[np.ndarray] = None   # bf16 bits [B][n_app][d_model]
    A: Optional[np.ndarray] = None   # bf16 bits [d_model][sum_r + r_v]
    needles: Optional[np.ndarray] = None

    @property
    def width(self) -> int:
        return sum(self.key_rank) + self.value_rank


def generate(w: Workload, seed: Optional[int] = None, peaked: int = 0,
             with_latents: bool = True, with_hidden: bool = False,
             n_hidden_tokens: Optional[int] = None) -> Inputs:
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    ranks = draw_ranks(w, rng)
    width = sum(ranks) + w.value_rank
    scale = sigmas(ranks + [w.value_rank])
    if w.outlier_frac > 0:
        n_out = int(np.ceil(w.outlier_frac * width))
        idx = rng.choice(width, size=n_out, replace=False)
        scale = scale.copy()
        scale[idx] *= 8.0
    d = w.head_dim
    Bk = np.concatenate([rng.standard_normal((r, d)) / np.sqrt(r) for r in ranks], axis=0)
    Bv = rng.standard_normal((w.value_rank, w.n_kv_heads * d)) / np.sqrt(w.value_rank)
    q = rng.standard_normal((w.batch, w.n_q_heads, d))
    strength = int(peaked)
    if strength:
        q = q * (4.0 * strength)
    if w.ragged is not None:
        lo, hi = w.ragged
        ctx = rng.integers(lo, hi + 1, size=w.batch).astype(np.int32)
    else:
        ctx = np.full(w.batch, w.ctx, np.int32)
    L = int(ctx.max()) if w.batch else 0
    latents = None
    if with_latents:
        latents = np.empty((w.batch, L, width), np.uint16)
        sc32 = scale.astype(np.float32)
        for b in range(w.batch):
            z = rng.standard_normal((L, width), dtype=np.float32)
            z *= sc32
            latents[b] = np.ascontiguousarray(z.astype(np.float16)).view(np.uint16)
    needles = None
    if peaked and with_latents:
        # up to four per sequence (fewer in a context shorter than four tokens)
        needles = [rng.choice(int(ctx[b]), size=min(4, int(ctx[b])), replace=False)
                   for b in range(w.batch)]
        ksum = sum(ranks)
        for b in range(w.batch):
            for t in needles[b]:
                v = latents[b, t, :ksum].view(np.float16).astype(np.float32) * (8.0 * strength)
                latents[b, t, :ksum] = np.ascontiguousarray(v.astype(np.float16)).view(np.uint16)
    x = A = None
    if with_hidden:
        n_tok = n_hidden_tokens if n_hidden_tokens is not None else w.append_tokens
        x = f32_to_bf16_bits(rng.standard_normal((w.batch, n_tok, w.d_model), dtype=np.float32))
        Af = rng.standard_normal((w.d_model, width), dtype=np.float32)
        Af *= (scale / np.sqrt(w.d_model)).astype(np.float32)
        A = f32_to_bf16_bits(Af)
    return Inputs(w=w, key_rank=ranks, value_rank=w.value_rank,
                  Bk=to_bits(Bk, DT_F16), Bv=to_bits(Bv, DT_F16),
                  q=to_bits(q, w.q_dtype), ctx_len=ctx, latents=latents, scale=scale,
                  x=x, A=A, needles=needles)


def absorbed_weights(w: Workload, d_out: int, seed: Optional[int] = None) -> np.ndarray:
    """fp16 bits [d_out][H_q * r_v]: the absorbed output weights, one column block per query
    head (drawn from their own stream, seed w.seed + 7919 unless given)."""
    rng = np.random.Generator(np.random.PCG64(w.seed + 7919 if seed is None else seed))
    k = w.n_q_heads * w.value_rank
    W = rng.standard_normal((d_out, k), dtype=np.float32)
    W *= np.float32(1.0 / np.sqrt(k))
    return to_bits(W, DT_F16)


def shrink(w: Workload, ctx: int, batch: Optional[int] = None, ragged=None) -> Workload:
    """Same heads, ranks and formats at a size the oracle finishes in seconds."""
    return w.with_(ctx=ctx, batch=w.batch if batch is None else batch, ragged=ragged,
                   name=w.name + f"_ctx{ctx}")
