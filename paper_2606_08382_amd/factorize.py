"""Offline factorization of key and value projections into the library's factors.

This is the step that runs once, before inference (Sec. 4.1-4.4): it turns the
dense projections W_K, W_V of one attention layer into the down-projection
A_all and the up-projections B_k, B_v that ``starkv_append`` and
``starkv_decode_attn`` consume.  CPU only (numpy, fp64); nothing here runs on
the decode path.

* Singular values are thresholded per projection (Sec. 4.2): a key head keeps
  the singular values sigma_i >= alpha_K,h of its own projection (head-wise
  decomposition), the values keep those >= alpha_V of the joint projection of
  all heads (joint decomposition); Sec. 4.3.3 gives the reasons for this
  hybrid, Lemmas 1 and 2 (Sec. 4.3.1-4.3.2) the approximation errors.
* The latent of a token is x . (U_r Sigma_r) and the up-projection V_r^T, so
  latent channels come ordered by singular value and scaled by it (Sec. 4.4:
  this is what makes the leading channels outliers).
* Block-wise Hadamard rotations (Sec. 4.4) are fused into the factors:
  A' = A H and B' = H^T B with H = diag(H_out, H_in), one orthonormal block for
  the outlier channels and one for the inliers, so A' B' = A B exactly and the
  library never applies H itself.

Readings (the paper leaves them open):
* The kernels need ranks that are multiples of 16; a thresholded rank is
  raised to the next multiple of 16 (at most the full rank), keeping the next
  singular values as well, which can only lower the approximation error.
* Hadamard matrices of sizes that are not powers of two are taken
  block-diagonal over the binary expansion of the size (Sylvester blocks,
  each normalized): orthonormal, and spreading energy within each block.
* The output projection can take the value up-projection in (Sec. 3.3, weight
  absorption): W'_out,i = W_out,i U_V,g(i) per query head i, stored next to each
  other as one [d_out][H_q * r_v] fp16 matrix (``absorb_output``).
* The outlier block has the library's size for the chosen cache precision
  (MIX8_4: 8*ceil(r/32); MIX4_3: a fifth of r to the nearest multiple of 8,
  at least 8); with no mixed precision there is a single block.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

Q_F16, Q_INT4, Q_MIX8_4, Q_MIX4_3 = 0, 1, 2, 3
RANK_MULTIPLE = 16


def hard_threshold(sigma: np.ndarray, alpha: float) -> int:
    """Effective rank under the hard threshold: the number of sigma_i >= alpha (Sec. 4.2)."""
    return int(np.count_nonzero(np.asarray(sigma) >= alpha))


def soft_threshold(x: np.ndarray, alpha: float, s: float, c: float = 0.0) -> np.ndarray:
    """The differentiable surrogate used while learning alpha (Sec. 4.2):
    x * tanh(s (x - alpha)) for x >= alpha, c * tanh(s (x - alpha)) below it."""
    x = np.asarray(x, dtype=np.float64)
    t = np.tanh(s * (x - alpha))
    return np.where(x >= alpha, x * t, c * t)


def round_rank(r_eff: int, full: int, multiple: int = RANK_MULTIPLE) -> int:
    """A thresholded rank raised to the next multiple the kernels accept (at least one
    multiple, at most the full rank rounded down to a multiple)."""
    cap = max(multiple, (full // multiple) * multiple)
    r = max(multiple, -(-r_eff // multiple) * multiple)
    return min(r, cap)


def truncated_svd(W: np.ndarray, r: int):
    """W (m x n) ~= (U_r Sigma_r) V_r^T: returns (A = U_r Sigma_r, B = V_r^T, sigma)."""
    U, sig, Vt = np.linalg.svd(np.asarray(W, dtype=np.float64), full_matrices=False)
    return U[:, :r] * sig[:r], Vt[:r], sig


def outlier_channels(qmode: int, r: int) -> int:
    if qmode == Q_MIX8_4:
        return 8 * ((r + 31) // 32)
    if qmode == Q_MIX4_3:
        return min(r, 8 * max(1, (r + 20) // 40))
    return 0


def hadamard(n: int) -> np.ndarray:
    """Orthonormal Hadamard-type matrix of order n: Sylvester blocks (normalized) along the
    binary expansion of n, largest first."""
    if n <= 0:
        return np.zeros((0, 0))
    out = np.zeros((n, n))
    pos = 0
    for bit in reversed(range(n.bit_length())):
        k = 1 << bit
        if not n & k:
            continue
        H = np.ones((1, 1))
        while H.shape[0] < k:
            H = np.block([[H, H], [H, -H]])
        out[pos:pos + k, pos:pos + k] = H / np.sqrt(k)
        pos += k
    return out


def block_hadamard(r: int, r_out: int) -> np.ndarray:
    """diag(H(r_out), H(r - r_out)): one rotation for the outlier block, one for the inliers."""
    H = np.zeros((r, r))
    if r_out > 0:
        H[:r_out, :r_out] = hadamard(r_out)
    H[r_out:, r_out:] = hadamard(r - r_out)
    return H


def fuse_hadamard(A: np.ndarray, B: np.ndarray, r_out: int):
    """(A H, H^T B) for the block Hadamard of the latent: the product is unchanged."""
    H = block_hadamard(A.shape[1], r_out)
    return A @ H, H.T @ B


@dataclass
class Factors:
    """Factors of one layer, in fp64 and in the library's storage formats."""
    key_rank: List[int]
    value_rank: int
    A_all: np.ndarray        # [d_model][sum r_g + r_v] fp64: key head blocks in order, then values
    B_k: np.ndarray          # [sum r_g][d] fp64: head g's block at row sum_{g' < g} r_g'
    B_v: np.ndarray          # [r_v][H_kv * d] fp64
    sigma_k: List[np.ndarray]
    sigma_v: np.ndarray

    def storage(self):
        """(A_all as bf16 bits, B_k and B_v as fp16 bits), the layouts starkv_append and
        starkv_decode_attn take."""
        a32 = self.A_all.astype(np.float32)
        u = a32.view(np.uint32).astype(np.uint64)
        # round to nearest even into the top 16 bits
        a_bf16 = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
        return (a_bf16, self.B_k.astype(np.float16).view(np.uint16),
                self.B_v.astype(np.float16).view(np.uint16))


def factorize_layer(W_k: np.ndarray, W_v: np.ndarray, n_kv_heads: int, head_dim: int,
                    alpha_k: Sequence[float], alpha_v: float, qmode: int = Q_MIX8_4,
                    hadamard_fuse: bool = True, key_rank: Optional[Sequence[int]] = None,
                    value_rank: Optional[int] = None) -> Factors:
    """Hybrid decomposition of one layer (Sec. 4.3.3): head-wise SVD of the key projection,
    joint SVD of the value projection, hard thresholds alpha_k (one per KV head) and
    alpha_v, ranks raised to multiples of 16, block Hadamard fused when the cache is mixed
    precision.  W_k, W_v: [d_model][H_kv * head_dim] (k = x W_k, v = x W_v).  Explicit
    key_rank / value_rank override the thresholds."""
    W_k = np.asarray(W_k, dtype=np.float64)
    W_v = np.asarray(W_v, dtype=np.float64)
    d_model = W_k.shape[0]
    assert W_k.shape == (d_model, n_kv_heads * head_dim) and W_v.shape == W_k.shape
    ranks, A_blocks, B_blocks, sig_k = [], [], [], []
    for g in range(n_kv_heads):
        Wg = W_k[:, g * head_dim:(g + 1) * head_dim]
        sig = np.linalg.svd(Wg, compute_uv=False)
        r = (int(key_rank[g]) if key_rank is not None
             else round_rank(hard_threshold(sig, alpha_k[g]), min(Wg.shape)))
        A, B, _ = truncated_svd(Wg, r)
        if hadamard_fuse and qmode in (Q_MIX8_4, Q_MIX4_3, Q_INT4):
            A, B = fuse_hadamard(A, B, outlier_channels(qmode, r))
        ranks.append(r)
        A_blocks.append(A)
        B_blocks.append(B)
        sig_k.append(sig)
    sig_v = np.linalg.svd(W_v, compute_uv=False)
    rv = (int(value_rank) if value_rank is not None
          else round_rank(hard_threshold(sig_v, alpha_v), min(W_v.shape)))
    Av, Bv, _ = truncated_svd(W_v, rv)
    if hadamard_fuse and qmode in (Q_MIX8_4, Q_MIX4_3, Q_INT4):
        Av, Bv = fuse_hadamard(Av, Bv, outlier_channels(qmode, rv))
    return Factors(ranks, rv, np.concatenate(A_blocks + [Av], axis=1), np.concatenate(B_blocks),
                   Bv, sig_k, sig_v)


def absorb_output(W_out: np.ndarray, B_v: np.ndarray, n_q_heads: int, n_kv_heads: int,
                  head_dim: int) -> np.ndarray:
    """Weight absorption of the value up-projection into the output projection (Sec. 3.3).

    W_out: [d_out][H_q * head_dim], the output projection (y = W_out . concat_i o_i);
    B_v:   [r_v][H_kv * head_dim], U_V^T as ``starkv_decode_attn`` takes it.
    Returns W_abs [d_out][H_q * r_v] in fp64 with columns i*r_v .. i*r_v + r_v - 1 holding
    W'_out,i = W_out,i U_V,g(i), g(i) = floor(i * H_kv / H_q), so that
    y = sum_i W'_out,i (a_i / l_i) for the normalized value latents a_i / l_i.  Stored as
    fp16 (``np.float16``) for ``starkv_decode_attn_absorbed``."""
    W_out = np.asarray(W_out, dtype=np.float64)
    B_v = np.asarray(B_v, dtype=np.float64)
    d_out = W_out.shape[0]
    r_v = B_v.shape[0]
    assert W_out.shape[1] == n_q_heads * head_dim and B_v.shape[1] == n_kv_heads * head_dim
    W_abs = np.empty((d_out, n_q_heads * r_v))
    for i in range(n_q_heads):
        g = i * n_kv_heads // n_q_heads
        W_abs[:, i * r_v:(i + 1) * r_v] = (W_out[:, i * head_dim:(i + 1) * head_dim]
                                           @ B_v[:, g * head_dim:(g + 1) * head_dim].T)
    return W_abs
