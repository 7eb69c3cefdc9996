"""The offline factorization (Sec. 4.1-4.4) against the facts the paper states for it:
Lemma 1 (Eckart-Young-Mirsky, spectral norm), Lemma 2 (joint beats head-wise under the same
budget), the hard threshold, the soft-threshold surrogate, and the block Hadamard fusion
(orthonormal, exact in the product, smoothing the quantized latent).  CPU only."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_08382_amd import factorize as F


def _spectrum_matrix(rng, m, n, decay=0.8):
    U, _ = np.linalg.qr(rng.standard_normal((m, m)))
    V, _ = np.linalg.qr(rng.standard_normal((n, n)))
    p = min(m, n)
    s = decay ** np.arange(p) * (1 + 0.1 * rng.random(p))
    s = np.sort(s)[::-1]
    return (U[:, :p] * s) @ V[:, :p].T, s


def test_lemma1_truncated_svd_spectral_error_is_next_singular_value():
    rng = np.random.default_rng(1)
    W, s = _spectrum_matrix(rng, 96, 64)
    for r in (1, 8, 16, 40):
        A, B, sig = F.truncated_svd(W, r)
        err = np.linalg.norm(W - A @ B, 2) / np.linalg.norm(W, 2)
        assert abs(err - sig[r] / sig[0]) < 1e-12
        # no other rank-r matrix does better: truncations of perturbed copies of W
        for _ in range(3):
            A2, B2, _ = F.truncated_svd(W + 1e-2 * rng.standard_normal(W.shape), r)
            assert np.linalg.norm(W - A2 @ B2, 2) / np.linalg.norm(W, 2) >= err - 1e-12


def test_lemma2_joint_rank_beats_headwise_at_equal_budget():
    rng = np.random.default_rng(2)
    for trial in range(5):
        h, dh, r = 4, 16, 4
        W = rng.standard_normal((80, h * dh)) @ np.diag(0.9 ** np.arange(h * dh))
        A, B, _ = F.truncated_svd(W, h * r)
        joint = np.linalg.norm(W - A @ B)
        parts = []
        for i in range(h):
            Ai, Bi, _ = F.truncated_svd(W[:, i * dh:(i + 1) * dh], r)
            parts.append(Ai @ Bi)
        hw = np.linalg.norm(W - np.concatenate(parts, axis=1))
        assert joint <= hw + 1e-12
        # the head-wise candidate has rank <= h r (the feasible-set argument of the proof)
        assert np.linalg.matrix_rank(np.concatenate(parts, axis=1)) <= h * r


def test_hard_threshold_and_rank_rounding():
    s = np.array([9.0, 5.0, 3.0, 2.0, 1.0, 0.5])
    assert [F.hard_threshold(s, a) for a in (10, 9, 4, 2, 0.1)] == [0, 1, 2, 4, 6]
    # raised to the next multiple of 16, at least 16, at most the full rank's multiple
    assert [F.round_rank(r, 128) for r in (0, 1, 16, 17, 100, 128)] == [16, 16, 16, 32, 112, 128]
    assert F.round_rank(70, 64) == 64


def test_soft_threshold_surrogate_limits():
    x = np.array([0.1, 0.9, 1.0, 1.5, 5.0])
    y = F.soft_threshold(x, 1.0, 50.0)
    assert np.all(y[:2] == 0.0)                      # c = 0: sub-threshold values suppressed
    assert y[2] == 0.0                               # tanh(0) at the threshold
    assert abs(y[4] - 5.0) < 1e-12                   # far above: preserved
    # sharper s approaches the hard cutoff x * 1{x >= alpha}
    xs = np.linspace(0, 3, 301)
    hard = xs * (xs >= 1.2)
    errs = [np.abs(F.soft_threshold(xs, 1.2, s) - hard)[np.abs(xs - 1.2) > 0.05].max()
            for s in (5, 50, 500)]
    assert errs[0] > errs[1] > errs[2]


@pytest.mark.parametrize("n", [8, 16, 24, 48, 80, 208])
def test_hadamard_blocks_are_orthonormal(n):
    H = F.hadamard(n)
    np.testing.assert_allclose(H @ H.T, np.eye(n), atol=1e-13)
    # entries are +-1/sqrt(block size) inside the blocks, zero outside
    assert np.all(np.isin(np.round(np.abs(H[H != 0]) ** -2), [1, 2, 4, 8, 16, 32, 64, 128, 256]))


@pytest.mark.parametrize("qmode,r", [(F.Q_MIX8_4, 48), (F.Q_MIX4_3, 128), (F.Q_INT4, 32)])
def test_fused_hadamard_keeps_the_product_and_the_block_boundary(qmode, r):
    rng = np.random.default_rng(3)
    A = rng.standard_normal((64, r))
    B = rng.standard_normal((r, 40))
    ro = F.outlier_channels(qmode, r)
    assert ro == O.outlier_channels({F.Q_MIX8_4: O.Q_MIX8_4, F.Q_MIX4_3: O.Q_MIX4_3,
                                     F.Q_INT4: O.Q_INT4}[qmode], r)
    A2, B2 = F.fuse_hadamard(A, B, ro)
    np.testing.assert_allclose(A2 @ B2, A @ B, rtol=1e-12, atol=1e-12)
    H = F.block_hadamard(r, ro)
    assert np.all(H[:ro, ro:] == 0) and np.all(H[ro:, :ro] == 0)   # regions stay apart


def test_block_hadamard_lowers_the_quantization_error_of_a_spiky_latent():
    """Sec. 4.4: the rotation spreads a dominant channel's energy over its block, so the
    per-token group quantizer wastes fewer levels on it (measured with the oracle's quantizer,
    after rotating back)."""
    rng = np.random.default_rng(4)
    r, qm = 64, O.Q_MIX4_3
    ro = O.outlier_channels(qm, r)
    H = F.block_hadamard(r, ro)
    worse = 0
    for _ in range(40):
        z = rng.standard_normal(r) * 0.05
        z[ro + rng.integers(0, r - ro)] += 4.0          # one spike among the inliers
        def err(v, rot):
            bits = O.f16_bits(v @ rot)
            codes, s, zz = O.quantize_block(qm, bits)
            deq = np.array([float(np.float16(np.uint16(zz[O.channel_group(qm, r, c)[0]]).view(np.float16)))
                            + codes[c] * float(np.uint16(s[O.channel_group(qm, r, c)[0]]).view(np.float16))
                            for c in range(r)])
            return np.linalg.norm(deq @ rot.T - v)
        worse += err(z, H) > err(z, np.eye(r))
    assert worse <= 4


def test_factors_feed_the_decode_path_end_to_end():
    """Factors of full rank reproduce dense attention with K = x W_K and V = x W_V through the
    oracle's cache path (fp16 latents, fp16 up-projections)."""
    rng = np.random.default_rng(5)
    d_model, Hkv, Hq, d, L = 64, 2, 4, 16, 12
    Wk = rng.standard_normal((d_model, Hkv * d)) / 8
    Wv = rng.standard_normal((d_model, Hkv * d)) / 8
    f = F.factorize_layer(Wk, Wv, Hkv, d, alpha_k=[0.0] * Hkv, alpha_v=0.0, qmode=F.Q_F16,
                          hadamard_fuse=False)
    assert f.key_rank == [16, 16] and f.value_rank == 32
    x = rng.standard_normal((L, d_model))
    lat = O.f16_bits(x @ f.A_all)
    _, Bk, Bv = f.storage()
    cfg = O.make_cfg(1, Hq, Hkv, d, L, f.key_rank, f.value_rank, O.Q_F16, 1e4)
    cache = O.new_cache(cfg)
    O.append(cfg, cache, lat.reshape(1, L, -1), [0])
    q = O.f16_bits(rng.standard_normal((1, Hq, d)))
    out, _ = O.decode_attn(cfg, cache, q, False, Bk, Bv, [L])
    K, V = x @ Wk, x @ Wv
    for i in range(Hq):
        g = i * Hkv // Hq
        ref = O.dense_attn(q[0, i].view(np.float16).astype(np.float64), K[:, g * d:(g + 1) * d],
                           V[:, g * d:(g + 1) * d], 1e4)
        np.testing.assert_allclose(out[0, i], ref, rtol=2e-2, atol=2e-3)


def test_storage_formats():
    rng = np.random.default_rng(6)
    f = F.factorize_layer(rng.standard_normal((32, 32)), rng.standard_normal((32, 32)), 2, 16,
                          alpha_k=[0.0, 0.0], alpha_v=0.0, qmode=F.Q_MIX8_4)
    a, bk, bv = f.storage()
    assert a.dtype == np.uint16 and a.shape == (32, 16 + 16 + 32)
    back = (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert np.all(np.abs(back - f.A_all) <= np.abs(f.A_all) * 2.0 ** -8)
    assert bk.shape == (32, 16) and bv.shape == (32, 32)


def test_absorbed_output_weights_match_the_per_head_products():
    """W'_out,i = W_out,i U_V,g(i) (Sec. 3.3), with GQA's head map, against an explicit
    contraction over the head dimension written with einsum."""
    rng = np.random.default_rng(7)
    Hq, Hkv, d, rv, d_out = 6, 2, 8, 16, 20
    W_out = rng.standard_normal((d_out, Hq * d))
    B_v = rng.standard_normal((rv, Hkv * d))
    W_abs = F.absorb_output(W_out, B_v, Hq, Hkv, d)
    Wo = W_out.reshape(d_out, Hq, d)
    Bv = B_v.reshape(rv, Hkv, d)
    g_of = np.array([i * Hkv // Hq for i in range(Hq)])
    ref = np.einsum("nij,cij->nic", Wo, Bv[:, g_of, :]).reshape(d_out, Hq * rv)
    np.testing.assert_allclose(W_abs, ref, rtol=1e-13, atol=1e-13)
    # y = W_out concat(o) for o_i = lat_i U_V,g(i): absorption changes nothing in fp64
    lat = rng.standard_normal((3, Hq, rv))
    o = np.stack([lat[:, i] @ Bv[:, g_of[i], :] for i in range(Hq)], axis=1)
    np.testing.assert_allclose(lat.reshape(3, -1) @ W_abs.T, o.reshape(3, -1) @ W_out.T,
                               rtol=1e-12, atol=1e-12)
