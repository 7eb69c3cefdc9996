"""The offline factorization's output on the HIP path (Sec. 4.3.3, Sec. 4.4).

factorize_layer turns dense W_K, W_V of a Llama-3.1-8B-shaped layer into the head-wise
key factors and the joint value factors, with the block Hadamard rotations fused into
A and B; Factors.storage() gives the bf16 / fp16 arrays the library takes.  The GPU then
appends hidden states through the down-projection and decodes.  Checks: the GPU's fp16
latents against the oracle's fp64 down-projection (1 fp16 ulp plus the fp32 summation
bound), the packed cache bit-exact when the oracle quantizes the GPU's latents, and every
attention output against the oracle on the same factors (fp32 output, bare bound).
"""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_08382_amd import factorize as F
from paper_2606_08382_amd import synth

from _helpers import assert_close, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _projection(rng, d_model, width, decay):
    """A dense projection with a decaying spectrum (singular values i^-decay), so that the
    thresholds and the outlier regions have something to act on."""
    U, _ = np.linalg.qr(rng.standard_normal((d_model, width)))
    V, _ = np.linalg.qr(rng.standard_normal((width, width)))
    s = np.arange(1, width + 1, dtype=np.float64) ** -decay
    return (U * s) @ V.T * 4.0


@pytest.mark.parametrize("qmode", [F.Q_MIX8_4, F.Q_MIX4_3])
def test_factorized_layer_on_the_gpu_path(qmode):
    from paper_2606_08382_amd.device import Layer, to_dev
    rng = np.random.default_rng(31 + qmode)
    d_model, Hq, Hkv, d, B, L = 1024, 32, 8, 128, 2, 1500
    Wk = np.concatenate([_projection(rng, d_model, d, 1.0) for _ in range(Hkv)], axis=1)
    Wv = _projection(rng, d_model, Hkv * d, 0.7)
    f = F.factorize_layer(Wk, Wv, Hkv, d, alpha_k=[0.05, 0.1, 0.2, 0.08, 0.3, 0.06, 0.12, 0.5],
                          alpha_v=0.1, qmode=qmode)
    say(f"factorized: key ranks {f.key_rank}, value rank {f.value_rank}, qmode {qmode}")
    assert len(set(f.key_rank)) > 1 and all(r % 16 == 0 for r in f.key_rank)
    A, Bk, Bv = f.storage()
    width = sum(f.key_rank) + f.value_rank
    x = synth.f32_to_bf16_bits(rng.standard_normal((B, L, d_model)).astype(np.float32))
    q = synth.f32_to_bf16_bits((rng.standard_normal((B, Hq, d)) * 3).astype(np.float32))
    layer = Layer(B, Hq, Hkv, d, L, f.key_rank, f.value_rank, qmode, 5e5, synth.DT_BF16,
                  synth.DT_F32, d_model=d_model)
    layer.append(to_dev(x), torch.zeros(B, dtype=torch.int32, device="cuda"), A_all=to_dev(A))
    ctx = np.full(B, L, np.int32)
    layer.decode(to_dev(q), to_dev(Bk), to_dev(Bv), to_dev(ctx))
    torch.cuda.synchronize()
    got = layer.out_float()
    lat_gpu = layer.app_ws[: B * L * width * 2].cpu().numpy().view(np.uint16).reshape(B, L, width)
    cfg = O.make_cfg(B, Hq, Hkv, d, L, f.key_rank, f.value_rank, qmode, 5e5, d_model=d_model)
    # latents: within 1 fp16 ulp of the fp64 product plus the fp32 summation bound
    lat_ref, _ = O.downproj(cfg, x[:, :64], True, A)          # the first 64 tokens of each
    g = lat_gpu[:, :64].reshape(-1, width).view(np.float16).astype(np.float64)
    r = lat_ref.view(np.float16).astype(np.float64)
    ulp = np.abs(np.spacing(r.astype(np.float16)).astype(np.float64))
    xf = (x[:, :64].reshape(-1, d_model).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    af = (A.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    acc_err = d_model * 2.0 ** -24 * (np.abs(xf) @ np.abs(af))
    assert np.all(np.abs(g - r) <= ulp + acc_err), f"latents: max diff {np.abs(g - r).max()}"
    # the cache: the oracle quantizes the GPU's latents, byte for byte
    cache = O.new_cache(cfg)
    O.append(cfg, cache, lat_gpu, [0] * B)
    assert np.array_equal(layer.cache.cpu().numpy(), cache)
    ref, _ = O.decode_attn(cfg, cache, q, True, Bk, Bv, ctx)
    e, s = assert_close(got, ref, "factorized decode", synth.DT_F32)
    say(f"  every output within the bare bound: max err {e:.3e}, max |o| {s:.3e}")
