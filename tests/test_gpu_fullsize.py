"""GPU parity at the benchmark sizes, in the launch configuration bench.py times.

Every workload at its full size: the packed cache byte for byte and every attention output
element against the fp64 oracle, once with the workload's 16-bit output (tolerance widened
by half an ulp of that type) and once with an fp32 output at the bare 2e-3 + 1e-3 |o|
bound.  Each case prints the split-kernel instance and the steps per split it reached, so
that a multi-step split is shown to have run.
"""
import math

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_08382_amd import synth

from _helpers import assert_close, oracle_cfg, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _dev(a):
    from paper_2606_08382_amd.device import to_dev
    return to_dev(a)


def _fill(w, inp, chunk=32768):
    """A layer of the workload's shape with every sequence's latents appended at row 0."""
    from paper_2606_08382_amd.device import Layer
    layer = Layer(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.ctx, inp.key_rank,
                  w.value_rank, w.qmode, w.rope_theta, w.q_dtype, w.out_dtype)
    pos = torch.zeros(w.batch, dtype=torch.int32, device="cuda")
    for t0 in range(0, inp.latents.shape[1], chunk):
        layer.append(_dev(np.ascontiguousarray(inp.latents[:, t0:t0 + chunk])), pos + t0)
    return layer


def _decode_both(w, inp, layer):
    """Outputs of one decode step with the workload's output type and with fp32, on the
    same cache (a second plan of the same layout)."""
    from paper_2606_08382_amd import starkv as S
    q, Bk, Bv, ctx = _dev(inp.q), _dev(inp.Bk), _dev(inp.Bv), _dev(inp.ctx_len)
    layer.decode(q, Bk, Bv, ctx)
    cfg32 = S.make_config(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.ctx, inp.key_rank,
                          w.value_rank, w.qmode, w.rope_theta, q_dtype=w.q_dtype,
                          out_dtype=S.DT_F32)
    plan32 = S.starkv_plan_create(cfg32)
    out32 = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    S.starkv_decode_attn(plan32, layer.cache, q, Bk, Bv, ctx, w.ctx, out32, layer.dec_ws)
    torch.cuda.synchronize()
    return layer.out_float(), out32.cpu().double().numpy()


def _describe(layer, ctx_len, max_ctx):
    from paper_2606_08382_amd import starkv as S
    plan = S.split_plan(S.starkv_decode_describe(layer.plan, max_ctx), ctx_len)
    say(f"  split kernel {plan['instance']}: {plan['split_tokens']} tokens "
        f"({plan['steps_per_split']} steps) per split, {plan['items']} work items")
    return plan


def _check_case(w, inp, what):
    say(f"{what}: {w.name} B={w.batch} ctx={w.ctx} ranks={inp.key_rank} r_v={w.value_rank} "
        f"qmode={w.qmode} lengths {int(inp.ctx_len.min())}..{int(inp.ctx_len.max())}")
    layer = _fill(w, inp)
    plan = _describe(layer, inp.ctx_len, w.ctx)
    got16, got32 = _decode_both(w, inp, layer)
    cfg = oracle_cfg(w, inp)
    cache = O.new_cache(cfg)
    O.append(cfg, cache, inp.latents, [0] * w.batch)
    diff = np.count_nonzero(layer.cache.cpu().numpy() != cache)
    assert diff == 0, f"{diff} cache bytes differ"
    ref, nt = O.decode_attn(cfg, cache, inp.q, w.q_dtype == synth.DT_BF16, inp.Bk, inp.Bv,
                            inp.ctx_len)
    e16, s = assert_close(got16, ref, f"{w.name} 16-bit output", w.out_dtype)
    e32, _ = assert_close(got32, ref, f"{w.name} fp32 output", synth.DT_F32)
    say(f"  all {ref.size} outputs: max err {e16:.3e} (16-bit), {e32:.3e} (fp32), "
        f"max |o| {s:.3e}; oracle on {nt} threads")
    return layer, plan, ref, cache


@pytest.mark.parametrize("name", ["c2", "c3", "c3q", "c4", "c5", "c5q"])
def test_full_size_every_output(name):
    """The workload at full size, every (sequence, query head) output: C2 4 x 32K int4, C3
    4 x 128K int8/int4, C3q the 4/3-bit quantizer, C4 32 ragged 2K-16K int4 (the device plan
    over ragged lengths), C5 2 x 64K with 64 query heads and r_v = 384, C5q its 4/3-bit
    variant (a value outlier region ending inside a wave's tiles)."""
    w = synth.WORKLOADS[name]
    inp = synth.generate(w)
    _, plan, _, _ = _check_case(w, inp, "full size")
    assert plan["steps_per_split"] > 1


def _plant_needles(inp, w, positions, key_gain, q_gain):
    """Scale the key latents of the given (sequence, token) positions by key_gain and every
    query by q_gain (the peaked workloads' recipe, at chosen positions)."""
    ksum = sum(inp.key_rank)
    for b, t in positions:
        v = inp.latents[b, t, :ksum].view(np.float16).astype(np.float32) * key_gain
        inp.latents[b, t, :ksum] = np.ascontiguousarray(v.astype(np.float16)).view(np.uint16)
    qf = synth.to_bits(_q_float(inp, w) * q_gain, w.q_dtype)
    inp.q[...] = qf


def _q_float(inp, w):
    if w.q_dtype == synth.DT_BF16:
        return (inp.q.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return inp.q.view(np.float16).astype(np.float64)


def _score_log2(cfg, cache, inp, w, b, i, t):
    """Exact score of query head i against token t, in log2 units (the kernels' scale)."""
    g = i * w.n_kv_heads // w.n_q_heads
    k = O.reconstruct_key(cfg, cache, inp.Bk, b, g, t, True)
    return float(_q_float(inp, w)[b, i] @ k) / math.sqrt(w.head_dim) * math.log2(math.e)


def test_full_size_late_needles_raise_the_softmax_reference():
    """C3 at full size (2048-token splits of 16 steps) with needle tokens at offset 1500 of
    their split, i.e. in step 11: steps 0-10 set the split's shared softmax reference from
    ordinary scores, and the needle's score exceeds it by far more than the 8 log2 units the
    split kernel tolerates, so the kernel must raise the reference in a late step and
    rescale value accumulators and sums that are already non-zero.  The test checks that
    precondition exactly (needle score minus the largest score of all earlier tokens of its
    split, an upper bound of the reference the kernel holds by then), then every output
    against the oracle with an fp32 output at the bare bound."""
    w = synth.WORKLOADS["c3"]
    inp = synth.generate(w)
    rng = np.random.default_rng(77)
    S = 2048
    pos = [(b, int(k) * S + 1500) for b in range(w.batch)
           for k in rng.choice(w.ctx // S, size=3, replace=False)]
    _plant_needles(inp, w, pos, key_gain=16.0, q_gain=4.0)
    layer, plan, ref, cache = _check_case(w, inp, "late needles")
    assert plan["split_tokens"] == S
    cfg = oracle_cfg(w, inp)
    best = -np.inf
    for b, t in pos[:3]:
        s0 = (t // S) * S                                # the split's first token
        i = max(range(w.n_q_heads), key=lambda h: _score_log2(cfg, cache, inp, w, b, h, t))
        needle = _score_log2(cfg, cache, inp, w, b, i, t)
        before = max(_score_log2(cfg, cache, inp, w, b, i, u) for u in range(s0, t))
        best = max(best, needle - before)
    say(f"  needle score above the largest earlier score of its split: {best:.1f} log2 units")
    assert best > 8.0


@pytest.mark.parametrize("name", ["c4", "c2"])
def test_full_size_peaked(name):
    """Peaked variants at full size (q x 4, four needles per sequence with key latents x 8):
    C4's ragged device plan and C2's int4 path with attention concentrated on a few tokens."""
    w = synth.WORKLOADS[name]
    inp = synth.generate(w, peaked=1)
    _check_case(w, inp, "peaked full size")
