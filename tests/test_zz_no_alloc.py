"""The no-allocation decode entry point (fixed device scratch array) against the
workspace entry point: the same kernels on the same inputs, so the outputs must be
identical, on two calls in a row, the second with a smaller problem."""
import numpy as np
import pytest

from paper_2606_08382_amd import synth

from _helpers import say, small

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _case(name, ctx, batch, peaked, out_dtype=None):
    from paper_2606_08382_amd import starkv as S
    from paper_2606_08382_amd.device import Layer, to_dev
    w = small(name, ctx, batch)
    if out_dtype is not None:
        w = w.with_(out_dtype=out_dtype)
    inp = synth.generate(w, peaked=peaked)
    say(f"no-alloc decode {w.name} B={w.batch} ranks={inp.key_rank} peaked={peaked}")
    layer = Layer(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.ctx, inp.key_rank,
                  w.value_rank, w.qmode, w.rope_theta, w.q_dtype, w.out_dtype)
    layer.append(to_dev(inp.latents), torch.zeros(w.batch, dtype=torch.int32, device="cuda"))
    q, Bk, Bv, ctx_len = to_dev(inp.q), to_dev(inp.Bk), to_dev(inp.Bv), to_dev(inp.ctx_len)
    ref = layer.decode(q, Bk, Bv, ctx_len).clone()
    got = torch.full_like(ref, 7)
    S.starkv_decode_attn_noalloc(layer.plan, layer.cache, q, Bk, Bv, ctx_len, w.ctx, got)
    torch.cuda.synchronize()
    assert torch.equal(got, ref), "no-alloc output differs from the workspace entry point"
    return got


def test_noalloc_matches_workspace_entry_point_twice_second_smaller():
    _case("c3", 3000, 4, 1)
    _case("c3q", 700, 2, 2, synth.DT_F32)


def test_noalloc_refuses_a_workspace_beyond_the_scratch_array():
    from paper_2606_08382_amd import starkv as S
    big = S.make_config(1024, 32, 8, 128, 8192, [16] * 8, 256, S.Q_INT4, 5e5)
    plan = S.starkv_plan_create(big)
    assert S.starkv_decode_workspace_bytes(plan, 8192) > 32 << 20
    with pytest.raises(S.StarkvError) as e:
        S.starkv_decode_attn_noalloc(plan, 256, 256, 256, 256, 256, 8192, 256)
    assert e.value.status == 4
