"""Host-side checks of the C ABI (no GPU needed: nothing here launches a kernel).

The library must load, export every function the public header declares,
validate its arguments before any launch, and describe the same cache layout
as the oracle's independent implementation of the format.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_08382_amd import starkv as S
from paper_2606_08382_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    text = open(os.path.join(ROOT, "include", "starkv.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(starkv_[a-z_]+)\s*\(", text)))


def test_library_exports_every_header_function():
    lib = S.lib()
    names = _header_functions()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(S.EXPORTS) == names


def test_status_strings():
    for st in range(7):
        assert S.starkv_status_string(st)
    assert S.starkv_status_string(99) == "unknown status"


def _cfg(**kw):
    base = dict(batch=2, n_q_heads=8, n_kv_heads=2, head_dim=128, capacity=1000,
                key_rank=[32, 48], value_rank=64, qmode=S.Q_MIX8_4, rope_theta=1e4)
    base.update(kw)
    return S.make_config(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(batch=0), 1), (dict(n_q_heads=7), 1), (dict(key_rank=[24, 32]), 1),
    (dict(key_rank=[32, 144]), 1), (dict(value_rank=40), 1), (dict(value_rank=272), 1),
    (dict(qmode=7), 1), (dict(qmode=4), 1), (dict(rope_theta=1.0), 1), (dict(capacity=0), 1),
    (dict(head_dim=96), 2), (dict(group_size=64), 2), (dict(n_q_heads=96, n_kv_heads=2), 2),
    (dict(n_q_heads=6, n_kv_heads=2), 2), (dict(d_model=100), 2),
    (dict(q_dtype=S.DT_F32), 1), (dict(out_dtype=3), 1),
])
def test_plan_create_rejects_bad_configs(kw, status):
    with pytest.raises(S.StarkvError) as ei:
        S.starkv_plan_create(_cfg(**kw))
    assert ei.value.status == status
    assert S.starkv_last_error()


def test_entry_points_validate_before_launch():
    plan = S.starkv_plan_create(_cfg())
    need = S.starkv_decode_workspace_bytes(plan, 1000)
    fake = 1 << 40          # never dereferenced: every call below fails validation first
    with pytest.raises(S.StarkvError) as ei:
        S.starkv_decode_attn(plan, fake, fake, fake, fake, fake, 1001, fake, fake, need)
    assert ei.value.status == 3                       # max_ctx > capacity
    with pytest.raises(S.StarkvError) as ei:
        S.starkv_decode_attn(plan, fake, fake, fake, fake, fake, 1000, fake, fake, need - 1)
    assert ei.value.status == 4                       # workspace too small
    with pytest.raises(S.StarkvError) as ei:
        S.starkv_decode_attn(plan, fake + 8, fake, fake, fake, fake, 1000, fake, fake, need)
    assert ei.value.status == 5                       # cache misaligned
    with pytest.raises(S.StarkvError) as ei:
        S.starkv_decode_attn(plan, fake, fake, fake, fake, None, 1000, fake, fake, need)
    assert ei.value.status == 1                       # NULL ctx_len
    with pytest.raises(S.StarkvError) as ei:
        S.starkv_decode_attn(plan, fake, fake, fake, fake, fake, 0, fake, fake, need)
    assert ei.value.status == 1
    with pytest.raises(S.StarkvError) as ei:            # B_v misaligned: caught before the split
        S.starkv_decode_attn(plan, fake, fake, fake, fake + 2, fake, 1000, fake, fake, need)
    assert ei.value.status == 5
    with pytest.raises(S.StarkvError) as ei:
        S.starkv_decode_combine(plan, fake, fake, None, fake, fake, 1000, fake, fake, need)
    assert ei.value.status == 1                       # combine re-reads the keys: B_k required
    with pytest.raises(S.StarkvError) as ei:
        S.starkv_decode_combine(plan, fake, fake, fake, fake, fake, 1000, fake + 4, fake, need)
    assert ei.value.status == 5                       # out misaligned
    with pytest.raises(S.StarkvError) as ei:
        S.starkv_decode_split(plan, fake, fake + 2, fake, fake, 1000, fake, need)
    assert ei.value.status == 5                       # q misaligned
    with pytest.raises(S.StarkvError) as ei:
        S.starkv_append(plan, fake, fake, None, fake, 0, None, 0)
    assert ei.value.status == 1                       # n_new < 1
    with pytest.raises(S.StarkvError) as ei:
        S.starkv_append(plan, fake + 4, fake, None, fake, 1, None, 0)
    assert ei.value.status == 5
    # absorbed output: B_v is not needed, W_abs, d_out and out are
    S.starkv_decode_attn_absorbed  # exported (above); argument errors come first
    for args, status in [((fake, fake, fake, None, 64, fake, 1000, fake), 1),   # W_abs NULL
                         ((fake, fake, fake, fake, 0, fake, 1000, fake), 1),    # d_out < 1
                         ((fake, fake, fake, fake, 64, fake, 1000, None), 1),   # out NULL
                         ((fake, fake, fake, fake + 8, 64, fake, 1000, fake), 5),
                         ((fake, fake, fake, fake, 64, fake, 1000, fake + 2), 5),
                         ((fake, fake, fake, fake, 64, fake, 1001, fake), 3)]:
        for fn in (S.starkv_decode_attn_absorbed, S.starkv_decode_combine_absorbed):
            with pytest.raises(S.StarkvError) as ei:
                fn(plan, *args, fake, need)
            assert ei.value.status == status, (fn.__name__, args)
    with pytest.raises(S.StarkvError) as ei:
        S.starkv_decode_attn_absorbed(plan, fake, fake, fake, fake, 64, fake, 1000, fake, fake,
                                      need - 1)
    assert ei.value.status == 4
    hid = S.starkv_plan_create(_cfg(d_model=256))
    with pytest.raises(S.StarkvError) as ei:
        S.starkv_append(hid, fake, fake, fake, fake, 3, fake, 10)
    assert ei.value.status == 4                       # append workspace too small
    with pytest.raises(S.StarkvError) as ei:
        S.starkv_append(hid, fake, fake, None, fake, 3, fake, 1 << 30)
    assert ei.value.status == 1                       # A_all missing


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5", "c3q", "c5q"])
def test_layout_matches_oracle_format(name):
    w = synth.WORKLOADS[name]
    inp = synth.generate(synth.shrink(w, ctx=64, batch=w.batch), with_latents=False)
    for cap in (1, 255, 300, w.ctx):
        plan = S.starkv_plan_create(S.make_config(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim,
                                                  cap, inp.key_rank, w.value_rank, w.qmode,
                                                  w.rope_theta))
        L = S.starkv_cache_layout(plan)
        oc = O.make_cfg(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, cap, inp.key_rank,
                        w.value_rank, w.qmode, w.rope_theta)
        assert L.total_bytes == O.cache_bytes(oc) == S.starkv_cache_bytes(plan)
        for g in range(w.n_kv_heads):
            assert L.key_code_offset[g] == O.plane_offset(oc, 0, g)
            assert L.key_meta_offset[g] == O.plane_offset(oc, 1, g)
            assert L.key_outlier_channels[g] == O.outlier_channels(w.qmode, inp.key_rank[g])
        assert L.value_code_offset == O.plane_offset(oc, 2)
        assert L.value_meta_offset == O.plane_offset(oc, 3)
        assert L.padded_capacity % 256 == 0 and L.padded_capacity >= cap


def test_bytes_per_token_of_the_128k_workload():
    w = synth.WORKLOADS["c3"]
    inp = synth.generate(synth.shrink(w, ctx=64), with_latents=False)
    plan = S.starkv_plan_create(S.make_config(4, 32, 8, 128, 131072, inp.key_rank, 256,
                                              S.Q_MIX8_4, 5e5))
    assert S.starkv_cache_bytes(plan) == 424 * 4 * 131072
    # workspace of the split partials and rescoring candidates stays a few percent of
    # the stream: 256 items x 32 heads x (264 floats + 64 candidates of 8 bytes), the
    # absorbed output's latents, and the per-sequence work plan (one 256-byte block)
    ws = S.starkv_decode_workspace_bytes(plan, 131072)
    assert ws == 256 * 32 * (264 * 4 + 64 * 8) + 2 * 4 * 32 * 256 * 2 + 256
    assert ws < 0.06 * S.starkv_cache_bytes(plan)
    assert S.starkv_decode_splits(plan, 131072) * S.starkv_decode_split_tokens(plan, 131072) >= 131072


@pytest.mark.parametrize("batch,max_ctx,splits_max", [(1, 524288, 256), (1, 1000, 8),
                                                      (2, 131072, 128), (70, 100000, 256),
                                                      (200, 524288, 256)])
def test_split_plan_limits(batch, max_ctx, splits_max):
    """Every split at most 8192 tokens, at most 256 splits per sequence, the splits cover
    max_ctx; larger batches (the per-sequence split grid) also at long contexts."""
    w = synth.WORKLOADS["c3"]
    inp = synth.generate(synth.shrink(w, ctx=64), with_latents=False)
    plan = S.starkv_plan_create(S.make_config(batch, 32, 8, 128, max_ctx, inp.key_rank, 256,
                                              S.Q_MIX8_4, 5e5))
    n, t = S.starkv_decode_splits(plan, max_ctx), S.starkv_decode_split_tokens(plan, max_ctx)
    assert t % 128 == 0 and 128 <= t <= 8192
    assert n * t >= max_ctx and (n - 1) * t < max_ctx and n <= splits_max
    assert S.starkv_decode_workspace_bytes(plan, max_ctx) > 0


def test_workspace_sizes():
    plan = S.starkv_plan_create(_cfg(d_model=256))
    assert S.starkv_append_workspace_bytes(plan, 5) >= 2 * 5 * (80 + 64) * 2
    assert S.starkv_decode_workspace_bytes(plan, 1) > 0
    assert S.starkv_decode_workspace_bytes(plan, 0) == 0
    plan0 = S.starkv_plan_create(_cfg())
    assert S.starkv_append_workspace_bytes(plan0, 5) == 0


def test_bytes_per_token_of_the_128k_workload_with_the_paper_quantizer():
    # C3's layer at 4/3 bits (outlier channels r_out = 8 for ranks 16..48, 48 of the 256
    # value channels): key codes 2*(4+3) + 4*(4+9) + 2*(4+15) = 104 B, key meta
    # (2*2 + 4*2 + 2*3 groups) * 4 = 72 B, value codes 48/2 + 208*3/8 = 102 B, value meta
    # (2+7)*4 = 36 B -> 314 B per token (424 B at 8/4 bits)
    w = synth.WORKLOADS["c3q"]
    inp = synth.generate(synth.shrink(w, ctx=64), with_latents=False)
    plan = S.starkv_plan_create(S.make_config(4, 32, 8, 128, 131072, inp.key_rank, 256,
                                              S.Q_MIX4_3, 5e5))
    assert S.starkv_cache_bytes(plan) == 314 * 4 * 131072


def test_read_stream_validates_before_launch():
    """The read-stream measurement aid refuses bad arguments before any launch."""
    lib = S.lib()
    sink = ctypes.create_string_buffer(64)   # host memory: only the checks read the pointers
    addr = ctypes.addressof(sink)
    cases = [
        (None, 1024, 1, addr, 64, 1),        # NULL src
        (4096, 0, 1, addr, 64, 1),           # zero bytes
        (4096, 1000, 1, addr, 64, 1),        # not a multiple of 16
        (4096, 1024, -1, addr, 64, 1),       # workgroups out of range
        (4096, 1024, 8, addr, 64, 1),        # sink too small for 8 workgroups
        (4104, 1024, 1, addr, 64, 5),        # src not 16-byte aligned
    ]
    for src, n, wg, snk, snk_bytes, status in cases:
        st = lib.starkv_read_stream(src, n, wg, snk, snk_bytes, None)
        assert st == status, (src, n, wg, st, S.starkv_last_error())
