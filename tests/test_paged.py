"""Paged cache on the CPU: plan validation, the pool layout against the oracle's, and the
host-side page allocator.  No kernel runs here."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_08382_amd import starkv as S
from paper_2606_08382_amd import synth
from paper_2606_08382_amd.device import PagePool

torch = pytest.importorskip("torch")

FAKE = 1 << 40          # never dereferenced by plan creation


def _cfg(**kw):
    base = dict(batch=3, n_q_heads=8, n_kv_heads=2, head_dim=128, capacity=1000,
                key_rank=[32, 48], value_rank=64, qmode=S.Q_MIX8_4, rope_theta=1e4,
                page_tokens=256, n_pages=10, block_table=FAKE)
    base.update(kw)
    return S.make_config(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(page_tokens=64), 1), (dict(page_tokens=384), 1), (dict(page_tokens=16384), 1),
    (dict(n_pages=0), 1), (dict(block_table=None), 1), (dict(block_table=FAKE + 2), 5),
    (dict(page_tokens=8192, n_pages=1 << 18), 2),
])
def test_paged_plan_rejects_bad_configs(kw, status):
    with pytest.raises(S.StarkvError) as ei:
        S.starkv_plan_create(_cfg(**kw))
    assert ei.value.status == status


@pytest.mark.parametrize("name,P,n_pages", [("c3", 128, 7), ("c4", 256, 40), ("c5q", 8192, 3),
                                            ("c1", 512, 1)])
def test_paged_layout_matches_oracle(name, P, n_pages):
    w = synth.WORKLOADS[name]
    inp = synth.generate(synth.shrink(w, ctx=64, batch=w.batch), with_latents=False)
    cap = 3000
    plan = S.starkv_plan_create(S.make_config(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim,
                                              cap, inp.key_rank, w.value_rank, w.qmode,
                                              w.rope_theta, page_tokens=P, n_pages=n_pages,
                                              block_table=FAKE))
    L = S.starkv_cache_layout(plan)
    per_seq = -(-cap // P)
    oc = O.make_cfg(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, cap, inp.key_rank,
                    w.value_rank, w.qmode, w.rope_theta, page_tokens=P, n_pages=n_pages,
                    table=np.zeros((w.batch, per_seq), np.int32))
    assert L.rows == n_pages * P and L.page_tokens == P and L.pages_per_sequence == per_seq
    assert L.total_bytes == O.cache_bytes(oc) == S.starkv_cache_bytes(plan)
    for g in range(w.n_kv_heads):
        assert L.key_code_offset[g] == O.plane_offset(oc, 0, g)
        assert L.key_meta_offset[g] == O.plane_offset(oc, 1, g)
    assert L.value_code_offset == O.plane_offset(oc, 2)
    assert L.value_meta_offset == O.plane_offset(oc, 3)
    # contiguous plans report their rows too
    flat = S.starkv_cache_layout(S.starkv_plan_create(S.make_config(
        w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, cap, inp.key_rank, w.value_rank,
        w.qmode, w.rope_theta)))
    assert flat.rows == w.batch * flat.padded_capacity and flat.page_tokens == 0


def test_page_pool_hands_out_and_reuses_pages():
    pool = PagePool(n_pages=6, page_tokens=128, batch=3, capacity=500, device="cpu")
    assert pool.per_seq == 4
    pool.ensure(0, 1)
    pool.ensure(1, 129)
    assert pool.host[0].tolist() == [0, -1, -1, -1] and pool.host[1].tolist() == [1, 2, -1, -1]
    pool.ensure(0, 300)                       # grows in place, keeps its first page
    assert pool.host[0].tolist() == [0, 3, 4, -1] and pool.pages_in_use() == 5
    with pytest.raises(ValueError):
        pool.ensure(2, 501)                   # beyond the capacity
    pool.ensure(2, 128)
    with pytest.raises(MemoryError):
        pool.ensure(2, 129)                   # the pool is exhausted
    pool.release(1)
    assert pool.pages_in_use() == 4 and sorted(pool.free) == [1, 2]
    pool.ensure(2, 256)
    assert pool.host[2, :2].tolist() == [5, 2]            # the most recently freed page first
    used = pool.host[pool.host >= 0]
    assert len(set(used.tolist())) == used.size           # no page is handed out twice
    pool.sync()
    assert np.array_equal(pool.table.numpy(), pool.host)


def test_page_pool_shuffled_free_list_is_a_permutation():
    pool = PagePool(n_pages=9, page_tokens=256, batch=2, capacity=1024, device="cpu",
                    rng=np.random.default_rng(3))
    pool.ensure(0, 1024)
    pool.ensure(1, 1024)
    used = pool.host.reshape(-1)
    assert sorted(used.tolist()) == sorted(set(used.tolist())) and len(pool.free) == 1
    assert used.tolist() != list(range(8))                # scattered, not in order
