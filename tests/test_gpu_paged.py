"""Paged cache on the GPU (continuous batching): the pool bytes bit-exact against the oracle
fed the same block table, decode outputs within tolerance, pages handed out and taken back
while a captured decode step is replayed."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2606_08382_amd import synth

from _helpers import assert_close, say, small

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _dev(a):
    from paper_2606_08382_amd.device import to_dev
    return to_dev(a)


def _layer(w, inp, P, n_pages, rng):
    from paper_2606_08382_amd.device import Layer
    return Layer(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.ctx, inp.key_rank,
                 w.value_rank, w.qmode, w.rope_theta, w.q_dtype, w.out_dtype,
                 page_tokens=P, n_pages=n_pages, page_rng=rng)


def _ocfg(w, inp, layer):
    """The oracle's view of the pool with the block table as it is now (a copy)."""
    pool = layer.pool
    return O.make_cfg(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.ctx, inp.key_rank,
                      w.value_rank, w.qmode, w.rope_theta, page_tokens=pool.page_tokens,
                      n_pages=pool.n_pages, table=pool.host.copy())


@pytest.mark.parametrize("name,ctx,batch,P,ragged", [
    ("c3", 1100, 2, 128, None), ("c4", 900, 6, 256, (1, 900)), ("c3q", 700, 2, 512, None),
    ("c1", 1024, None, 128, None), ("c5", 600, 2, 8192, None), ("c2", 1500, 3, 1024, (200, 1500)),
    ("c1", 300, 70, 128, (5, 300))])
def test_paged_pool_and_decode_match_oracle(name, ctx, batch, P, ragged):
    """Sequences scattered over a shuffled pool with spare pages; appends in chunks that cross
    page boundaries; the whole pool bit-exact, decode and the absorbed output in tolerance.
    More than 64 sequences take the per-sequence split grid instead of the work plan."""
    w = small(name, ctx, batch, ragged=ragged)
    inp = synth.generate(w, peaked=1)
    rng = np.random.default_rng(100 + P)
    ctx_len = inp.ctx_len
    n_pages = int(sum(-(-int(L) // P) for L in ctx_len)) + 5
    say(f"paged {w.name} B={w.batch} P={P} pages={n_pages} ctx={ctx_len.tolist()}")
    layer = _layer(w, inp, P, n_pages, rng)
    for b in range(w.batch):
        layer.pool.ensure(b, int(ctx_len[b]))
    layer.pool.sync()
    cfg = _ocfg(w, inp, layer)
    cache = O.new_cache(cfg)
    start, L = 0, inp.latents.shape[1]
    for n in (1, 100, 300, L):
        n = min(n, L - start)
        if n <= 0:
            break
        chunk = np.ascontiguousarray(inp.latents[:, start:start + n])
        pos = np.full(w.batch, start, np.int32)
        layer.append(_dev(chunk), _dev(pos))
        O.append(cfg, cache, chunk, pos)
        start += n
    torch.cuda.synchronize()
    got = layer.cache.cpu().numpy()
    diff = np.nonzero(got != cache)[0]
    assert diff.size == 0, f"{diff.size} pool bytes differ, first at {diff[:6]}"
    out = layer.decode(_dev(inp.q), _dev(inp.Bk), _dev(inp.Bv), _dev(ctx_len))
    torch.cuda.synchronize()
    ref, _ = O.decode_attn(cfg, cache, inp.q, w.q_dtype == synth.DT_BF16, inp.Bk, inp.Bv, ctx_len)
    e, s = assert_close(layer.out_float(out), ref, w.name, w.out_dtype)
    say(f"  pool bit-exact; max err {e:.3e} |o| {s:.3e}")
    W = synth.absorbed_weights(w, 96)
    y = layer.decode_absorbed(_dev(inp.q), _dev(inp.Bk), _dev(W), _dev(ctx_len))
    yref, _ = O.decode_attn_absorbed(cfg, cache, inp.q, w.q_dtype == synth.DT_BF16, inp.Bk, W,
                                     ctx_len)
    assert_close(layer.out_float(y), yref, w.name + " absorbed", w.out_dtype)


def test_continuous_batching_with_a_replayed_decode_step():
    """Four sequence slots over a shared pool: prefill, then decode steps replayed from one
    captured graph (append one token per sequence + decode) while the host hands out pages
    as sequences grow, retires a sequence, frees its pages and starts a new one in its slot
    on the recycled pages.  The oracle replays every append with the block table as it was
    at that step; pool bytes and the final outputs are compared."""
    w = small("c3", ctx=1024, batch=4)
    inp = synth.generate(w)
    P = 128
    rng = np.random.default_rng(9)
    layer = _layer(w, inp, P, 20, rng)
    pool = layer.pool
    width = inp.width
    lens = np.array([300, 129, 0, 700], np.int32)
    say(f"continuous batching: pool {pool.n_pages} pages, prefill {lens.tolist()}")
    cache = O.new_cache(_ocfg(w, inp, layer))

    def prefill(b, n, seed):
        lat = synth.to_bits(np.random.default_rng(seed).standard_normal((w.batch, n, width)) * 0.5,
                            synth.DT_F16)
        pool.ensure(b, n)
        pool.sync()
        pos = np.zeros(w.batch, np.int32)
        pos[np.arange(w.batch) != b] = 1 << 30          # other sequences: rows dropped
        layer.append(_dev(lat), _dev(pos))
        O.append(_ocfg(w, inp, layer), cache, lat, pos)

    for b in range(w.batch):
        if lens[b]:
            prefill(b, int(lens[b]), 50 + b)
    # the decode step, captured once on static inputs
    q = _dev(inp.q)
    Bk, Bv = _dev(inp.Bk), _dev(inp.Bv)
    lat1 = _dev(np.zeros((w.batch, 1, width), np.uint16))
    pos = _dev(np.zeros(w.batch, np.int32))
    ctx = _dev(np.zeros(w.batch, np.int32))
    layer.append(lat1, _dev(np.full(w.batch, 1 << 30, np.int32)))   # warm-up, drops every row
    layer.decode(q, Bk, Bv, ctx)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        layer.append(lat1, pos)
        layer.decode(q, Bk, Bv, ctx)
    active = lens > 0
    step_rng = np.random.default_rng(77)
    for step in range(40):
        if step == 15:                                  # slot 1 retires, slot 2 starts
            pool.release(1)
            lens[1] = 0
            active[1] = False
            prefill(2, 200, 90)
            lens[2], active[2] = 200, True
        if step == 25:                                  # a new sequence in slot 1
            prefill(1, 250, 91)
            lens[1], active[1] = 250, True
        lat = synth.to_bits(step_rng.standard_normal((w.batch, 1, width)) * 0.5, synth.DT_F16)
        p = np.where(active, lens, 1 << 30).astype(np.int32)
        for b in np.nonzero(active)[0]:
            pool.ensure(int(b), int(lens[b]) + 1)
        pool.sync()
        lens = lens + active.astype(np.int32)
        lat1.copy_(_dev(lat))
        pos.copy_(_dev(p))
        ctx.copy_(_dev(lens))
        q.copy_(_dev(synth.to_bits(step_rng.standard_normal(inp.q.shape), w.q_dtype)))
        g.replay()
        O.append(_ocfg(w, inp, layer), cache, lat, p)
    torch.cuda.synchronize()
    got = layer.cache.cpu().numpy()
    diff = np.nonzero(got != cache)[0]
    assert diff.size == 0, f"{diff.size} pool bytes differ, first at {diff[:6]}"
    assert pool.pages_in_use() == sum(-(-int(L) // P) for L in lens)
    q_last = q.cpu().numpy().view(np.uint16)
    ref, _ = O.decode_attn(_ocfg(w, inp, layer), cache, q_last, True, inp.Bk, inp.Bv, lens)
    e, s = assert_close(layer.out_float(), ref, "continuous batching", w.out_dtype)
    say(f"  lengths {lens.tolist()}, pool bit-exact, max err {e:.3e} |o| {s:.3e}")
