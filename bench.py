"""Decode-attention throughput on one MI355X at the Llama-3.1-8B 128K workload.

One step = starkv_append of one new token per sequence from bf16 hidden states
(down-projection + quantize/pack) followed by starkv_decode_attn over the whole
context (split pass + combine pass), on one layer's cache.  The timed steps
replay the step captured in a HIP graph (one per layer cache); per-kernel times
come from an eager pass with HIP events.  Five layer caches
(> 1 GB together) are used in rotation so the 256 MB last-level cache cannot
serve the latent stream.  Inputs are seeded synthetic arrays of the workload's
shape, resident in HBM before timing starts.

Prints one JSON line; per-kernel times are measured with HIP events on the
stream the kernels run on.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0   # dense fp16 matrix peak
COPY_BYTES = 256 << 20           # the plain device-to-device copy timed beside the path
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "decode_split_c3_traffic.json")
SQ_SUMMARY = os.path.join(ROOT, "profiles", "decode_split_c3_sq_counters.json")
SPLIT_SOURCE = os.path.join(ROOT, "paper_2606_08382_amd", "csrc", "decode.hip")


_DT_NAMES = {0: "f16", 1: "bf16", 2: "f32"}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_baseline(w, inp, sample_ctx: int, n_seq: int = 4):
    """The fp64 oracle on the first n_seq sequences (all heads) over the first sample_ctx
    tokens (about 10-30 s of CPU work at the 128K layer), scaled linearly to the full
    context when the sample is shorter."""
    from oracle import oracle as O
    from paper_2606_08382_amd import synth
    n_seq = min(n_seq, w.batch)
    cfg = O.make_cfg(n_seq, w.n_q_heads, w.n_kv_heads, w.head_dim, sample_ctx, inp.key_rank,
                     w.value_rank, w.qmode, w.rope_theta)
    cache = O.new_cache(cfg)
    O.append(cfg, cache, np.ascontiguousarray(inp.latents[:n_seq, :sample_ctx]), [0] * n_seq)
    t0 = time.perf_counter()
    _, threads = O.decode_attn(cfg, cache, np.ascontiguousarray(inp.q[:n_seq]),
                               w.q_dtype == synth.DT_BF16, inp.Bk,
                               inp.Bv, np.full(n_seq, sample_ctx, np.int32))
    dt = time.perf_counter() - t0
    full = dt * (w.ctx / sample_ctx)            # seconds for n_seq decode tokens at full context
    span = (f"all {w.ctx} tokens" if sample_ctx == w.ctx else
            f"the first {sample_ctx} of {w.ctx} tokens (scaled linearly in context length)")
    return {"value": n_seq / full, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": (f"{n_seq} decode tokens: {n_seq} sequences x {w.n_q_heads} query heads "
                       f"over {span} took {dt:.2f} s")}


def _counter_summary(path, workload_name):
    """A committed rocprofv3 counter summary of the split kernel, or None when it is missing,
    covers another workload, or the kernel source has changed since the counters were taken."""
    import hashlib
    try:
        with open(path) as f:
            t = json.load(f)
        with open(SPLIT_SOURCE, "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()
    except (OSError, ValueError):
        return None
    if t.get("source_sha256") != sha or t.get("workload") != workload_name:
        return None
    return t


def measured_traffic(workload_name):
    """HBM bytes per split launch from the committed counter summary (FETCH_SIZE and
    WRITE_SIZE, each scaled by the same counter's reading for a copy of known size), or None."""
    t = _counter_summary(TRAFFIC_SUMMARY, workload_name)
    if t is None:
        return None, None
    return float(t["traffic_bytes_per_launch"]), t


def copy_stream(torch, stream, reps=5):
    """Bandwidth of a plain device-to-device copy of COPY_BYTES (read + write), for context."""
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda")
    src.fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(reps)]
    for a, b in evs:
        a.record(stream)
        dst.copy_(src)
        b.record(stream)
    torch.cuda.synchronize()
    ms = float(np.mean([a.elapsed_time(b) for a, b in evs]))
    return {"bytes_read": COPY_BYTES, "bytes_written": COPY_BYTES, "us": ms * 1e3,
            "GBps": 2 * COPY_BYTES / (ms / 1e3) / 1e9}


def read_stream(torch, stream, n_bytes=1 << 30, reps=7):
    """Bandwidth of the plain HBM read stream (the library's hand-written read kernel:
    16-byte loads, sixteen in flight per lane, one word written per wave) over n_bytes, at a
    few grid sizes; the best median is the measured read ceiling."""
    from paper_2606_08382_amd import starkv as S
    x = torch.ones(n_bytes // 4, dtype=torch.float32, device="cuda")
    best = None
    for wg in (1024, 2048, 4096, 8192):
        sink = torch.empty(wg * 4, dtype=torch.int32, device="cuda")
        S.starkv_read_stream(x, n_bytes, sink, wg)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(reps)]
        for a, b in evs:
            a.record(stream)
            S.starkv_read_stream(x, n_bytes, sink, wg)
            b.record(stream)
        torch.cuda.synchronize()
        ms = float(np.median([a.elapsed_time(b) for a, b in evs]))
        r = {"bytes_read": n_bytes, "workgroups": wg, "us": ms * 1e3,
             "GBps": n_bytes / (ms / 1e3) / 1e9, "kernel": "starkv_read_stream"}
        if best is None or r["GBps"] > best["GBps"]:
            best = r
    del x
    return best


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="c3")
    ap.add_argument("--layers", type=int, default=5)
    ap.add_argument("--cpu-sample-ctx", type=int, default=0,
                    help="context tokens of the oracle sample (0: the full context)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true", help="time eager launches, not graph replays")
    ap.add_argument("--page-tokens", type=int, default=0,
                    help="paged cache: pool pages of this many tokens, handed out in shuffled "
                         "order (0: each sequence owns a contiguous run of rows)")
    ap.add_argument("--no-absorbed", action="store_true",
                    help="skip the step variant with the weight-absorbed output")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(decode attention would shard by sequence or by context range).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_08382_amd import starkv as S
    from paper_2606_08382_amd import synth
    from paper_2606_08382_amd.device import Layer, to_dev

    w = synth.WORKLOADS[args.workload]
    torch.cuda.set_device(0)
    log(f"generating {w.name}")
    inp = synth.generate(w, with_hidden=w.d_model > 0, n_hidden_tokens=1)
    B, L = w.batch, w.ctx
    layers = []
    lat_chunk = 16384
    P = args.page_tokens
    for li in range(args.layers):
        paged = {}
        if P:
            n_pages = int(sum(-(-int(x) // P) for x in inp.ctx_len))
            paged = dict(page_tokens=P, n_pages=n_pages, page_rng=np.random.default_rng(1000 + li))
        layer = Layer(B, w.n_q_heads, w.n_kv_heads, w.head_dim, L, inp.key_rank, w.value_rank,
                      w.qmode, w.rope_theta, w.q_dtype, w.out_dtype, d_model=w.d_model, **paged)
        if P:
            for b in range(B):
                layer.pool.ensure(b, int(inp.ctx_len[b]))
            layer.pool.sync()
        pos = torch.zeros(B, dtype=torch.int32, device="cuda")
        for t0 in range(0, L, lat_chunk):
            chunk = to_dev(np.ascontiguousarray(inp.latents[:, t0:t0 + lat_chunk]))
            # the caches are filled through a latent-input plan with the same layout
            S.starkv_append(_fill_plan(layer, w, inp), layer.cache, chunk, None, pos + t0,
                            chunk.shape[1], None, 0)
        layers.append(layer)
        log(f"layer {li} filled ({S.starkv_cache_bytes(layer.plan) / 1e6:.1f} MB)")
    torch.cuda.synchronize()
    q = to_dev(inp.q)
    Bk, Bv = to_dev(inp.Bk), to_dev(inp.Bv)
    ctx = to_dev(inp.ctx_len)
    x = to_dev(inp.x) if inp.x is not None else None
    A = to_dev(inp.A) if inp.A is not None else None
    pos_new = to_dev((inp.ctx_len - 1).astype(np.int32))
    stream = torch.cuda.current_stream()
    n_ev = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(n_ev)]

    def step(i, events=None):
        layer = layers[i % len(layers)]
        if events:
            events[0].record(stream)
        if x is not None:
            layer.append(x, pos_new, A_all=A)
        if events:
            events[1].record(stream)
        S.starkv_decode_split(layer.plan, layer.cache, q, Bk, ctx, L, layer.dec_ws)
        if events:
            events[2].record(stream)
        S.starkv_decode_combine(layer.plan, layer.cache, q, Bk, Bv, ctx, L, layer.out, layer.dec_ws)
        if events:
            events[3].record(stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    # eager pass: per-kernel times from HIP events on the launch stream
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i, ev[i])
    torch.cuda.synchronize()
    wall_eager = time.perf_counter() - t0
    t_app = np.array([e[0].elapsed_time(e[1]) for e in ev])
    t_split = np.array([e[1].elapsed_time(e[2]) for e in ev])
    t_comb = np.array([e[2].elapsed_time(e[3]) for e in ev])
    ms_eager = wall_eager * 1e3 / args.steps
    ms_step = ms_eager
    if not args.no_graph:
        # the step captured once per layer cache in a HIP graph (no launch gaps)
        graphs = []
        for li in range(len(layers)):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                step(li)
            graphs.append(g)
        for i in range(args.warmup):
            graphs[i % len(graphs)].replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            graphs[i % len(graphs)].replay()
        torch.cuda.synchronize()
        ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    absorbed = None if args.no_absorbed else time_absorbed(args, w, inp, layers, q, Bk, ctx, x,
                                                           pos_new, A, stream)
    prefill = time_prefill(args, w, inp, layers[0], A, stream) if w.append_tokens > 1 else None
    tokens = int(inp.ctx_len.sum())
    layout = S.starkv_cache_layout(layers[0].plan)
    per_token = (sum(layout.key_row_bytes[g] + 4 * layout.key_groups[g]
                     for g in range(w.n_kv_heads))
                 + layout.value_row_bytes + 4 * layout.value_groups)
    alg_bytes = per_token * tokens
    # useful flops per cached token: key reconstruction 2*sum(r)*d, scores 2*H_q*d,
    # value latents 2*H_q*r_v
    flops_token = (2 * sum(inp.key_rank) * w.head_dim + 2 * w.n_q_heads * w.head_dim
                   + 2 * w.n_q_heads * w.value_rank)
    alg_flops = flops_token * tokens
    split_s = float(t_split.mean()) / 1e3
    achieved = alg_bytes / split_s / 1e9
    log(f"append {t_app.mean() * 1e3:.1f} us  split {t_split.mean() * 1e3:.1f} us "
        f"(median {np.median(t_split) * 1e3:.1f})  combine {t_comb.mean() * 1e3:.1f} us  "
        f"wall/step {ms_step * 1e3:.1f} us (eager {ms_eager * 1e3:.1f} us)")
    copy = copy_stream(torch, stream)
    rstream = read_stream(torch, stream)
    log(f"read stream {rstream['GBps']:.0f} GB/s")
    log(f"device copy {copy['GBps']:.0f} GB/s (read + write)")
    traffic, tsum = measured_traffic(w.name)
    result = {
        "metric": "decode-attention tokens/s at 128K ctx; achieved HBM GB/s vs peak",
        "value": B / (ms_step / 1e3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "precision": {"compute": "fp16 MFMA operands, fp32 accumulation",
                      "q": _DT_NAMES[w.q_dtype], "out": _DT_NAMES[w.out_dtype],
                      "cache": {0: "fp16", 1: "int4", 2: "int8/int4", 3: "int4/int3"}[w.qmode]},
        "config": {"workload": w.name, "batch": B, "ctx": L, "q_heads": w.n_q_heads,
                   "kv_heads": w.n_kv_heads, "head_dim": w.head_dim,
                   "key_ranks": inp.key_rank, "value_rank": w.value_rank,
                   "cache": {0: "fp16", 1: "int4", 2: "int8/int4 mixed", 3: "int4/int3 mixed"}[w.qmode]
                            + ", 32-channel groups"
                            + (f", paged ({P}-token pages, shuffled pool)" if P else ""),
                   "layers_rotated": args.layers,
                   "append": f"{w.append_tokens} token/seq from bf16 hidden {w.d_model}",
                   "launch": "eager" if args.no_graph else "hip graph per layer",
                   "ms_per_step_eager": ms_eager},
        "kernels_us": {"append": float(t_app.mean() * 1e3), "decode_split": float(t_split.mean() * 1e3),
                       "decode_combine": float(t_comb.mean() * 1e3)},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": "decode_split", "alg_bytes_per_launch": alg_bytes,
                     "bytes_per_token": per_token,
                     "frac_of_read_stream": achieved / rstream["GBps"]},
        "roofline_mfma": {"achieved": alg_flops / split_s / 1e12, "peak": MFMA_F16_PEAK_TFLOPS,
                          "unit": "TFLOP/s", "frac": alg_flops / split_s / 1e12 / MFMA_F16_PEAK_TFLOPS,
                          "flops_per_token": flops_token,
                          "note": "useful fp16 MFMA work: key reconstruction, scores, p.V'"},
        "decode_split_us_median": float(np.median(t_split) * 1e3),
        "context_tokens_per_s": tokens / (ms_step / 1e3),
        "copy_stream": copy,
        "read_stream": rstream,
    }
    if absorbed is not None:
        result["absorbed_output"] = absorbed
    if prefill is not None:
        result["prefill"] = prefill
    sq = _counter_summary(SQ_SUMMARY, w.name)
    if sq is not None:       # what the matrix cores and vector ALUs did, from the SQ counters
        result["roofline_mfma"]["measured"] = {
            "mfma_busy": sq["simd_fraction"]["mfma_busy"],
            "valu_active": sq["simd_fraction"]["valu_active"],
            "mfma_valu_coexec": sq["simd_fraction"]["mfma_valu_coexec"],
            "source": "profiles/decode_split_c3_sq_counters.json (fractions of SIMD cycles)"}
    if tsum is not None:
        result["roofline"]["traffic_detail"] = {
            k: tsum[k] for k in ("fetch_bytes_per_launch", "write_bytes_per_launch",
                                 "fetch_scale", "write_scale") if k in tsum}
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        result["cpu_baseline"] = cpu_baseline(w, inp, min(args.cpu_sample_ctx or L, L))
    print(json.dumps(result), flush=True)


def time_absorbed(args, w, inp, layers, q, Bk, ctx, x, pos_new, A, stream):
    """The same decode step with the value up-projection absorbed into the output
    projection (Sec. 3.3): append, split, then the merge writing the normalized latents and
    their product with W_abs [d_out][H_q * r_v] into the block output [B][d_out]."""
    import torch
    from paper_2606_08382_amd import starkv as S
    from paper_2606_08382_amd import synth
    from paper_2606_08382_amd.device import to_dev
    B, L = w.batch, w.ctx
    d_out = w.d_model or w.n_q_heads * w.head_dim
    W = to_dev(synth.absorbed_weights(w, d_out))
    y = torch.empty((B, d_out), dtype=torch.float32 if w.out_dtype == synth.DT_F32 else torch.int16,
                    device="cuda")
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]

    def step(i, events=None):
        layer = layers[i % len(layers)]
        if x is not None:
            layer.append(x, pos_new, A_all=A)
        if events:
            events[0].record(stream)
        S.starkv_decode_split(layer.plan, layer.cache, q, Bk, ctx, L, layer.dec_ws)
        if events:
            events[1].record(stream)
        S.starkv_decode_combine_absorbed(layer.plan, layer.cache, q, Bk, W, d_out, ctx, L, y,
                                         layer.dec_ws)
        if events:
            events[2].record(stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    for i in range(args.steps):
        step(i, ev[i])
    torch.cuda.synchronize()
    t_comb = np.array([e[1].elapsed_time(e[2]) for e in ev]) * 1e3
    ms_step = None
    if not args.no_graph:
        graphs = []
        for li in range(len(layers)):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                step(li)
            graphs.append(g)
        for i in range(args.warmup):
            graphs[i % len(graphs)].replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            graphs[i % len(graphs)].replay()
        torch.cuda.synchronize()
        ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    w_bytes = d_out * w.n_q_heads * w.value_rank * 2
    log(f"absorbed output: combine + product {t_comb.mean():.1f} us, wall/step "
        f"{(ms_step or 0) * 1e3:.1f} us (W_abs {w_bytes / 1e6:.1f} MB)")
    return {"d_out": d_out, "W_abs_bytes": w_bytes,
            "combine_and_product_us": float(t_comb.mean()),
            "ms_per_step": ms_step,
            "tokens_per_s": (B / (ms_step / 1e3)) if ms_step else None,
            "note": "append + split + merge to normalized latents + product with W'_out; "
                    "the output is the attention block's [B][d_out] (after the output projection)"}


def time_prefill(args, w, inp, layer, A, stream):
    """The workload's prefill append (w.append_tokens tokens per sequence from bf16 hidden
    states): the down-projection GEMM (bf16 MFMA, fp32 accumulation) and the pack, timed with
    HIP events on the launch stream.  It writes rows 0 .. n-1 of one layer's cache, after the
    decode timing."""
    import torch
    from paper_2606_08382_amd import synth
    from paper_2606_08382_amd.device import to_dev
    n = w.append_tokens
    rng = np.random.default_rng(w.seed + 31)
    x = to_dev(synth.f32_to_bf16_bits(rng.standard_normal((w.batch, n, w.d_model),
                                                         dtype=np.float32)))
    pos = torch.zeros(w.batch, dtype=torch.int32, device="cuda")
    reps = max(3, min(args.steps, 10))
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    layer.append(x, pos, A_all=A)            # warm-up (and workspace sizing)
    torch.cuda.synchronize()
    for a, b in ev:
        a.record(stream)
        layer.append(x, pos, A_all=A)
        b.record(stream)
    torch.cuda.synchronize()
    us = float(np.median([a.elapsed_time(b) * 1e3 for a, b in ev]))
    M, N, K = w.batch * n, inp.width, w.d_model
    flops = 2.0 * M * N * K
    tf = flops / (us * 1e-6) / 1e12
    log(f"prefill: {M} rows x {N} x {K}: {us:.1f} us (down-projection and pack), {tf:.0f} TFLOP/s")
    return {"tokens": M, "gemm": [M, N, K], "us": us, "flops": flops, "tflops": tf,
            "peak_tflops": MFMA_F16_PEAK_TFLOPS, "frac": tf / MFMA_F16_PEAK_TFLOPS,
            "note": "append of the prefill from bf16 hidden states: down-projection GEMM (bf16 "
                    "operands, fp32 accumulation) plus the pack of every token; median of HIP "
                    "events; frac against the dense bf16 MFMA peak"}


_fill_plans = {}


def _fill_plan(layer, w, inp):
    """A plan with the layer's cache layout taking fp16 latents directly (d_model = 0), used to
    fill the caches before timing."""
    from paper_2606_08382_amd import starkv as S
    key = id(layer)
    if key not in _fill_plans:
        pool = layer.pool
        cfg = S.make_config(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.ctx, inp.key_rank,
                            w.value_rank, w.qmode, w.rope_theta, d_model=0,
                            q_dtype=w.q_dtype, out_dtype=w.out_dtype,
                            page_tokens=pool.page_tokens if pool else 0,
                            n_pages=pool.n_pages if pool else 0,
                            block_table=pool.table if pool else None)
        _fill_plans[key] = S.starkv_plan_create(cfg)
    return _fill_plans[key]


if __name__ == "__main__":
    main()
