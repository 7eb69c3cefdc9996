"""ctypes binding of libstarkv.so (argument marshalling only).

Every entry point has the C name.  Device arguments may be torch tensors (their
``data_ptr()`` is passed) or integer addresses.  ``stream`` defaults to torch's
current stream.  There is no fallback: if the HIP library is missing, loading
it raises.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libstarkv.so")

STARKV_OK = 0
STATUS_NAMES = {0: "OK", 1: "INVALID_ARG", 2: "UNSUPPORTED", 3: "CAPACITY", 4: "WORKSPACE",
                5: "ALIGNMENT", 6: "HIP"}
Q_F16, Q_INT4, Q_MIX8_4, Q_MIX4_3 = 0, 1, 2, 3
DT_F16, DT_BF16, DT_F32 = 0, 1, 2   # F32: attention output only
MAX_KV_HEADS = 16


class StarkvError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"STARKV_ERR_{STATUS_NAMES.get(status, status)}: {detail}")
        self.status = status


class starkv_config(C.Structure):
    _fields_ = [("batch", C.c_int32), ("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("capacity", C.c_int32),
                ("key_rank", C.POINTER(C.c_int32)), ("value_rank", C.c_int32),
                ("qmode", C.c_int32), ("group_size", C.c_int32), ("rope_theta", C.c_double),
                ("d_model", C.c_int32), ("q_dtype", C.c_int32), ("out_dtype", C.c_int32),
                ("x_dtype", C.c_int32), ("page_tokens", C.c_int32), ("n_pages", C.c_int32),
                ("block_table", C.c_void_p)]


class starkv_layout(C.Structure):
    _fields_ = [("total_bytes", C.c_int64), ("padded_capacity", C.c_int32),
                ("sum_key_rank", C.c_int32),
                ("key_code_offset", C.c_int64 * MAX_KV_HEADS),
                ("key_meta_offset", C.c_int64 * MAX_KV_HEADS),
                ("key_row_bytes", C.c_int32 * MAX_KV_HEADS),
                ("key_groups", C.c_int32 * MAX_KV_HEADS),
                ("key_outlier_channels", C.c_int32 * MAX_KV_HEADS),
                ("value_code_offset", C.c_int64), ("value_meta_offset", C.c_int64),
                ("value_row_bytes", C.c_int32), ("value_groups", C.c_int32),
                ("value_outlier_channels", C.c_int32), ("rows", C.c_int64),
                ("page_tokens", C.c_int32), ("pages_per_sequence", C.c_int32)]


class starkv_decode_info(C.Structure):
    _fields_ = [("head_dim", C.c_int32), ("qmode", C.c_int32), ("score_tiles", C.c_int32),
                ("value_tiles", C.c_int32), ("head_groups", C.c_int32),
                ("device_plan", C.c_int32), ("k_lo", C.c_int32), ("items", C.c_int32),
                ("split_tokens", C.c_int32), ("lds_bytes", C.c_int32)]


EXPORTS = ["starkv_plan_create", "starkv_plan_destroy", "starkv_cache_bytes",
           "starkv_cache_layout", "starkv_append_workspace_bytes",
           "starkv_decode_workspace_bytes", "starkv_append", "starkv_decode_attn",
           "starkv_decode_split", "starkv_decode_combine", "starkv_decode_splits",
           "starkv_decode_split_tokens", "starkv_status_string", "starkv_last_error",
           "starkv_decode_attn_absorbed", "starkv_decode_combine_absorbed",
           "starkv_decode_describe", "starkv_decode_attn_noalloc", "starkv_read_stream"]

_lib = None


def lib():
    """Open libstarkv.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        P, S = C.c_void_p, C.c_size_t
        L.starkv_plan_create.argtypes = [C.POINTER(starkv_config), C.POINTER(C.c_void_p)]
        L.starkv_plan_create.restype = C.c_int
        L.starkv_plan_destroy.argtypes = [P]
        L.starkv_plan_destroy.restype = None
        L.starkv_cache_bytes.argtypes = [P]
        L.starkv_cache_bytes.restype = S
        L.starkv_cache_layout.argtypes = [P, C.POINTER(starkv_layout)]
        L.starkv_cache_layout.restype = C.c_int
        L.starkv_append_workspace_bytes.argtypes = [P, C.c_int32]
        L.starkv_append_workspace_bytes.restype = S
        L.starkv_decode_workspace_bytes.argtypes = [P, C.c_int32]
        L.starkv_decode_workspace_bytes.restype = S
        L.starkv_append.argtypes = [P, P, P, P, P, C.c_int32, P, S, P]
        L.starkv_append.restype = C.c_int
        L.starkv_decode_attn.argtypes = [P, P, P, P, P, P, C.c_int32, P, P, S, P]
        L.starkv_decode_attn.restype = C.c_int
        L.starkv_decode_split.argtypes = [P, P, P, P, P, C.c_int32, P, S, P]
        L.starkv_decode_split.restype = C.c_int
        L.starkv_decode_combine.argtypes = [P, P, P, P, P, P, C.c_int32, P, P, S, P]
        L.starkv_decode_combine.restype = C.c_int
        L.starkv_decode_attn_absorbed.argtypes = [P, P, P, P, P, C.c_int32, P, C.c_int32, P, P,
                                                  S, P]
        L.starkv_decode_attn_absorbed.restype = C.c_int
        L.starkv_decode_combine_absorbed.argtypes = [P, P, P, P, P, C.c_int32, P, C.c_int32, P,
                                                     P, S, P]
        L.starkv_decode_combine_absorbed.restype = C.c_int
        L.starkv_decode_splits.argtypes = [P, C.c_int32]
        L.starkv_decode_splits.restype = C.c_int32
        L.starkv_decode_split_tokens.argtypes = [P, C.c_int32]
        L.starkv_decode_split_tokens.restype = C.c_int32
        L.starkv_decode_attn_noalloc.argtypes = [P, P, P, P, P, P, C.c_int32, P, P]
        L.starkv_decode_attn_noalloc.restype = C.c_int
        L.starkv_decode_describe.argtypes = [P, C.c_int32, C.POINTER(starkv_decode_info)]
        L.starkv_decode_describe.restype = C.c_int
        L.starkv_read_stream.argtypes = [P, S, C.c_int32, P, S, P]
        L.starkv_read_stream.restype = C.c_int
        L.starkv_status_string.argtypes = [C.c_int]
        L.starkv_status_string.restype = C.c_char_p
        L.starkv_last_error.argtypes = []
        L.starkv_last_error.restype = C.c_char_p
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != STARKV_OK:
        raise StarkvError(status, lib().starkv_last_error().decode())


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream):
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    if torch.cuda.is_available() and torch.cuda.is_initialized():
        return torch.cuda.current_stream().cuda_stream
    return None


class Plan:
    """Owns a starkv_plan*; destroyed with the object."""

    def __init__(self, handle: int, cfg: starkv_config, key_rank: Sequence[int]):
        self.handle = handle
        self.cfg = cfg
        self.key_rank = list(key_rank)

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.starkv_plan_destroy(self.handle)
            self.handle = None


def make_config(batch, n_q_heads, n_kv_heads, head_dim, capacity, key_rank, value_rank,
                qmode, rope_theta, d_model=0, q_dtype=DT_BF16, out_dtype=DT_BF16,
                x_dtype=DT_BF16, group_size=32, page_tokens=0, n_pages=0, block_table=None):
    """block_table: device int32 [batch][ceil(capacity / page_tokens)] (tensor or address)
    for a paged cache."""
    ranks = (C.c_int32 * max(len(key_rank), 1))(*[int(r) for r in key_rank])
    cfg = starkv_config(batch, n_q_heads, n_kv_heads, head_dim, capacity,
                        C.cast(ranks, C.POINTER(C.c_int32)), value_rank, qmode, group_size,
                        float(rope_theta), d_model, q_dtype, out_dtype, x_dtype,
                        page_tokens, n_pages, _ptr(block_table))
    cfg._ranks = ranks   # keep the array alive with the struct
    return cfg


def starkv_plan_create(cfg: starkv_config) -> Plan:
    h = C.c_void_p()
    _check(lib().starkv_plan_create(C.byref(cfg), C.byref(h)))
    n_kv = cfg.n_kv_heads
    return Plan(h.value, cfg, [cfg.key_rank[i] for i in range(n_kv)])


def starkv_cache_bytes(plan: Plan) -> int:
    return lib().starkv_cache_bytes(plan.handle)


def starkv_cache_layout(plan: Plan) -> starkv_layout:
    out = starkv_layout()
    _check(lib().starkv_cache_layout(plan.handle, C.byref(out)))
    return out


def starkv_append_workspace_bytes(plan: Plan, n_new: int) -> int:
    return lib().starkv_append_workspace_bytes(plan.handle, n_new)


def starkv_decode_workspace_bytes(plan: Plan, max_ctx: int) -> int:
    return lib().starkv_decode_workspace_bytes(plan.handle, max_ctx)


def starkv_decode_splits(plan: Plan, max_ctx: int) -> int:
    return lib().starkv_decode_splits(plan.handle, max_ctx)


def starkv_decode_split_tokens(plan: Plan, max_ctx: int) -> int:
    return lib().starkv_decode_split_tokens(plan.handle, max_ctx)


def starkv_decode_describe(plan: Plan, max_ctx: int) -> dict:
    d = starkv_decode_info()
    _check(lib().starkv_decode_describe(plan.handle, max_ctx, C.byref(d)))
    return {k: getattr(d, k) for k, _ in starkv_decode_info._fields_}


def split_plan(info: dict, ctx_len) -> dict:
    """The split pass's work plan for these context lengths, as the kernels derive it (the
    device plan over the actual lengths, or equal splits): split length, steps per split and
    the number of work items with tokens."""
    lens = [max(0, int(x)) for x in ctx_len]
    if info["device_plan"]:
        k = None
        for kk in range(info["k_lo"], 65):
            steps = [-(-L // 128) for L in lens]
            if sum(-(-m // kk) for m in steps) <= info["items"]:
                k = kk
                break
        S = 128 * (k if k is not None else 64)
    else:
        S = info["split_tokens"]
    items = sum(-(-L // S) for L in lens)
    return {"split_tokens": S, "steps_per_split": S // 128, "items": items,
            "instance": f"<{info['head_dim']},{info['qmode']},{info['score_tiles']},"
                        f"{info['value_tiles']}> x {info['head_groups']} head groups"}


def _nbytes(t) -> int:
    if t is None or isinstance(t, int):
        return 1 << 62 if isinstance(t, int) else 0
    return t.numel() * t.element_size()


def starkv_append(plan: Plan, cache, x_or_latents, A_all, pos, n_new: int, ws=None,
                  ws_bytes: Optional[int] = None, stream=None) -> None:
    _check(lib().starkv_append(plan.handle, _ptr(cache), _ptr(x_or_latents), _ptr(A_all),
                               _ptr(pos), n_new, _ptr(ws),
                               _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream)))


def starkv_decode_attn(plan: Plan, cache, q, B_k, B_v, ctx_len, max_ctx: int, out, ws,
                       ws_bytes: Optional[int] = None, stream=None) -> None:
    _check(lib().starkv_decode_attn(plan.handle, _ptr(cache), _ptr(q), _ptr(B_k), _ptr(B_v),
                                    _ptr(ctx_len), max_ctx, _ptr(out), _ptr(ws),
                                    _nbytes(ws) if ws_bytes is None else ws_bytes,
                                    _stream(stream)))


def starkv_decode_attn_noalloc(plan: Plan, cache, q, B_k, B_v, ctx_len, max_ctx: int, out,
                               stream=None) -> None:
    _check(lib().starkv_decode_attn_noalloc(plan.handle, _ptr(cache), _ptr(q), _ptr(B_k),
                                            _ptr(B_v), _ptr(ctx_len), max_ctx, _ptr(out),
                                            _stream(stream)))


def starkv_read_stream(src, n_bytes: int, sink, workgroups: int = 0, stream=None) -> None:
    """The plain HBM read stream (a measurement aid): reads n_bytes at src once."""
    sink_bytes = sink.numel() * sink.element_size() if hasattr(sink, "numel") else 0
    _check(lib().starkv_read_stream(_ptr(src), n_bytes, workgroups, _ptr(sink), sink_bytes,
                                    _stream(stream)))


def starkv_decode_split(plan: Plan, cache, q, B_k, ctx_len, max_ctx: int, ws,
                        ws_bytes: Optional[int] = None, stream=None) -> None:
    _check(lib().starkv_decode_split(plan.handle, _ptr(cache), _ptr(q), _ptr(B_k),
                                     _ptr(ctx_len), max_ctx, _ptr(ws),
                                     _nbytes(ws) if ws_bytes is None else ws_bytes,
                                     _stream(stream)))


def starkv_decode_combine(plan: Plan, cache, q, B_k, B_v, ctx_len, max_ctx: int, out, ws,
                          ws_bytes: Optional[int] = None, stream=None) -> None:
    _check(lib().starkv_decode_combine(plan.handle, _ptr(cache), _ptr(q), _ptr(B_k), _ptr(B_v),
                                       _ptr(ctx_len), max_ctx, _ptr(out), _ptr(ws),
                                       _nbytes(ws) if ws_bytes is None else ws_bytes,
                                       _stream(stream)))


def starkv_decode_attn_absorbed(plan: Plan, cache, q, B_k, W_abs, d_out: int, ctx_len,
                                max_ctx: int, out, ws, ws_bytes: Optional[int] = None,
                                stream=None) -> None:
    _check(lib().starkv_decode_attn_absorbed(plan.handle, _ptr(cache), _ptr(q), _ptr(B_k),
                                             _ptr(W_abs), d_out, _ptr(ctx_len), max_ctx,
                                             _ptr(out), _ptr(ws),
                                             _nbytes(ws) if ws_bytes is None else ws_bytes,
                                             _stream(stream)))


def starkv_decode_combine_absorbed(plan: Plan, cache, q, B_k, W_abs, d_out: int, ctx_len,
                                   max_ctx: int, out, ws, ws_bytes: Optional[int] = None,
                                   stream=None) -> None:
    _check(lib().starkv_decode_combine_absorbed(plan.handle, _ptr(cache), _ptr(q), _ptr(B_k),
                                                _ptr(W_abs), d_out, _ptr(ctx_len), max_ctx,
                                                _ptr(out), _ptr(ws),
                                                _nbytes(ws) if ws_bytes is None else ws_bytes,
                                                _stream(stream)))


def starkv_status_string(status: int) -> str:
    return lib().starkv_status_string(status).decode()


def starkv_last_error() -> str:
    return lib().starkv_last_error().decode()
