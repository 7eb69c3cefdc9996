"""numpy front end for the fp64 CPU oracle (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` import this module.  It loads ``liborc_starkv.so`` (built from
``oracle.c`` by ``oracle/build.py``) and shares no code with the product
library.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(HERE, "liborc_starkv.so")
_lib = None

Q_F16, Q_INT4, Q_MIX8_4, Q_MIX4_3 = 0, 1, 2, 3


class OrcCfg(C.Structure):
    _fields_ = [("batch", C.c_int32), ("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("capacity", C.c_int32),
                ("key_rank", C.c_int32 * 64), ("value_rank", C.c_int32),
                ("qmode", C.c_int32), ("rope_theta", C.c_double), ("d_model", C.c_int32),
                ("page_tokens", C.c_int32), ("n_pages", C.c_int32), ("table", C.c_void_p)]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from oracle import build as _b  # noqa: WPS433 (lazy build of the checker)
            _b.build()
        L = C.CDLL(_LIB_PATH)
        P = C.c_void_p
        L.orc_f16_to_double.restype = C.c_double
        L.orc_f16_to_double.argtypes = [C.c_uint16]
        L.orc_double_to_f16.restype = C.c_uint16
        L.orc_double_to_f16.argtypes = [C.c_double]
        L.orc_f16_ceil.restype = C.c_uint16
        L.orc_f16_ceil.argtypes = [C.c_double]
        L.orc_bf16_to_double.restype = C.c_double
        L.orc_bf16_to_double.argtypes = [C.c_uint16]
        L.orc_n_groups.argtypes = [C.c_int, C.c_int]
        L.orc_outlier_channels.argtypes = [C.c_int, C.c_int]
        L.orc_quantize_block.argtypes = [C.c_int, C.c_int, P, P, P, P]
        L.orc_channel_group.argtypes = [C.c_int, C.c_int, C.c_int, C.POINTER(C.c_int)]
        L.orc_cache_bytes.restype = C.c_int64
        L.orc_cache_bytes.argtypes = [C.POINTER(OrcCfg)]
        L.orc_plane_offset.restype = C.c_int64
        L.orc_plane_offset.argtypes = [C.POINTER(OrcCfg), C.c_int, C.c_int]
        L.orc_append.argtypes = [C.POINTER(OrcCfg), P, P, P, C.c_int]
        L.orc_downproj.argtypes = [C.POINTER(OrcCfg), P, C.c_int, P, C.c_int, P, P]
        L.orc_read_token.argtypes = [C.POINTER(OrcCfg), P, C.c_int, C.c_int, P, P]
        L.orc_reconstruct_key.argtypes = [C.POINTER(OrcCfg), P, P, C.c_int, C.c_int,
                                          C.c_int, C.c_int, P]
        L.orc_rope.argtypes = [P, C.c_int, C.c_double, C.c_double]
        L.orc_rope.restype = None
        L.orc_decode_attn.argtypes = [C.POINTER(OrcCfg), P, P, C.c_int, P, P, P, P,
                                      C.c_int, P, C.c_int]
        L.orc_decode_latent.argtypes = [C.POINTER(OrcCfg), P, P, C.c_int, P, P, P,
                                        C.c_int, P, C.c_int]
        L.orc_decode_latent.restype = C.c_int
        L.orc_dense_attn.argtypes = [C.c_int, C.c_int, P, P, P, C.c_double, P]
        L.orc_dense_attn.restype = None
        _lib = L
    return _lib


def _p(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(C.c_void_p)


def make_cfg(batch, n_q_heads, n_kv_heads, head_dim, capacity, key_rank, value_rank,
             qmode, rope_theta, d_model=0, page_tokens=0, n_pages=0, table=None) -> OrcCfg:
    """page_tokens > 0: a paged cache of n_pages pages; table [batch][ceil(capacity /
    page_tokens)] int32 gives the pool page of each sequence's page (kept alive here)."""
    c = OrcCfg()
    c.page_tokens, c.n_pages = int(page_tokens), int(n_pages)
    if page_tokens:
        per_seq = -(-capacity // page_tokens)
        t = np.ascontiguousarray(np.asarray(table, dtype=np.int32).reshape(batch, per_seq))
        c._table = t
        c.table = t.ctypes.data_as(C.c_void_p).value
    c.batch, c.n_q_heads, c.n_kv_heads = batch, n_q_heads, n_kv_heads
    c.head_dim, c.capacity = head_dim, capacity
    for g, r in enumerate(key_rank):
        c.key_rank[g] = int(r)
    c.value_rank, c.qmode, c.rope_theta, c.d_model = value_rank, qmode, float(rope_theta), d_model
    return c


def f16_bits(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.float16)).view(np.uint16)


def f16_to_double(h: int) -> float:
    return lib().orc_f16_to_double(int(h))


def double_to_f16(x: float) -> int:
    return lib().orc_double_to_f16(float(x))


def f16_ceil(q: float) -> int:
    return lib().orc_f16_ceil(float(q))


def bf16_to_double(b: int) -> float:
    return lib().orc_bf16_to_double(int(b))


def n_groups(qmode: int, r: int) -> int:
    return lib().orc_n_groups(qmode, r)


def outlier_channels(qmode: int, r: int) -> int:
    return lib().orc_outlier_channels(qmode, r)


def channel_group(qmode: int, r: int, c: int):
    bits = C.c_int(0)
    g = lib().orc_channel_group(qmode, r, c, C.byref(bits))
    return g, bits.value


def quantize_block(qmode: int, x_bits: np.ndarray):
    """x_bits: fp16 bit patterns (uint16) of one latent block.  Returns (codes, s, z)."""
    x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
    r = x_bits.size
    codes = np.zeros(r, np.uint8)
    ng = max(n_groups(qmode, r), 1)
    s = np.zeros(ng, np.uint16)
    z = np.zeros(ng, np.uint16)
    lib().orc_quantize_block(qmode, r, _p(x_bits), _p(codes), _p(s), _p(z))
    return codes, s[:n_groups(qmode, r)], z[:n_groups(qmode, r)]


def cache_bytes(cfg: OrcCfg) -> int:
    return lib().orc_cache_bytes(C.byref(cfg))


def plane_offset(cfg: OrcCfg, which: int, head: int = 0) -> int:
    return lib().orc_plane_offset(C.byref(cfg), which, head)


def new_cache(cfg: OrcCfg) -> np.ndarray:
    return np.zeros(cache_bytes(cfg), np.uint8)


def append(cfg: OrcCfg, cache: np.ndarray, latents_bits: np.ndarray, pos) -> None:
    lat = np.ascontiguousarray(latents_bits, dtype=np.uint16)
    pos = np.ascontiguousarray(pos, dtype=np.int32)
    n_new = lat.shape[1]
    if lib().orc_append(C.byref(cfg), _p(cache), _p(lat), _p(pos), n_new) != 0:
        raise ValueError(f"oracle append refused: batch {cfg.batch} (at most 1024), n_new {n_new}")


def downproj(cfg: OrcCfg, x_bits: np.ndarray, x_is_bf16: bool, A_bits: np.ndarray):
    """Returns (fp16 latent bits [n_tok][width], fp64 unrounded [n_tok][width])."""
    x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
    A_bits = np.ascontiguousarray(A_bits, dtype=np.uint16)
    n_tok = x_bits.size // cfg.d_model
    width = A_bits.shape[-1]
    lat = np.zeros((n_tok, width), np.uint16)
    z64 = np.zeros((n_tok, width), np.float64)
    lib().orc_downproj(C.byref(cfg), _p(x_bits), int(x_is_bf16), _p(A_bits), n_tok,
                       _p(lat), _p(z64))
    return lat, z64


def read_token(cfg: OrcCfg, cache: np.ndarray, b: int, t: int):
    sum_r = sum(cfg.key_rank[g] for g in range(cfg.n_kv_heads))
    kh = np.zeros(max(sum_r, 1), np.float64)
    vh = np.zeros(max(cfg.value_rank, 1), np.float64)
    lib().orc_read_token(C.byref(cfg), _p(cache), b, t, _p(kh), _p(vh))
    return kh[:sum_r], vh[:cfg.value_rank]


def reconstruct_key(cfg: OrcCfg, cache, Bk_bits, b, g, t, rope: bool) -> np.ndarray:
    k = np.zeros(cfg.head_dim, np.float64)
    Bk_bits = np.ascontiguousarray(Bk_bits, dtype=np.uint16)
    lib().orc_reconstruct_key(C.byref(cfg), _p(cache), _p(Bk_bits), b, g, t, int(rope), _p(k))
    return k


def rope(v: np.ndarray, t: float, theta: float) -> np.ndarray:
    v = np.ascontiguousarray(v, dtype=np.float64).copy()
    lib().orc_rope(_p(v), v.size, float(t), float(theta))
    return v


def decode_attn(cfg: OrcCfg, cache, q_bits, q_is_bf16, Bk_bits, Bv_bits, ctx_len,
                sel=None, n_threads: int = 0):
    """Returns (out fp64 [B][H_q][d], threads used).  sel: list of (b, head) pairs."""
    q_bits = np.ascontiguousarray(q_bits, dtype=np.uint16)
    Bk_bits = np.ascontiguousarray(Bk_bits, dtype=np.uint16)
    Bv_bits = np.ascontiguousarray(Bv_bits, dtype=np.uint16)
    ctx = np.ascontiguousarray(ctx_len, dtype=np.int32)
    out = np.full((cfg.batch, cfg.n_q_heads, cfg.head_dim), np.nan, np.float64)
    if sel is not None:
        s = np.ascontiguousarray(np.asarray(sel, dtype=np.int32).reshape(-1))
        n_sel = s.size // 2
        sp = _p(s)
    else:
        s, n_sel, sp = None, 0, None
    nt = lib().orc_decode_attn(C.byref(cfg), _p(cache), _p(q_bits), int(q_is_bf16),
                               _p(Bk_bits), _p(Bv_bits), _p(ctx), sp, n_sel, _p(out),
                               int(n_threads))
    if nt < 0:
        raise ValueError("oracle decode refused: a context length outside [0, capacity] "
                         "or a selected pair out of range")
    return out, nt


def decode_latent(cfg: OrcCfg, cache, q_bits, q_is_bf16, Bk_bits, ctx_len, sel=None,
                  n_threads: int = 0):
    """The normalized value latent a_i / l_i per query head, fp64 [B][H_q][r_v] (NaN where
    not selected; zero for an empty context).  sel: list of (b, head) pairs."""
    q_bits = np.ascontiguousarray(q_bits, dtype=np.uint16)
    Bk_bits = np.ascontiguousarray(Bk_bits, dtype=np.uint16)
    ctx = np.ascontiguousarray(ctx_len, dtype=np.int32)
    lat = np.full((cfg.batch, cfg.n_q_heads, cfg.value_rank), np.nan, np.float64)
    if sel is not None:
        s = np.ascontiguousarray(np.asarray(sel, dtype=np.int32).reshape(-1))
        n_sel, sp = s.size // 2, _p(s)
    else:
        s, n_sel, sp = None, 0, None
    nt = lib().orc_decode_latent(C.byref(cfg), _p(cache), _p(q_bits), int(q_is_bf16),
                                 _p(Bk_bits), _p(ctx), sp, n_sel, _p(lat), int(n_threads))
    if nt < 0:
        raise ValueError("oracle decode refused: a context length outside [0, capacity] "
                         "or a selected pair out of range")
    return lat, nt


def decode_attn_absorbed(cfg: OrcCfg, cache, q_bits, q_is_bf16, Bk_bits, W_abs_bits, ctx_len,
                         batches=None, n_threads: int = 0):
    """Attention output with the value up-projection absorbed into the output projection
    (Sec. 3.3, weight absorption): y_b = sum_i (a_i / l_i) . W'_out,i^T, where W_abs_bits
    [d_out][H_q * r_v] fp16 holds W'_out,i = W_out,i U_V,g(i) of query head i in columns
    i*r_v .. i*r_v + r_v - 1.  The sum over heads and latent channels is one fp64 matrix
    product.  batches: the sequences to compute (others are NaN).  Returns (y fp64
    [B][d_out], threads used)."""
    H, rv = cfg.n_q_heads, cfg.value_rank
    bs = list(range(cfg.batch)) if batches is None else list(batches)
    sel = [(b, i) for b in bs for i in range(H)]
    lat, nt = decode_latent(cfg, cache, q_bits, q_is_bf16, Bk_bits, ctx_len, sel, n_threads)
    W = np.ascontiguousarray(W_abs_bits, dtype=np.uint16).view(np.float16).astype(np.float64)
    assert W.shape[1] == H * rv
    y = np.full((cfg.batch, W.shape[0]), np.nan, np.float64)
    if bs:
        y[bs] = lat[bs].reshape(len(bs), H * rv) @ W.T
    return y, nt


def dense_attn(q: np.ndarray, K: np.ndarray, V: np.ndarray, theta: float) -> np.ndarray:
    q = np.ascontiguousarray(q, np.float64)
    K = np.ascontiguousarray(K, np.float64)
    V = np.ascontiguousarray(V, np.float64)
    out = np.zeros(q.size, np.float64)
    lib().orc_dense_attn(q.size, K.shape[0], _p(q), _p(K), _p(V), float(theta), _p(out))
    return out
