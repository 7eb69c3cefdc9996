"""Device-memory plumbing around the C ABI: one layer's cache, factors and workspaces.

PyTorch provides device memory and the stream; every computation runs in the
library's HIP kernels.
"""
from __future__ import annotations

from typing import Optional

import numpy as np

from . import starkv as S


def to_dev(bits: np.ndarray, device="cuda"):
    """uint16 / int32 / uint8 numpy array -> device tensor with the same bytes."""
    import torch
    a = np.ascontiguousarray(bits)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a.copy()).to(device)


class PagePool:
    """Host-side page allocator of a paged cache (continuous batching).

    Keeps the free pool pages and, per sequence slot, the pages it holds; the block
    table lives on the device (the plan reads it) with a host copy that ``sync``
    uploads.  Pages are handed out lowest-free-first unless ``rng`` shuffles the
    free list (tests use that to scatter sequences over the pool)."""

    def __init__(self, n_pages: int, page_tokens: int, batch: int, capacity: int,
                 device="cuda", rng: Optional[np.random.Generator] = None):
        import torch
        self.n_pages, self.page_tokens, self.batch = n_pages, page_tokens, batch
        self.capacity = capacity
        self.per_seq = -(-capacity // page_tokens)
        free = np.arange(n_pages, dtype=np.int32)
        if rng is not None:
            free = rng.permutation(free).astype(np.int32)
        self.free = list(free[::-1])                 # pop() hands out free[0] first
        self.host = np.full((batch, self.per_seq), -1, np.int32)
        self.table = torch.full((batch, self.per_seq), -1, dtype=torch.int32, device=device)

    def ensure(self, b: int, n_tokens: int) -> None:
        """Give sequence b pages for its first n_tokens tokens."""
        need = -(-n_tokens // self.page_tokens)
        if n_tokens > self.capacity:
            raise ValueError(f"sequence {b}: {n_tokens} tokens exceed the capacity")
        for j in range(need):
            if self.host[b, j] < 0:
                if not self.free:
                    raise MemoryError("page pool exhausted")
                self.host[b, j] = self.free.pop()

    def release(self, b: int) -> None:
        """Return all pages of sequence b to the pool."""
        for j in range(self.per_seq):
            if self.host[b, j] >= 0:
                self.free.append(int(self.host[b, j]))
                self.host[b, j] = -1

    def pages_in_use(self) -> int:
        return int((self.host >= 0).sum())

    def sync(self) -> None:
        """Upload the host table (stream-ordered before later library calls)."""
        import torch
        self.table.copy_(torch.from_numpy(self.host))


class Layer:
    """Plan + cache + workspaces of one attention layer (contiguous, or paged when
    page_tokens > 0: then ``pool`` is the layer's PagePool)."""

    def __init__(self, batch, n_q_heads, n_kv_heads, head_dim, capacity, key_rank, value_rank,
                 qmode, rope_theta, q_dtype, out_dtype, d_model=0, device="cuda",
                 max_ctx: Optional[int] = None, page_tokens: int = 0, n_pages: int = 0,
                 page_rng: Optional[np.random.Generator] = None):
        import torch
        self.pool = None
        if page_tokens:
            self.pool = PagePool(n_pages, page_tokens, batch, capacity, device, page_rng)
        self.cfg = S.make_config(batch, n_q_heads, n_kv_heads, head_dim, capacity, key_rank,
                                 value_rank, qmode, rope_theta, d_model=d_model,
                                 q_dtype=q_dtype, out_dtype=out_dtype, page_tokens=page_tokens,
                                 n_pages=n_pages,
                                 block_table=self.pool.table if self.pool else None)
        self.plan = S.starkv_plan_create(self.cfg)
        self.device = device
        self.batch, self.n_q, self.head_dim = batch, n_q_heads, head_dim
        self.capacity = capacity
        self.out_dtype = out_dtype
        self.cache = torch.zeros(S.starkv_cache_bytes(self.plan), dtype=torch.uint8, device=device)
        self.max_ctx = capacity if max_ctx is None else max_ctx
        self.dec_ws = torch.empty(max(S.starkv_decode_workspace_bytes(self.plan, self.max_ctx), 256),
                                  dtype=torch.uint8, device=device)
        self.app_ws = None
        self.out = torch.empty((batch, n_q_heads, head_dim),
                               dtype=torch.float32 if out_dtype == S.DT_F32 else torch.int16,
                               device=device)

    def _app_ws(self, n_new: int):
        import torch
        need = S.starkv_append_workspace_bytes(self.plan, n_new)
        if need == 0:
            return None
        if self.app_ws is None or self.app_ws.numel() < need:
            self.app_ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        return self.app_ws

    def append(self, x_or_latents, pos, A_all=None, stream=None):
        n_new = int(x_or_latents.shape[1])
        ws = self._app_ws(n_new)
        S.starkv_append(self.plan, self.cache, x_or_latents, A_all, pos, n_new, ws, stream=stream)

    def decode(self, q, B_k, B_v, ctx_len, max_ctx: Optional[int] = None, out=None, stream=None):
        mc = self.max_ctx if max_ctx is None else max_ctx
        out = self.out if out is None else out
        S.starkv_decode_attn(self.plan, self.cache, q, B_k, B_v, ctx_len, mc, out, self.dec_ws,
                             stream=stream)
        return out

    def decode_absorbed(self, q, B_k, W_abs, ctx_len, max_ctx: Optional[int] = None, out=None,
                        stream=None):
        """Attention-block output [B][d_out] with the value up-projection absorbed into the
        output projection; W_abs [d_out][H_q * r_v] fp16 bits (int16 tensor)."""
        import torch
        mc = self.max_ctx if max_ctx is None else max_ctx
        d_out = int(W_abs.shape[0])
        if out is None:
            out = torch.empty((self.batch, d_out),
                              dtype=torch.float32 if self.out_dtype == S.DT_F32 else torch.int16,
                              device=self.device)
        S.starkv_decode_attn_absorbed(self.plan, self.cache, q, B_k, W_abs, d_out, ctx_len, mc,
                                      out, self.dec_ws, stream=stream)
        return out

    def out_float(self, out=None):
        """Output bit patterns -> float64 numpy."""
        import torch
        o = (self.out if out is None else out).cpu()
        if self.out_dtype == S.DT_F32:
            return o.to(torch.float64).numpy()
        if self.out_dtype == S.DT_BF16:
            return o.view(torch.bfloat16).to(torch.float64).numpy()
        return o.view(torch.float16).to(torch.float64).numpy()
