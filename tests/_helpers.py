"""Shared helpers for the GPU parity tests (the HIP path and the oracle fed the same inputs)."""
import sys

import numpy as np

from oracle import oracle as O
from paper_2606_08382_amd import synth

ATOL, RTOL, NORM = 2e-3, 1e-3, 1e-2


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def half_ulp(ref, out_dtype):
    """Half a unit in the last place of the output type at |ref|: the rounding of the fp32
    result into a 16-bit output adds up to this much on top of the arithmetic's error."""
    if out_dtype == synth.DT_F32:
        return np.zeros_like(ref)
    a = np.maximum(np.abs(ref), 2.0 ** -14)
    mant = 7 if out_dtype == synth.DT_BF16 else 10
    return 2.0 ** (np.floor(np.log2(a)) - mant - 1)


def assert_close(got, ref, what="", out_dtype=synth.DT_F32):
    """Elementwise |gpu - oracle| <= 2e-3 + 1e-3 |oracle| (+ half an ulp of a 16-bit output
    type), and max error <= 1 % of max |oracle|."""
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = np.abs(got - ref)
    tol = ATOL + RTOL * np.abs(ref) + half_ulp(ref, out_dtype)
    bad = err > tol
    assert not bad.any(), (f"{what}: {bad.sum()} elements out of tolerance, worst err "
                           f"{err.max():.3e} at {np.unravel_index(err.argmax(), err.shape)}")
    scale = np.abs(ref).max()
    if scale > 0:
        assert err.max() <= NORM * scale, f"{what}: max err {err.max():.3e} vs max |o| {scale:.3e}"
    return err.max(), scale


def oracle_cfg(w, inp, capacity=None, d_model=0):
    return O.make_cfg(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim,
                      w.ctx if capacity is None else capacity, inp.key_rank, w.value_rank,
                      w.qmode, w.rope_theta, d_model=d_model)


def small(name, ctx, batch=None, ragged=None):
    return synth.shrink(synth.WORKLOADS[name], ctx=ctx, batch=batch, ragged=ragged)
