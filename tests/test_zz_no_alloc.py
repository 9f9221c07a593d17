"""atom_k_attn_bwd_noalloc (scratch in a library-owned device array) against
atom_k_attn_bwd (scratch passed in), through the C ABI.

Both run the same kernels on the same inputs, so dqkv must be bitwise equal.
Two calls in a row, the second smaller than the first: the array keeps the
first call's D values, which the second must not read.  A size beyond the
array is refused before anything is launched.
"""
import numpy as np
import pytest

from paper_2403_10504_amd import atom as A
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def stream():
    return U.torch().cuda.current_stream().cuda_stream


def inputs(B, T, H, dh, dtype, seed):
    r = U.rng(seed)
    d = H * dh
    qkv = U.dev(U.rep(r.standard_normal((B * T, 3 * d)), dtype), dtype)
    do = U.dev(U.rep(r.standard_normal((B * T, d)), dtype), dtype)
    o = U.empty((B * T, d), dtype)
    lse = U.empty((B, H, T), "f32")
    A.atom_k_attn_fwd(U.dt_code(dtype), U.ptr(qkv), U.ptr(o), U.ptr(lse), B, T, H, dh, stream())
    return qkv, do, o, lse


def both(B, T, H, dh, dtype, seed):
    d = H * dh
    qkv, do, o, lse = inputs(B, T, H, dh, dtype, seed)
    delta = U.empty((B, H, T), "f32")
    ref = U.empty((B * T, 3 * d), dtype)
    got = U.empty((B * T, 3 * d), dtype)
    got.fill_(float("nan"))
    A.atom_k_attn_bwd(U.dt_code(dtype), U.ptr(qkv), U.ptr(o), U.ptr(do), U.ptr(lse), U.ptr(delta), U.ptr(ref),
                      B, T, H, dh, stream())
    A.atom_k_attn_bwd_noalloc(U.dt_code(dtype), U.ptr(qkv), U.ptr(o), U.ptr(do), U.ptr(lse), U.ptr(got),
                              B, T, H, dh, stream())
    U.sync()
    return ref, got


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_equals_scratch_argument_twice_shrinking(dtype):
    t = U.torch()
    # first a larger problem (several key and query tiles, a ragged tail), then
    # a smaller one whose D rows are a prefix of what the array already holds
    for (B, T, H, dh), seed in (((2, 700, 3, 128), 11), ((1, 130, 2, 64), 12)):
        print(f"noalloc {dtype} B={B} T={T} H={H} dh={dh}", flush=True)
        ref, got = both(B, T, H, dh, dtype, seed)
        assert t.equal(ref.view(t.int16) if dtype == "bf16" else ref.view(t.int32),
                       got.view(t.int16) if dtype == "bf16" else got.view(t.int32)), (B, T, H, dh)
        assert bool(t.isfinite(got.float()).all())


def test_noalloc_refuses_sizes_beyond_its_array():
    # B * H * T one past the array: refused on the host, nothing launched
    B, H, dh = 1, 1, 64
    T = A.ATOM_ATTN_NOALLOC_MAX_ROWS + 1
    x = U.empty((16,), "f32")
    with pytest.raises(A.AtomError) as e:
        A.atom_k_attn_bwd_noalloc(A.ATOM_BF16, U.ptr(x), U.ptr(x), U.ptr(x), U.ptr(x), U.ptr(x), B, T, H, dh,
                                  stream())
    assert e.value.status == A.ATOM_EINVAL
