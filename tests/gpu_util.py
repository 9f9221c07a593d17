"""Helpers for GPU parity tests: seeded inputs, device buffers, error norms."""
import numpy as np

import synthetic


def torch():
    import torch as t

    return t


def rng(seed):
    return np.random.default_rng(seed)


def rep(x, dtype):
    """Round a float array to the values representable in `dtype` ('bf16' or 'f32')."""
    x = np.asarray(x, np.float32)
    if dtype == "bf16":
        return synthetic.bf16_bits_to_f32(synthetic.round_to_bf16_bits(x)).reshape(x.shape)
    return x


def dev(x, dtype):
    """numpy (already representable) -> device tensor holding `dtype` elements."""
    t = torch()
    a = t.from_numpy(np.ascontiguousarray(np.asarray(x, np.float32)))
    if dtype == "bf16":
        a = a.to(t.bfloat16)
    return a.cuda()


def dev_f32(x):
    return dev(x, "f32")


def dev_i32(x):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(np.asarray(x, np.int32))).cuda()


def empty(shape, dtype):
    t = torch()
    return t.zeros(shape, dtype=t.bfloat16 if dtype == "bf16" else t.float32, device="cuda")


def host(t_):
    return t_.float().cpu().numpy().astype(np.float64)


def ptr(t_):
    return t_.data_ptr()


def rel_err(got, ref):
    """Normwise (max-norm) relative error: max|got - ref| / max|ref|."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / (den if den > 0 else 1.0))


def elem_err(got, ref, floor=1e-2):
    """Elementwise relative error with a floor: max_i |g_i - r_i| / max(|r_i|, floor * max|r|).

    Complements the normwise rel_err: an element far below the tensor's scale
    is measured against floor * max|r| instead of its own magnitude."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    top = np.max(np.abs(ref))
    den = np.maximum(np.abs(ref), floor * (top if top > 0 else 1.0))
    return float(np.max(np.abs(got - ref) / den))


def dt_code(dtype):
    from paper_2403_10504_amd import atom as A

    return A.ATOM_BF16 if dtype == "bf16" else A.ATOM_F32


def sync():
    torch().cuda.synchronize()


def host_digests(sess, which):
    """SHA-256 of the raw bytes of each node's host buffer `which` (list over nodes).

    Nodes are hashed in parallel (hashlib releases the GIL on large buffers)."""
    import ctypes
    import hashlib
    from concurrent.futures import ThreadPoolExecutor

    from paper_2403_10504_amd import atom as A

    def one(node):
        ptr, nbytes = A.atom_host_tensor(sess.ctx, node, which)
        return hashlib.sha256((ctypes.c_char * nbytes).from_address(ptr)).hexdigest()

    with ThreadPoolExecutor(8) as ex:
        return list(ex.map(one, range(sess.n_nodes)))
