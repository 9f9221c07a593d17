"""ctypes binding of libatom (include/atom.h, include/atom_kernels.h).

Argument marshalling only: every function here forwards to the C ABI function
of the same name; no step of the method runs in Python.  PyTorch is used by
`Session` for the device arena (one uint8 tensor) and the compute stream.

The library must have been built (`python -m paper_2403_10504_amd.build`);
loading fails loudly otherwise.  There is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libatom.so")

ATOM_MAX_NODES = 256
ATOM_MAX_GSLOTS = 16
MAX_STEPS_PER_CALL = 64  # atom_steps limit
ATOM_OK, ATOM_EINVAL, ATOM_ENOPLAN, ATOM_EBUDGET, ATOM_EHIP, ATOM_ESTATE, ATOM_ENOMEM_HOST = 0, -1, -2, -3, -4, -5, -6
ATOM_F32, ATOM_BF16 = 0, 1
ATOM_CKPT_DEVICE, ATOM_CKPT_HOST = 0, 1
(ATOM_EPI_STORE, ATOM_EPI_STORE_F32, ATOM_EPI_ACC_F32, ATOM_EPI_BIAS, ATOM_EPI_BIAS_GELU, ATOM_EPI_BIAS_RESID,
 ATOM_EPI_GELU_BWD) = range(7)
WEIGHTS, GRAD_ACC, GRAD_LAST, MASTER, MOMENT1, MOMENT2 = 0, 1, 2, 3, 4, 5


class atom_config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("n_layer", "d_model", "n_head", "d_mlp", "vocab", "seq_len", "batch", "accum", "dtype", "ckpt")]


ATOM_RULE_PAPER, ATOM_RULE_TIME, ATOM_RULE_FIXED = 0, 1, 2
ATOM_DEFAULT_DUPLEX = 0.85
COST_FIELDS = ("weight_bytes", "mem_bytes", "cut_bytes", "t_fwd", "t_bwd", "t_load", "t_store")


class atom_node_cost(ctypes.Structure):
    _fields_ = [("weight_bytes", ctypes.c_uint64), ("mem_bytes", ctypes.c_uint64), ("cut_bytes", ctypes.c_uint64),
                ("t_fwd", ctypes.c_double), ("t_bwd", ctypes.c_double),
                ("t_load", ctypes.c_double), ("t_store", ctypes.c_double)]

    def as_dict(self):
        return {k: getattr(self, k) for k in COST_FIELDS}


class atom_plan_opts(ctypes.Structure):
    _fields_ = [("strict", ctypes.c_int32), ("duplex", ctypes.c_double)]


class atom_plan(ctypes.Structure):
    _fields_ = [("n_nodes", ctypes.c_int32), ("n_groups", ctypes.c_int32), ("n_slots", ctypes.c_int32),
                ("overlap_ok", ctypes.c_int32), ("exhaustive", ctypes.c_int32), ("accum", ctypes.c_int32),
                ("n_gslots", ctypes.c_int32), ("rule", ctypes.c_int32),
                ("first", ctypes.c_int32 * ATOM_MAX_NODES), ("last", ctypes.c_int32 * ATOM_MAX_NODES),
                ("budget_bytes", ctypes.c_uint64), ("reserve_bytes", ctypes.c_uint64),
                ("slot_bytes", ctypes.c_uint64), ("arena_bytes", ctypes.c_uint64), ("work_bytes", ctypes.c_uint64),
                ("h2d_bytes", ctypes.c_uint64), ("d2h_bytes", ctypes.c_uint64),
                ("forced_h2d_bytes", ctypes.c_uint64), ("cut_bytes", ctypes.c_uint64),
                ("pred_fwd_s", ctypes.c_double), ("pred_first_step_s", ctypes.c_double),
                ("pred_step_s", ctypes.c_double), ("duplex", ctypes.c_double), ("n_evaluated", ctypes.c_int64)]

    def groups(self):
        return [(self.first[g], self.last[g]) for g in range(self.n_groups)]


class atom_tensor_desc(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 16), ("rows", ctypes.c_int32), ("cols", ctypes.c_int32),
                ("offset", ctypes.c_uint64), ("bytes", ctypes.c_uint64)]


class atom_stats(ctypes.Structure):
    _fields_ = [("h2d_bytes", ctypes.c_uint64), ("d2h_bytes", ctypes.c_uint64), ("step_s", ctypes.c_double),
                ("host_accum_s", ctypes.c_double), ("swap_ins", ctypes.c_int32), ("swap_outs", ctypes.c_int32),
                ("host_update_s", ctypes.c_double), ("updated_groups", ctypes.c_int32),
                ("opt_state_pinned", ctypes.c_int32)]


class AtomError(RuntimeError):
    def __init__(self, status, msg=""):
        self.status = status
        super().__init__(f"{status_string(status)} ({status}){': ' + msg if msg else ''}")


_lib = None
P = ctypes.c_void_p
I32, I64, U64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
_SIGS = {
    "atom_version": (ctypes.c_char_p, []),
    "atom_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "atom_node_layout": (ctypes.c_int, [P, I32, P, I32, P, P]),
    "atom_node_costs": (ctypes.c_int, [P, P, I32]),
    "atom_reserve_bytes": (ctypes.c_int, [P, P]),
    "atom_plan_search": (ctypes.c_int, [P, U64, U64, P, I32, P, P]),
    "atom_plan_partition": (ctypes.c_int, [P, U64, P, I32, P, P]),
    "atom_plan_predict": (ctypes.c_int, [P, P, P, I32, ctypes.c_double, I32, I32, P, P]),
    "atom_plan_fixed": (ctypes.c_int, [P, I32, P, I32, I32, P]),
    "atom_ctx_create": (ctypes.c_int, [P, P, P, U64, P, P]),
    "atom_ctx_destroy": (None, [P]),
    "atom_host_tensor": (ctypes.c_int, [P, I32, I32, P, P]),
    "atom_zero_grads": (ctypes.c_int, [P]),
    "atom_set_tokens": (ctypes.c_int, [P, P]),
    "atom_swap_in": (ctypes.c_int, [P, I32]),
    "atom_block_fwd": (ctypes.c_int, [P, I32, I32]),
    "atom_block_bwd": (ctypes.c_int, [P, I32, I32]),
    "atom_swap_out": (ctypes.c_int, [P, I32]),
    "atom_sync": (ctypes.c_int, [P, P]),
    "atom_step": (ctypes.c_int, [P, P, P]),
    "atom_steps": (ctypes.c_int, [P, P, ctypes.c_int32, P]),
    "atom_set_retention": (ctypes.c_int, [P, ctypes.c_int32]),
    "atom_set_embedding_rows": (ctypes.c_int, [P, ctypes.c_int32]),
    "atom_get_stats": (ctypes.c_int, [P, P]),
    "atom_ctx_config": (ctypes.c_int, [P, P, P]),
    "atom_probe_gemm": (ctypes.c_int, [P, I32, I32, I32]),
    "atom_probe_read": (ctypes.c_int, [P, P, P, P, P]),
    "atom_link_bench": (ctypes.c_int, [P, U64, I32, P, P, P]),
    "atom_profile_nodes": (ctypes.c_int, [P, P, P, I32]),
    "atom_optimizer_init": (ctypes.c_int, [P]),
    "atom_optimizer_step": (ctypes.c_int, [P, P, ctypes.c_float, I32]),
    "atom_optimizer_arm": (ctypes.c_int, [P, P, ctypes.c_float, I32]),
    "atom_last_error": (ctypes.c_char_p, [P]),
    "atom_k_gemm": (ctypes.c_int, [ctypes.c_int] * 7 + [P, I64, P, I64, P, I64, P, P, P, I64, P, U64, P]),
    "atom_k_layernorm_fwd": (ctypes.c_int, [ctypes.c_int, P, P, P, P, P, P, I64, ctypes.c_int, P]),
    "atom_k_layernorm_bwd_part_floats": (I64, [I64, ctypes.c_int]),
    "atom_k_layernorm_bwd": (ctypes.c_int, [ctypes.c_int, P, P, P, P, P, P, P, ctypes.c_int, P, P, P, I64,
                                            ctypes.c_int, P]),
    "atom_k_attn_fwd": (ctypes.c_int, [ctypes.c_int, P, P, P] + [ctypes.c_int] * 4 + [P]),
    "atom_k_attn_bwd": (ctypes.c_int, [ctypes.c_int, P, P, P, P, P, P] + [ctypes.c_int] * 4 + [P]),
    "atom_k_attn_bwd_noalloc": (ctypes.c_int, [ctypes.c_int, P, P, P, P, P] + [ctypes.c_int] * 4 + [P]),
    "atom_k_colsum_part_floats": (I64, [I64, ctypes.c_int]),
    "atom_k_colsum": (ctypes.c_int, [ctypes.c_int, P, I64, ctypes.c_int, P, P, P]),
    "atom_k_xent": (ctypes.c_int, [ctypes.c_int, P, I64, P, P, I64, P, I64, ctypes.c_int, ctypes.c_float, P]),
    "atom_k_embed_fwd": (ctypes.c_int, [ctypes.c_int, P, P, P, P, I64, ctypes.c_int, ctypes.c_int, ctypes.c_int, P]),
    "atom_k_copy": (ctypes.c_int, [P, P, I64, P]),
}
EXPORTED = tuple(_SIGS)


def _mapped(name):
    """Files whose path contains `name` mapped into this process (Linux)."""
    try:
        with open("/proc/self/maps") as f:
            return sorted({ln.split()[-1] for ln in f if name in ln})
    except OSError:
        return []


def lib():
    """The loaded libatom (raises if it was not built).

    libatom must run on the same HIP runtime as torch, which owns the device
    memory and the streams it is handed: torch is imported first, so the
    runtime it loaded (HIP and ROCr) satisfies libatom's dependencies (same
    sonames).  Loading libatom first would bring in a second HIP runtime,
    which fails to find the device or mixes two device contexts; that is
    checked here.  A second ROCr copy can be present when a profiler preloads
    its own; libatom's direct ROCr calls (the DMA copies) must then reach the
    instance HIP uses, which atom_ctx_create checks on the arena and the
    pinned host model (ATOM_EHIP otherwise)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2403_10504_amd.build`")
        import torch  # noqa: F401  (loads torch's HIP runtime first)

        h = ctypes.CDLL(LIB_PATH)
        for name in ("libamdhip64",):
            runtimes = _mapped(name)
            if len(runtimes) > 1:
                raise RuntimeError(f"two copies of {name} in one process ({runtimes}): libatom must bind to torch's")
        for name, (res, args) in _SIGS.items():
            fn = getattr(h, name)
            fn.restype = res
            fn.argtypes = args
        _lib = h
    return _lib


def status_string(status):
    return lib().atom_status_string(status).decode()


def _check(status, ctx=None):
    if status != ATOM_OK:
        msg = lib().atom_last_error(ctx).decode() if ctx else ""
        raise AtomError(status, msg)


def _ref(x):
    return ctypes.byref(x)


def make_config(cfg) -> atom_config:
    """atom_config from a synthetic.Config (or any object with the same fields)."""
    return atom_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_mlp, cfg.vocab, cfg.seq_len, cfg.batch,
                       cfg.accum, ATOM_BF16 if cfg.dtype == "bf16" else ATOM_F32,
                       ATOM_CKPT_HOST if getattr(cfg, "ckpt_host", False) else ATOM_CKPT_DEVICE)


# ------------------------------------------------------------------ planner
def atom_version():
    return lib().atom_version().decode()


def atom_node_layout(c: atom_config, node: int):
    descs = (atom_tensor_desc * 16)()
    n = I32()
    nb = U64()
    _check(lib().atom_node_layout(_ref(c), node, descs, 16, _ref(n), _ref(nb)))
    return [(d.name.decode(), d.rows, d.cols, d.offset, d.bytes) for d in descs[: n.value]], nb.value


def atom_node_costs(c: atom_config):
    n = c.n_layer + 2
    out = (atom_node_cost * n)()
    _check(lib().atom_node_costs(_ref(c), out, n))
    return out


def atom_reserve_bytes(c: atom_config) -> int:
    v = U64()
    _check(lib().atom_reserve_bytes(_ref(c), _ref(v)))
    return v.value


def costs_array(costs):
    """atom_node_cost array from a list of dicts (COST_FIELDS; mem_bytes and cut_bytes default to 0)."""
    if isinstance(costs, ctypes.Array):
        return costs
    arr = (atom_node_cost * len(costs))()
    for i, x in enumerate(costs):
        arr[i] = atom_node_cost(int(x["weight_bytes"]), int(x.get("mem_bytes", 0)), int(x.get("cut_bytes", 0)),
                                x["t_fwd"], x["t_bwd"], x["t_load"], x["t_store"])
    return arr


def _opts(strict=False, duplex=0.0):
    return atom_plan_opts(int(bool(strict)), float(duplex))


def atom_plan_search(c: atom_config, budget: int, base: int, costs, strict=False, duplex=0.0) -> atom_plan:
    p = atom_plan()
    arr = costs_array(costs)
    o = _opts(strict, duplex)
    _check(lib().atom_plan_search(_ref(c), budget, base, arr, len(arr), _ref(o), _ref(p)))
    return p


def atom_plan_partition(c: atom_config, budget: int, costs=None, strict=False, duplex=0.0) -> atom_plan:
    p = atom_plan()
    o = _opts(strict, duplex)
    if costs is None:
        _check(lib().atom_plan_partition(_ref(c), budget, None, 0, _ref(o), _ref(p)))
    else:
        arr = costs_array(costs)
        _check(lib().atom_plan_partition(_ref(c), budget, arr, len(arr), _ref(o), _ref(p)))
    return p


def atom_plan_predict(c: atom_config, plan: atom_plan, costs=None, duplex=0.0, n_steps=1, retain=False):
    """(step end times of one call of n_steps steps, forward end of step 0);
    retain: weights kept across the steps of the call (atom_set_retention)."""
    ends = (ctypes.c_double * n_steps)()
    fwd = ctypes.c_double()
    r = 1 if retain else 0
    if costs is None:
        _check(lib().atom_plan_predict(_ref(c), _ref(plan), None, 0, float(duplex), n_steps, r, ends, _ref(fwd)))
    else:
        arr = costs_array(costs)
        _check(lib().atom_plan_predict(_ref(c), _ref(plan), arr, len(arr), float(duplex), n_steps, r, ends,
                                       _ref(fwd)))
    return list(ends), fwd.value


def atom_plan_fixed(c: atom_config, last_nodes, n_slots: int, n_gslots: int = 2) -> atom_plan:
    p = atom_plan()
    arr = (I32 * len(last_nodes))(*last_nodes)
    _check(lib().atom_plan_fixed(_ref(c), len(last_nodes), arr, n_slots, n_gslots, _ref(p)))
    return p


# ------------------------------------------------------------------ context
def atom_ctx_create(c: atom_config, plan: atom_plan, arena_ptr: int, arena_bytes: int, cs: int):
    ctx = P()
    status = lib().atom_ctx_create(_ref(c), _ref(plan), arena_ptr, arena_bytes, cs, _ref(ctx))
    if status != ATOM_OK:
        raise AtomError(status, lib().atom_last_error(None).decode())
    return ctx


def atom_ctx_destroy(ctx):
    lib().atom_ctx_destroy(ctx)


def atom_host_tensor(ctx, node: int, which: int):
    ptr = P()
    nb = U64()
    _check(lib().atom_host_tensor(ctx, node, which, _ref(ptr), _ref(nb)), ctx)
    return ptr.value, nb.value


def atom_zero_grads(ctx):
    _check(lib().atom_zero_grads(ctx), ctx)


def atom_ctx_config(ctx):
    """(atom_config, atom_plan) the context was created with."""
    c, p = atom_config(), atom_plan()
    _check(lib().atom_ctx_config(ctx, _ref(c), _ref(p)), ctx)
    return c, p


def _tokens_ptr(ctx, tokens, steps=False):
    """int32 copy of `tokens` and its pointer, after checking the shape the C
    side will read: [accum][batch][seq_len + 1], with a leading step count
    for atom_steps."""
    t = np.ascontiguousarray(tokens, dtype=np.int32)
    c, _ = atom_ctx_config(ctx)
    want = (c.accum, c.batch, c.seq_len + 1)
    if (t.shape[1:] if steps else t.shape) != want or (steps and (t.ndim != 4 or t.shape[0] < 1)):
        lead = "[n_steps]" if steps else ""
        raise ValueError(f"tokens must be {lead}[accum][batch][seq_len + 1] = {lead}{list(want)}, got {list(t.shape)}")
    return t, t.ctypes.data_as(P)


def atom_set_tokens(ctx, tokens):
    t, p = _tokens_ptr(ctx, tokens)
    _check(lib().atom_set_tokens(ctx, p), ctx)


def atom_swap_in(ctx, group: int):
    _check(lib().atom_swap_in(ctx, group), ctx)


def atom_block_fwd(ctx, node: int, micro: int):
    _check(lib().atom_block_fwd(ctx, node, micro), ctx)


def atom_block_bwd(ctx, node: int, micro: int):
    _check(lib().atom_block_bwd(ctx, node, micro), ctx)


def atom_swap_out(ctx, group: int):
    _check(lib().atom_swap_out(ctx, group), ctx)


def atom_sync(ctx) -> float:
    v = ctypes.c_float()
    _check(lib().atom_sync(ctx, _ref(v)), ctx)
    return v.value


def atom_step(ctx, tokens) -> float:
    t, p = _tokens_ptr(ctx, tokens)
    v = ctypes.c_float()
    _check(lib().atom_step(ctx, p, _ref(v)), ctx)
    return v.value


def atom_set_retention(ctx, on: bool):
    _check(lib().atom_set_retention(ctx, int(bool(on))), ctx)


def atom_set_embedding_rows(ctx, on: bool):
    _check(lib().atom_set_embedding_rows(ctx, int(bool(on))), ctx)


def atom_steps(ctx, tokens) -> np.ndarray:
    """tokens: int32 [n_steps][accum][batch][seq_len + 1]; returns the losses."""
    t, p = _tokens_ptr(ctx, tokens, steps=True)
    n = t.shape[0]
    out = np.zeros(n, dtype=np.float32)
    _check(lib().atom_steps(ctx, p, n, out.ctypes.data_as(P)), ctx)
    return out


def atom_get_stats(ctx) -> atom_stats:
    s = atom_stats()
    _check(lib().atom_get_stats(ctx, _ref(s)), ctx)
    return s


def atom_probe_gemm(ctx, a_kcontig: int, b_kcontig: int, epi: int):
    _check(lib().atom_probe_gemm(ctx, a_kcontig, b_kcontig, epi), ctx)


def atom_probe_read(ctx):
    n = I64()
    sec = ctypes.c_double()
    fl = ctypes.c_double()
    by = ctypes.c_double()
    _check(lib().atom_probe_read(ctx, _ref(n), _ref(sec), _ref(fl), _ref(by)), ctx)
    return n.value, sec.value, fl.value, by.value


def atom_profile_nodes(ctx, c: atom_config, tokens):
    """Measured node costs (ctypes array of atom_node_cost) from one step on `tokens`."""
    n = c.n_layer + 2
    out = (atom_node_cost * n)()
    t, p = _tokens_ptr(ctx, tokens)
    _check(lib().atom_profile_nodes(ctx, p, out, n), ctx)
    return out


class atom_adamw(ctypes.Structure):
    _fields_ = [(n, ctypes.c_float) for n in ("lr", "beta1", "beta2", "eps", "weight_decay")]


def atom_optimizer_init(ctx):
    _check(lib().atom_optimizer_init(ctx), ctx)


def atom_optimizer_step(ctx, lr, grad_scale, step, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0):
    hp = atom_adamw(lr, beta1, beta2, eps, weight_decay)
    _check(lib().atom_optimizer_step(ctx, _ref(hp), grad_scale, step), ctx)


def atom_optimizer_arm(ctx, lr, grad_scale, step, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0):
    hp = atom_adamw(lr, beta1, beta2, eps, weight_decay)
    _check(lib().atom_optimizer_arm(ctx, _ref(hp), grad_scale, step), ctx)


def atom_link_bench(ctx, nbytes: int, iters: int):
    h, d, b = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    _check(lib().atom_link_bench(ctx, nbytes, iters, _ref(h), _ref(d), _ref(b)), ctx)
    return h.value, d.value, b.value


# ------------------------------------------------------------------ kernels
def _kcall(name, *args):
    _check(getattr(lib(), name)(*args))


def atom_k_gemm(dtype, a_kcontig, b_kcontig, epi, M, N, K, A, lda, B, ldb, C, ldc, bias=None, resid=None, aux=None,
                ldaux=0, stream=None, ws=None, ws_bytes=0):
    _kcall("atom_k_gemm", dtype, int(a_kcontig), int(b_kcontig), epi, M, N, K, A, lda, B, ldb, C, ldc, bias, resid,
           aux, ldaux, ws, ws_bytes, stream)


def atom_k_layernorm_fwd(dtype, x, gamma, beta, y, mean, rstd, rows, d, stream=None):
    _kcall("atom_k_layernorm_fwd", dtype, x, gamma, beta, y, mean, rstd, rows, d, stream)


def atom_k_layernorm_bwd_part_floats(rows, d):
    return lib().atom_k_layernorm_bwd_part_floats(rows, d)


def atom_k_layernorm_bwd(dtype, dy, x, mean, rstd, gamma, dres, dres_lp, accumulate, dgamma, dbeta, part, rows, d,
                         stream=None):
    _kcall("atom_k_layernorm_bwd", dtype, dy, x, mean, rstd, gamma, dres, dres_lp, int(accumulate), dgamma, dbeta,
           part, rows, d, stream)


def atom_k_attn_fwd(dtype, qkv, o, lse, B, T, H, dh, stream=None):
    _kcall("atom_k_attn_fwd", dtype, qkv, o, lse, B, T, H, dh, stream)


def atom_k_attn_bwd(dtype, qkv, o, dout, lse, delta, dqkv, B, T, H, dh, stream=None):
    _kcall("atom_k_attn_bwd", dtype, qkv, o, dout, lse, delta, dqkv, B, T, H, dh, stream)


ATOM_ATTN_NOALLOC_MAX_ROWS = 1 << 20


def atom_k_attn_bwd_noalloc(dtype, qkv, o, dout, lse, dqkv, B, T, H, dh, stream=None):
    _kcall("atom_k_attn_bwd_noalloc", dtype, qkv, o, dout, lse, dqkv, B, T, H, dh, stream)


def atom_k_colsum_part_floats(rows, cols):
    return lib().atom_k_colsum_part_floats(rows, cols)


def atom_k_colsum(dtype, x, rows, cols, out, part, stream=None):
    _kcall("atom_k_colsum", dtype, x, rows, cols, out, part, stream)


def atom_k_xent(dtype, logits, ldz, tgt, dz, lddz, loss_rows, rows, V, scale, stream=None):
    _kcall("atom_k_xent", dtype, logits, ldz, tgt, dz, lddz, loss_rows, rows, V, ctypes.c_float(scale), stream)


def atom_k_embed_fwd(dtype, tok, wte, wpe, x, n_tok, T, V, d, stream=None):
    _kcall("atom_k_embed_fwd", dtype, tok, wte, wpe, x, n_tok, T, V, d, stream)


def atom_k_copy(src, dst, nbytes, stream=None):
    _kcall("atom_k_copy", src, dst, nbytes, stream)
