"""Session: a context whose device arena and compute stream come from PyTorch.

Plumbing only.  The arena is one torch uint8 tensor of exactly the plan's
arena size (so the device budget is enforced by construction), the compute
stream is a torch stream at the default priority, and the host model lives
in the library's pinned buffers, exposed here as numpy views.
"""
from __future__ import annotations

import numpy as np

from . import atom as A


class Session:
    def __init__(self, cfg, budget: int | None = None, plan: A.atom_plan | None = None):
        import torch

        if not torch.cuda.is_available():
            raise RuntimeError("Session needs a GPU (the library has no CPU path)")
        self.cfg = cfg
        self.c = A.make_config(cfg)
        if plan is None:
            if budget is None:
                budget = cfg.budget_bytes or (1 << 50)
            plan = A.atom_plan_partition(self.c, budget)
        self.plan = plan
        self.arena = torch.empty(plan.arena_bytes, dtype=torch.uint8, device="cuda")
        self.stream = torch.cuda.Stream()
        self.ctx = A.atom_ctx_create(self.c, plan, self.arena.data_ptr(), plan.arena_bytes, self.stream.cuda_stream)
        self.n_nodes = cfg.n_layer + 2
        self.layout = [A.atom_node_layout(self.c, n)[0] for n in range(self.n_nodes)]
        self.elem = np.uint16 if cfg.dtype == "bf16" else np.float32

    # ---------------------------------------------------------------- host
    def host_view(self, node: int, name: str, which: int = A.WEIGHTS) -> np.ndarray:
        """numpy view of one tensor of the host model (no copy)."""
        ptr, nbytes = A.atom_host_tensor(self.ctx, node, which)
        for tname, rows, cols, off, tbytes in self.layout[node]:
            if tname == name:
                esz = np.dtype(self.elem).itemsize
                if which in (A.GRAD_ACC, A.MASTER, A.MOMENT1, A.MOMENT2):  # fp32, element-indexed
                    dtype, off, count = np.float32, off // esz * 4, tbytes // esz
                else:
                    dtype, count = self.elem, tbytes // esz
                buf = (np.ctypeslib.as_array((np.ctypeslib.ctypes.c_uint8 * (off + count * np.dtype(dtype).itemsize))
                                             .from_address(ptr)))
                arr = buf[off:].view(dtype)[:count]
                return arr.reshape(rows, cols) if cols > 1 else arr
        raise KeyError(name)

    def load_weights(self, seed=None):
        """Fill the host model from the seeded synthetic generator."""
        import synthetic

        seed = synthetic.WEIGHT_SEED if seed is None else seed
        for node in range(self.n_nodes):
            for name, shape, _ in synthetic.param_specs(self.cfg, node):
                v = self.host_view(node, name)
                synthetic.fill_param(v[: shape[0]] if name == "w_head" else v, self.cfg, node, name, seed)

    def set_weights(self, weights):
        """Copy float32 arrays (list over nodes of {name: array}) into the host model."""
        import synthetic

        for node, p in enumerate(weights):
            for name, val in p.items():
                v = self.host_view(node, name)
                if name == "w_head":
                    v = v[: val.shape[0]]
                val = np.asarray(val, np.float32)
                if self.elem == np.uint16:
                    v[...] = synthetic.round_to_bf16_bits(val).reshape(v.shape)
                else:
                    v[...] = val.reshape(v.shape)

    def weights(self):
        """The host model as float32 arrays (list over nodes of {name: array})."""
        return self.grads(A.WEIGHTS)

    def grads(self, which: int = A.GRAD_ACC):
        """Gradients as float32 arrays: accumulators (default) or the last step's;
        also the weights (WEIGHTS) and the optimizer's fp32 master weights and
        moments (MASTER, MOMENT1, MOMENT2)."""
        import synthetic

        out = []
        for node in range(self.n_nodes):
            p = {}
            for name, rows, cols, _, _ in self.layout[node]:
                v = np.array(self.host_view(node, name, which))
                if which in (A.WEIGHTS, A.GRAD_LAST) and self.elem == np.uint16:
                    v = synthetic.bf16_bits_to_f32(v)
                if name == "w_head":
                    v = v[: self.cfg.vocab]
                p[name] = v.astype(np.float32)
            out.append(p)
        return out

    # ---------------------------------------------------------------- step
    def step(self, tokens) -> float:
        return A.atom_step(self.ctx, tokens)

    def steps(self, tokens) -> np.ndarray:
        """Pipelined steps of one global batch; tokens [n][C][B][T+1]."""
        return A.atom_steps(self.ctx, tokens)

    def set_retention(self, on: bool):
        """Load each group once per steps() call when every group has a slot."""
        A.atom_set_retention(self.ctx, on)

    def set_embedding_rows(self, on: bool):
        """Move only the embedding rows a step's tokens use across the host link."""
        A.atom_set_embedding_rows(self.ctx, on)

    def zero_grads(self):
        A.atom_zero_grads(self.ctx)

    def stats(self):
        return A.atom_get_stats(self.ctx)

    def close(self):
        if self.ctx is not None:
            A.atom_ctx_destroy(self.ctx)
            self.ctx = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
