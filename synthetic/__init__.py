"""Seeded synthetic inputs for the swapped GPT training step.

This module is the only code shared by the oracle and the GPU path.  It holds
no arithmetic of the method: it names the model configurations, lists the
parameter tensors of each node of the layer chain, and draws seeded random
numbers for them.

Recipe (the paper trains minGPT-style GPT-3 models, Section III-B, and gives
the shapes in Table II; the paper prints no initialisation, so this one is a
stated choice):

* weight matrices and both embeddings ~ N(0, 0.02), biases 0, LayerNorm gain 1
  and shift 0, no residual-projection rescaling;
* tokens uniform over the vocabulary, shape [accum][batch][seq_len + 1]; the
  inputs are [..., :T] and the next-token targets are [..., 1:T+1];
* in bf16 mode the drawn fp32 values are rounded to the nearest bfloat16 (ties
  to even) here, so both sides consume the same bf16-representable weights.

Every tensor is drawn from its own PCG64 stream keyed by (seed, node, tensor
index, chunk), so the values do not depend on how many threads fill them.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

F32 = "f32"
BF16 = "bf16"

WEIGHT_SEED = 1234
TOKEN_SEED = 5678
INIT_STD = 0.02

_CHUNK = 1 << 22  # elements per independent random stream


@dataclasses.dataclass(frozen=True)
class Config:
    """Shape of one GPT model and one training step."""

    name: str
    n_layer: int
    d_model: int
    n_head: int
    d_mlp: int
    vocab: int
    seq_len: int
    batch: int
    accum: int = 1
    dtype: str = BF16
    budget_bytes: int = 0  # 0 = whole model may stay resident
    ckpt_host: bool = False  # block-input checkpoints kept in host memory

    @property
    def n_nodes(self) -> int:
        return self.n_layer + 2

    @property
    def d_head(self) -> int:
        return self.d_model // self.n_head

    @property
    def tokens_per_micro(self) -> int:
        return self.batch * self.seq_len

    @property
    def tokens_per_step(self) -> int:
        return self.accum * self.batch * self.seq_len

    def with_(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


GIB = 1 << 30

CONFIGS = {
    # Tiny decoder used for exact fp32 parity (budget of one block forces swapping).
    "tiny": Config("tiny", 2, 256, 4, 1024, 1024, 128, 2, 1, F32, 0),
    # GPT-3 Small (125M), resident.
    "small": Config("small", 12, 768, 12, 3072, 50257, 2048, 8, 1, BF16, 0),
    # GPT-3 XL (1.3B) with 16 heads, device budget 8 GB.
    "xl": Config("xl", 24, 2048, 16, 8192, 50257, 2048, 4, 1, BF16, 8 * 10**9),
    # GPT-3 6.7B, device budget 24 GB.
    "6.7b": Config("6.7b", 32, 4096, 32, 16384, 50257, 2048, 2, 1, BF16, 24 * 10**9),
    # GPT-3 13B, device budget 24 GB, checkpoints on the host.
    "13b": Config("13b", 40, 5120, 40, 20480, 50257, 2048, 1, 1, BF16, 24 * 10**9, True),
}


def param_specs(cfg: Config, node: int):
    """List of (name, shape, init) for node `node` of the layer chain.

    Node 0 is the embedding, nodes 1..L are decoder blocks, node L+1 is the
    final LayerNorm plus the LM head ("Logits").  Linear weights are stored
    [out][in], so a linear layer computes y = x W^T + b.
    """
    d, f, V, T = cfg.d_model, cfg.d_mlp, cfg.vocab, cfg.seq_len
    if node == 0:
        return [("wte", (V, d), "normal"), ("wpe", (T, d), "normal")]
    if 1 <= node <= cfg.n_layer:
        return [
            ("ln1_g", (d,), "one"), ("ln1_b", (d,), "zero"),
            ("w_qkv", (3 * d, d), "normal"), ("b_qkv", (3 * d,), "zero"),
            ("w_o", (d, d), "normal"), ("b_o", (d,), "zero"),
            ("ln2_g", (d,), "one"), ("ln2_b", (d,), "zero"),
            ("w_fc", (f, d), "normal"), ("b_fc", (f,), "zero"),
            ("w_pr", (d, f), "normal"), ("b_pr", (d,), "zero"),
        ]
    if node == cfg.n_layer + 1:
        return [("lnf_g", (d,), "one"), ("lnf_b", (d,), "zero"), ("w_head", (V, d), "normal")]
    raise ValueError(f"node {node} out of range for {cfg.n_nodes} nodes")


def round_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bfloat16 bit patterns (uint16), round to nearest, ties to even.

    Inputs are finite draws of a normal distribution; NaN handling is not needed.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _draw_chunk(seed, node, tidx, chunk, n, std):
    ss = np.random.SeedSequence([seed, node, tidx, chunk])
    g = np.random.Generator(np.random.PCG64(ss))
    out = g.standard_normal(n, dtype=np.float32)
    out *= np.float32(std)
    return out


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def fill_param(out: np.ndarray, cfg: Config, node: int, name: str, seed: int = WEIGHT_SEED) -> None:
    """Write parameter `name` of `node` into `out` (flat view).

    `out` is float32 (fp32 mode, or bf16-representable values for a fp32
    consumer) or uint16 (bf16 bit patterns).  Large tensors are filled by a
    thread pool; numpy's generators release the GIL while drawing.
    """
    specs = param_specs(cfg, node)
    tidx = [s[0] for s in specs].index(name)
    _, shape, init = specs[tidx]
    n = int(np.prod(shape))
    flat = out.reshape(-1)
    if flat.size != n:
        raise ValueError(f"{name}: buffer has {flat.size} elements, expected {n}")
    as_bits = flat.dtype == np.uint16
    if init != "normal":
        val = 1.0 if init == "one" else 0.0
        if as_bits:
            flat[:] = round_to_bf16_bits(np.array([val], np.float32))[0]
        else:
            flat[:] = val
        return
    round_bf16 = as_bits or cfg.dtype == BF16

    def job(c):
        lo = c * _CHUNK
        hi = min(n, lo + _CHUNK)
        vals = _draw_chunk(seed, node, tidx, c, hi - lo, INIT_STD)
        if as_bits:
            flat[lo:hi] = round_to_bf16_bits(vals)
        elif round_bf16:
            flat[lo:hi] = bf16_bits_to_f32(round_to_bf16_bits(vals))
        else:
            flat[lo:hi] = vals

    n_chunks = (n + _CHUNK - 1) // _CHUNK
    if n_chunks == 1:
        job(0)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(job, range(n_chunks)))


def gen_param(cfg: Config, node: int, name: str, seed: int = WEIGHT_SEED) -> np.ndarray:
    shape = dict((s[0], s[1]) for s in param_specs(cfg, node))[name]
    out = np.empty(shape, np.float32)
    fill_param(out, cfg, node, name, seed)
    return out


def gen_weights(cfg: Config, seed: int = WEIGHT_SEED):
    """All parameters as float32 arrays: list over nodes of {name: array}."""
    return [
        {name: gen_param(cfg, node, name, seed) for name, _, _ in param_specs(cfg, node)}
        for node in range(cfg.n_nodes)
    ]


def gen_tokens(cfg: Config, seed: int = TOKEN_SEED) -> np.ndarray:
    """Uniform token ids, int32 [accum][batch][seq_len + 1]."""
    g = np.random.Generator(np.random.PCG64(seed))
    return g.integers(0, cfg.vocab, size=(cfg.accum, cfg.batch, cfg.seq_len + 1), dtype=np.int32)


def param_count(cfg: Config) -> int:
    return sum(int(np.prod(s)) for node in range(cfg.n_nodes) for _, s, _ in param_specs(cfg, node))
