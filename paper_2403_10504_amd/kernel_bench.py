"""Times single kernels through the C ABI on seeded inputs (for profiling).

python -m paper_2403_10504_amd.kernel_bench attention [fwd|bwd|all] [iters]
python -m paper_2403_10504_amd.kernel_bench gemm [iters]
python -m paper_2403_10504_amd.kernel_bench gemm_layouts [iters]
python -m paper_2403_10504_amd.kernel_bench layernorm [iters]
python -m paper_2403_10504_amd.kernel_bench xent [iters]

attention: causal attention at the 6.7B shape (B 2, T 2048, 32 heads of 128),
GPT-3 Small's (B 8, 12 heads of 64) and 13B's (B 1, 40 heads of 128); the
forward output is checked against a plain fp32 torch computation.
gemm: the weight-gradient GEMM (neither operand k-contiguous, bf16 store) at
the 6.7B layer shapes for k = 2048, 4096, 8192, with the fit t = a + b k.
gemm_layouts: the 6.7B block's GEMMs in the three operand layouts the step
uses (forward, data gradient, weight gradient), store epilogue.
layernorm: the LayerNorm backward (accumulate, bf16 copy, both partial sums)
and forward (bf16 output, row statistics) at the four GPT-3 widths.  One line per measurement; times from HIP events.
"""
from __future__ import annotations

import sys

import torch

from . import atom as A

ATTN_SHAPES = [(2, 2048, 32, 128), (8, 2048, 12, 64), (1, 2048, 40, 128)]


def _time(fn, iters):
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(iters):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1000 / iters


def _attn_reference(qkv, B, T, H, dh):
    x = qkv.float().view(B, T, 3, H, dh)
    q = x[:, :, 0].permute(0, 2, 1, 3).contiguous()
    kt = x[:, :, 1].permute(0, 2, 3, 1).contiguous()
    v = x[:, :, 2].permute(0, 2, 1, 3).contiguous()
    s = torch.matmul(q, kt) / dh ** 0.5
    s.masked_fill_(torch.ones(T, T, device=s.device, dtype=torch.bool).triu(1), float("-inf"))
    return torch.matmul(torch.softmax(s, -1), v).permute(0, 2, 1, 3).reshape(B * T, H * dh)


def attention(which="all", iters=20):
    for B, T, H, dh in ATTN_SHAPES:
        d = H * dh
        g = torch.Generator(device="cuda").manual_seed(1)
        qkv = (torch.randn(B * T, 3 * d, device="cuda", generator=g) * 0.5).to(torch.bfloat16)
        o = torch.empty(B * T, d, device="cuda", dtype=torch.bfloat16)
        lse = torch.empty(B * H * T, device="cuda")
        dout = (torch.randn(B * T, d, device="cuda", generator=g) * 0.1).to(torch.bfloat16)
        delta = torch.empty(B * H * T, device="cuda")
        dqkv = torch.empty_like(qkv)
        fwd = lambda: A.atom_k_attn_fwd(1, qkv.data_ptr(), o.data_ptr(), lse.data_ptr(), B, T, H, dh)
        bwd = lambda: A.atom_k_attn_bwd(1, qkv.data_ptr(), o.data_ptr(), dout.data_ptr(), lse.data_ptr(),
                                        delta.data_ptr(), dqkv.data_ptr(), B, T, H, dh)
        fwd()
        torch.cuda.synchronize()
        ref = _attn_reference(qkv, B, T, H, dh)
        err = ((o.float() - ref).abs().max() / ref.abs().max()).item()
        del ref
        if not err < 1.5e-2:
            raise RuntimeError(f"attention forward off by {err} at B={B} T={T} H={H} dh={dh}")
        flop = 2 * 2 * B * H * T * T * dh / 2  # two causal products
        for name, fn, mult in (("fwd", fwd, 1.0), ("bwd", bwd, 2.5)):
            if which in ("all", name):
                us = _time(fn, iters)
                print(f"attention {name} B={B} T={T} H={H} dh={dh}: {us:.1f} us, "
                      f"{flop * mult / us / 1e6:.0f} TFLOP/s (algorithmic)", flush=True)


def gemm_layouts(iters=20):
    """The 6.7B block's GEMM shapes in every operand layout the step uses (store epilogue)."""
    tok, d, f = 4096, 4096, 16384
    cases = [("forward QKV", 1, 1, tok, 3 * d, d), ("forward O", 1, 1, tok, d, d), ("forward FC", 1, 1, tok, f, d),
             ("forward PR", 1, 1, tok, d, f), ("data grad QKV", 1, 0, tok, d, 3 * d), ("data grad FC", 1, 0, tok, d, f),
             ("data grad PR", 1, 0, tok, f, d), ("weight grad QKV", 0, 0, 3 * d, d, tok),
             ("weight grad FC", 0, 0, f, d, tok), ("weight grad PR", 0, 0, d, f, tok)]
    for name, akc, bkc, M, N, K in cases:
        # A(m, k) = A[m*lda + k] if k-contiguous else A[k*lda + m]; likewise B(k, n)
        a = (torch.randn(M * K, device="cuda") * 0.05).to(torch.bfloat16)
        b = (torch.randn(N * K, device="cuda") * 0.05).to(torch.bfloat16)
        c = torch.empty(M, N, device="cuda", dtype=torch.bfloat16)
        lda, ldb = (K if akc else M), (K if bkc else N)
        us = _time(lambda: A.atom_k_gemm(1, akc, bkc, A.ATOM_EPI_STORE, M, N, K, a.data_ptr(), lda, b.data_ptr(), ldb,
                                         c.data_ptr(), N), iters)
        print(f"gemm {name} (A k-contiguous {akc}, B k-contiguous {bkc}) {M}x{N}x{K}: {us:.1f} us, "
              f"{2 * M * N * K / us / 1e6:.0f} TFLOP/s", flush=True)
        del a, b, c


def gemm(iters=20):
    for M, N in ((4096, 16384), (16384, 4096), (4096, 4096), (12288, 4096), (50304, 4096)):
        res = []
        for K in (2048, 4096, 8192):
            a = (torch.randn(K, M, device="cuda") * 0.05).to(torch.bfloat16)
            b = (torch.randn(K, N, device="cuda") * 0.05).to(torch.bfloat16)
            c = torch.empty(M, N, device="cuda", dtype=torch.bfloat16)
            us = _time(lambda: A.atom_k_gemm(1, 0, 0, A.ATOM_EPI_STORE, M, N, K, a.data_ptr(), M, b.data_ptr(), N,
                                             c.data_ptr(), N), iters)
            res.append((K, us))
            print(f"gemm wgrad M={M} N={N} K={K}: {us:.1f} us, {2 * M * N * K / us / 1e6:.0f} TFLOP/s", flush=True)
            del a, b, c
        (k1, t1), _, (k3, t3) = res
        slope = (t3 - t1) / (k3 - k1)
        print(f"gemm wgrad M={M} N={N}: t = {t1 - slope * k1:.1f} us + k x {slope * 1e3:.2f} ns "
              f"(k loop alone {2 * M * N / slope / 1e6:.0f} TFLOP/s)", flush=True)


def layernorm(iters=50):
    for rows, d in ((4096, 4096), (8192, 2048), (2048, 5120), (16384, 768)):
        dy = torch.randn(rows, d, device="cuda").to(torch.bfloat16)
        x = torch.randn(rows, d, device="cuda")
        mean = x.mean(1).contiguous()
        rs = (1 / (x.var(1, unbiased=False) + 1e-5).sqrt()).contiguous()
        gm = torch.ones(d, device="cuda").to(torch.bfloat16)
        dres = torch.randn(rows, d, device="cuda")
        lp = torch.empty(rows, d, device="cuda", dtype=torch.bfloat16)
        dgam = torch.empty(d, device="cuda")
        dbet = torch.empty(d, device="cuda")
        part = torch.empty(A.atom_k_layernorm_bwd_part_floats(rows, d), device="cuda")
        us = _time(lambda: A.atom_k_layernorm_bwd(1, dy.data_ptr(), x.data_ptr(), mean.data_ptr(), rs.data_ptr(),
                                                  gm.data_ptr(), dres.data_ptr(), lp.data_ptr(), 1, dgam.data_ptr(),
                                                  dbet.data_ptr(), part.data_ptr(), rows, d, None), iters)
        alg = rows * d * (2 + 4 + 4 + 4 + 2)
        print(f"layernorm bwd rows={rows} d={d}: {us:.1f} us, {alg / us / 1e3:.0f} GB/s algorithmic", flush=True)
        bt = torch.zeros(d, device="cuda").to(torch.bfloat16)
        us = _time(lambda: A.atom_k_layernorm_fwd(1, x.data_ptr(), gm.data_ptr(), bt.data_ptr(), lp.data_ptr(),
                                                  mean.data_ptr(), rs.data_ptr(), rows, d, None), iters)
        alg = rows * (d * (4 + 2) + 8)
        print(f"layernorm fwd rows={rows} d={d}: {us:.1f} us, {alg / us / 1e3:.0f} GB/s algorithmic", flush=True)


def xent(iters=20):
    """The LM head's cross-entropy over 2048-row chunks of fp32 logits (GPT-3 vocabulary)."""
    for rows, V, ld in ((2048, 50257, 50304), (4096, 50257, 50304)):
        z = torch.randn(rows, ld, device="cuda") * 3
        tgt = torch.randint(0, V, (rows,), device="cuda", dtype=torch.int32)
        dz = torch.empty(rows, ld, device="cuda", dtype=torch.bfloat16)
        loss = torch.empty(rows, device="cuda")
        us = _time(lambda: A.atom_k_xent(1, z.data_ptr(), ld, tgt.data_ptr(), dz.data_ptr(), ld, loss.data_ptr(), rows,
                                         V, 1.0 / rows), iters)
        alg = rows * ld * (4 + 2)
        print(f"xent rows={rows} V={V}: {us:.1f} us, {alg / us / 1e3:.0f} GB/s algorithmic "
              f"(fp32 logits read once, bf16 dz written once)", flush=True)


def main(argv):
    if not torch.cuda.is_available():
        raise SystemExit("kernel_bench needs a GPU")
    what = argv[1] if len(argv) > 1 else "attention"
    if what == "attention":
        attention(argv[2] if len(argv) > 2 else "all", int(argv[3]) if len(argv) > 3 else 20)
    elif what == "gemm":
        gemm(int(argv[2]) if len(argv) > 2 else 20)
    elif what == "gemm_layouts":
        gemm_layouts(int(argv[2]) if len(argv) > 2 else 20)
    elif what == "xent":
        xent(int(argv[2]) if len(argv) > 2 else 20)
    elif what == "layernorm":
        layernorm(int(argv[2]) if len(argv) > 2 else 50)
    else:
        raise SystemExit(f"unknown kernel family {what!r}")


if __name__ == "__main__":
    main(sys.argv)
