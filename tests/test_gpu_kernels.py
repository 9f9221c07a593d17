"""Kernel-level parity: each HIP kernel through the C ABI vs the fp64 oracle.

Inputs are seeded, rounded to the working precision before both sides see
them.  Sizes span several tiles and end in ragged tails.  Tolerances
(normwise max-norm relative error, see gpu_util.rel_err):
  * bf16 outputs: one rounding to bf16 (2^-9 relative) on top of an fp32
    accumulation -> 8e-3;
  * fp32 outputs from bf16 inputs: products are exact in fp32, the sums round
    at 2^-24 per add -> 1e-4 for K up to a few thousand;
  * fp32 mode: 1e-5.
"""
import numpy as np
import pytest

from oracle import gpt
from paper_2403_10504_amd import atom as A
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

TOL_OUT = {"bf16": 8e-3, "f32": 1e-5}


def stream():
    return U.torch().cuda.current_stream().cuda_stream


# ---------------------------------------------------------------------- GEMM
def gemm_case(dtype, akc, bkc, M, N, K, epi, seed):
    r = U.rng(seed)
    a_shape = (M, K) if akc else (K, M)
    b_shape = (N, K) if bkc else (K, N)
    Am = U.rep(r.standard_normal(a_shape), dtype)
    Bm = U.rep(r.standard_normal(b_shape), dtype)
    Aop = Am if akc else Am.T
    Bop = Bm.T if bkc else Bm  # [K][N]
    acc = Aop.astype(np.float64) @ Bop.astype(np.float64)
    bias = U.rep(r.standard_normal(N), dtype)
    resid = r.standard_normal((M, N)).astype(np.float32)
    aux = U.rep(r.standard_normal((M, N)), dtype)
    cinit = r.standard_normal((M, N)).astype(np.float32)
    dA, dB = U.dev(Am, dtype), U.dev(Bm, dtype)
    out_f32 = epi in (A.ATOM_EPI_STORE_F32, A.ATOM_EPI_ACC_F32, A.ATOM_EPI_BIAS_RESID)
    dC = U.dev_f32(cinit) if epi == A.ATOM_EPI_ACC_F32 else U.empty((M, N), "f32" if out_f32 else dtype)
    dbias, dres, daux = U.dev(bias, dtype), U.dev_f32(resid), U.dev(aux, dtype)
    if epi == A.ATOM_EPI_BIAS_GELU:
        daux = U.empty((M, N), dtype)
    A.atom_k_gemm(U.dt_code(dtype), akc, bkc, epi, M, N, K, U.ptr(dA), a_shape[1], U.ptr(dB), b_shape[1], U.ptr(dC), N,
                  U.ptr(dbias), U.ptr(dres), U.ptr(daux), N, stream())
    U.sync()
    got = U.host(dC)
    if epi == A.ATOM_EPI_STORE or epi == A.ATOM_EPI_STORE_F32:
        ref = acc
    elif epi == A.ATOM_EPI_ACC_F32:
        ref = cinit + acc
    elif epi == A.ATOM_EPI_BIAS:
        ref = acc + bias
    elif epi == A.ATOM_EPI_BIAS_RESID:
        ref = resid + acc + bias
    elif epi == A.ATOM_EPI_BIAS_GELU:
        u = acc + bias
        assert U.rel_err(U.host(daux), u) < TOL_OUT[dtype]
        ref = gpt.gelu(U.rep(u, dtype).astype(np.float64))
    elif epi == A.ATOM_EPI_GELU_BWD:
        ref = acc * gpt.gelu_grad(aux.astype(np.float64))
    tol = 1e-4 if (out_f32 and dtype == "bf16") else TOL_OUT[dtype]
    return U.rel_err(got, ref), tol


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("akc,bkc", [(1, 1), (1, 0), (0, 0), (0, 1)])
@pytest.mark.parametrize("M,N,K", [(200, 136, 72), (256, 384, 512), (130, 66, 520), (2, 2, 8)])
def test_gemm_layouts(dtype, akc, bkc, M, N, K):
    err, tol = gemm_case(dtype, akc, bkc, M, N, K, A.ATOM_EPI_STORE, seed=M * 7 + N + K)
    assert err < tol, err


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("epi", [A.ATOM_EPI_STORE_F32, A.ATOM_EPI_ACC_F32, A.ATOM_EPI_BIAS, A.ATOM_EPI_BIAS_GELU,
                                 A.ATOM_EPI_BIAS_RESID, A.ATOM_EPI_GELU_BWD])
def test_gemm_epilogues(dtype, epi):
    for akc, bkc in ((1, 1), (1, 0), (0, 0)):
        err, tol = gemm_case(dtype, akc, bkc, 260, 196, 136, epi, seed=epi * 3 + akc + 2 * bkc)
        assert err < tol, (akc, bkc, err)


def sampled_gemm_check(dtype, akc, bkc, M, N, K, ws_bytes=0, seed=0, rows=48):
    """Large GEMM: compare a random sample of full output rows with fp64 dot products."""
    r = U.rng(seed)
    a_shape = (M, K) if akc else (K, M)
    b_shape = (N, K) if bkc else (K, N)
    Am = U.rep(r.standard_normal(a_shape), dtype)
    Bm = U.rep(r.standard_normal(b_shape), dtype)
    dA, dB = U.dev(Am, dtype), U.dev(Bm, dtype)
    dC = U.empty((M, N), "f32")
    ws = U.empty(max(1, ws_bytes // 4), "f32")
    A.atom_k_gemm(U.dt_code(dtype), akc, bkc, A.ATOM_EPI_STORE_F32, M, N, K, U.ptr(dA), a_shape[1], U.ptr(dB),
                  b_shape[1], U.ptr(dC), N, stream=stream(), ws=U.ptr(ws) if ws_bytes else None, ws_bytes=ws_bytes)
    U.sync()
    got = U.host(dC)
    pick = np.sort(r.choice(M, size=min(rows, M), replace=False))
    pick[-1] = M - 1  # always include the ragged last row
    Aop = (Am if akc else Am.T)[pick].astype(np.float64)
    Bop = (Bm.T if bkc else Bm).astype(np.float64)
    return U.rel_err(got[pick], Aop @ Bop), got


@pytest.mark.parametrize("akc,bkc", [(1, 1), (1, 0), (0, 0)])
def test_gemm_large_tile_path(akc, bkc):
    # >= 256 output tiles of 256x256 selects the large-tile kernel; ragged edges
    err, _ = sampled_gemm_check("bf16", akc, bkc, 4100, 4104, 264, seed=akc + 2 * bkc)
    assert err < 1e-4, err


ALL_EPI = [A.ATOM_EPI_STORE, A.ATOM_EPI_STORE_F32, A.ATOM_EPI_ACC_F32, A.ATOM_EPI_BIAS, A.ATOM_EPI_BIAS_GELU,
           A.ATOM_EPI_BIAS_RESID, A.ATOM_EPI_GELU_BWD]


@pytest.mark.parametrize("K", [352, 384, 128])
@pytest.mark.parametrize("akc,bkc", [(1, 1), (1, 0), (0, 0), (0, 1)])
@pytest.mark.parametrize("epi", ALL_EPI)
def test_gemm_pipelined_path(akc, bkc, epi, K):
    """bf16 problems with >= 256 tiles of 256x256 and k a multiple of 32 take the
    four-stage direct-to-LDS kernels: sixteen waves for k = 352, and for k a
    multiple of 128 (384: three loop trips; 128: the prologue's tiles only) the
    four-wave kernel for every epilogue.  M and N end in partial tiles (ragged
    by 8 and 24 rows) whose loads are clamped to the last valid rows and whose
    epilogue takes the bounds-tested copy."""
    check_pipelined(akc, bkc, epi, 4104, 4120, K, seed=akc + 2 * bkc + 4 * epi + K)


@pytest.mark.parametrize("akc,bkc", [(1, 1), (1, 0), (0, 0)])
@pytest.mark.parametrize("epi", [A.ATOM_EPI_STORE, A.ATOM_EPI_BIAS_GELU, A.ATOM_EPI_BIAS_RESID, A.ATOM_EPI_GELU_BWD])
def test_gemm_pipelined_rotated_k(akc, bkc, epi):
    """A whole number of 256x256 tiles per XCD (4096 x 4096: 256 tiles) makes
    the four-wave kernel start each XCD's k loop at its own eighth of k
    (k = 1152: 36 tiles of 32, offsets 0, 4, ..., 28) and takes the
    branch-free epilogue in every tile."""
    check_pipelined(akc, bkc, epi, 4096, 4096, 1152, seed=100 + akc + 2 * bkc + 4 * epi)


@pytest.mark.parametrize("akc,bkc", [(1, 1), (1, 0), (0, 0)])
@pytest.mark.parametrize("M,N,K,epi", [
    (3072, 4096, 1024, A.ATOM_EPI_BIAS_GELU),  # 192 tiles: four waves, no split
    (3072, 4096, 1024, A.ATOM_EPI_GELU_BWD),
    (2048, 2048, 4096, A.ATOM_EPI_STORE),  # 64 tiles: four splits of k
    (1544, 1032, 2048, A.ATOM_EPI_ACC_F32),  # 35 ragged tiles: eight splits
    (1544, 1032, 2048, A.ATOM_EPI_STORE_F32),
    (3072, 768, 16384, A.ATOM_EPI_STORE),  # 36 tiles: eight splits would overflow 64 MB, so four
])
def test_gemm_four_wave_few_tiles(akc, bkc, M, N, K, epi):
    """Fewer 256x256 tiles than CUs: the four-wave kernel takes problems from
    192 tiles on as they are, and fewer tiles over 2-16 ranges of k whose fp32
    partial sums splitk_reduce adds in order (as many splits as bring the
    workgroups to 192, or as the workspace holds if that leaves 96)."""
    seed = 200 + akc + 2 * bkc + 4 * epi + M
    check_pipelined(akc, bkc, epi, M, N, K, seed=seed, ws_bytes=64 << 20)
    if epi == A.ATOM_EPI_STORE_F32:
        # the split sum is deterministic and differs from the unsplit order
        c1 = check_pipelined(akc, bkc, epi, M, N, K, seed=seed, ws_bytes=64 << 20)
        c2 = check_pipelined(akc, bkc, epi, M, N, K, seed=seed, ws_bytes=64 << 20)
        c0 = check_pipelined(akc, bkc, epi, M, N, K, seed=seed, ws_bytes=0)
        assert np.array_equal(c1, c2)
        assert not np.array_equal(c0, c1)


def check_pipelined(akc, bkc, epi, M, N, K, seed, ws_bytes=0):
    r = U.rng(seed)
    a_shape = (M, K) if akc else (K, M)
    b_shape = (N, K) if bkc else (K, N)
    Am = U.rep(r.standard_normal(a_shape), "bf16")
    Bm = U.rep(r.standard_normal(b_shape), "bf16")
    bias = U.rep(r.standard_normal(N), "bf16")
    resid = r.standard_normal((M, N)).astype(np.float32)
    aux = U.rep(r.standard_normal((M, N)), "bf16")
    cinit = r.standard_normal((M, N)).astype(np.float32)
    dA, dB, dbias, dres = U.dev(Am, "bf16"), U.dev(Bm, "bf16"), U.dev(bias, "bf16"), U.dev_f32(resid)
    out_f32 = epi in (A.ATOM_EPI_STORE_F32, A.ATOM_EPI_ACC_F32, A.ATOM_EPI_BIAS_RESID)
    dC = U.dev_f32(cinit) if epi == A.ATOM_EPI_ACC_F32 else U.empty((M, N), "f32" if out_f32 else "bf16")
    daux = U.dev(aux, "bf16") if epi == A.ATOM_EPI_GELU_BWD else U.empty((M, N), "bf16")
    dws = U.empty((ws_bytes // 4,), "f32") if ws_bytes else None
    A.atom_k_gemm(A.ATOM_BF16, akc, bkc, epi, M, N, K, U.ptr(dA), a_shape[1], U.ptr(dB), b_shape[1], U.ptr(dC), N,
                  U.ptr(dbias), U.ptr(dres), U.ptr(daux), N, stream(), ws=U.ptr(dws) if ws_bytes else None,
                  ws_bytes=ws_bytes)
    U.sync()
    pick = np.sort(np.unique(np.concatenate([U.rng(7).choice(M, 40, replace=False), [M - 9, M - 1]])))
    acc = (Am if akc else Am.T)[pick].astype(np.float64) @ (Bm.T if bkc else Bm).astype(np.float64)
    got = U.host(dC)[pick]
    if epi == A.ATOM_EPI_BIAS_GELU:
        u = acc + bias
        assert U.rel_err(U.host(daux)[pick], u) < 8e-3
        ref = gpt.gelu(U.rep(u, "bf16").astype(np.float64))
    elif epi == A.ATOM_EPI_BIAS_RESID:
        ref = resid[pick] + acc + bias
    elif epi == A.ATOM_EPI_ACC_F32:
        ref = cinit[pick] + acc
    elif epi == A.ATOM_EPI_BIAS:
        ref = acc + bias
    elif epi == A.ATOM_EPI_GELU_BWD:
        ref = acc * gpt.gelu_grad(aux[pick].astype(np.float64))
    else:
        ref = acc
    tol = 1e-4 if out_f32 else 8e-3
    assert U.rel_err(got, ref) < tol
    # the last columns (a partial tile) too
    assert U.rel_err(got[:, -24:], ref[:, -24:]) < tol
    return got


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_gemm_split_k_is_exact_and_deterministic(dtype):
    M, N, K = 256, 392, 8192  # few output tiles, long k: splits over k
    ws = 16 * M * N * 4
    err, c1 = sampled_gemm_check(dtype, 0, 0, M, N, K, ws_bytes=ws, seed=5, rows=M)
    assert err < 1e-4, err
    _, c2 = sampled_gemm_check(dtype, 0, 0, M, N, K, ws_bytes=ws, seed=5, rows=8)
    assert np.array_equal(c1, c2)
    err0, c0 = sampled_gemm_check(dtype, 0, 0, M, N, K, ws_bytes=0, seed=5, rows=M)
    assert err0 < 1e-4
    assert not np.array_equal(c0, c1)  # the split path really ran (different summation order)


def test_gemm_rejects_unsupported_shapes():
    t = U.empty((64, 64), "bf16")
    with pytest.raises(A.AtomError):  # K not a multiple of 8
        A.atom_k_gemm(A.ATOM_BF16, 1, 1, 0, 64, 64, 60, U.ptr(t), 64, U.ptr(t), 64, U.ptr(t), 64)
    with pytest.raises(A.AtomError):  # odd rows for a non-k-contiguous bf16 operand
        A.atom_k_gemm(A.ATOM_BF16, 0, 1, 0, 63, 64, 64, U.ptr(t), 64, U.ptr(t), 64, U.ptr(t), 64)


# ----------------------------------------------------------------- LayerNorm
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("rows,d", [(37, 256), (130, 768), (17, 320), (5, 4096), (3, 5120), (4100, 256),
                                    (300, 2048), (1031, 5120), (77, 1088), (16, 8192), (41, 1024)])
def test_layernorm_fwd_bwd(dtype, rows, d):
    r = U.rng(rows + d)
    x = (r.standard_normal((rows, d)) * 2 + 0.5).astype(np.float32)
    g = U.rep(1 + 0.2 * r.standard_normal(d), dtype)
    b = U.rep(0.1 * r.standard_normal(d), dtype)
    dy = U.rep(r.standard_normal((rows, d)), dtype)
    dres0 = r.standard_normal((rows, d)).astype(np.float32)
    y_ref, (xhat, rstd) = gpt.layer_norm(x.astype(np.float64), g, b)
    dx_ref, dg_ref, db_ref = gpt.layer_norm_backward(dy.astype(np.float64), xhat, rstd, g)
    dx, dg_, db_ = U.dev_f32(x), U.dev(g, dtype), U.dev(b, dtype)
    y = U.empty((rows, d), dtype)
    mean, rs = U.empty(rows, "f32"), U.empty(rows, "f32")
    A.atom_k_layernorm_fwd(U.dt_code(dtype), U.ptr(dx), U.ptr(dg_), U.ptr(db_), U.ptr(y), U.ptr(mean), U.ptr(rs),
                           rows, d, stream())
    U.sync()
    assert U.rel_err(U.host(y), y_ref) < TOL_OUT[dtype]
    assert U.rel_err(U.host(rs), rstd[:, 0]) < 1e-5
    assert U.rel_err(U.host(mean), x.astype(np.float64).mean(axis=1)) < 1e-5
    for acc in (0, 1):
        ddy = U.dev(dy, dtype)
        dres = U.dev_f32(dres0)
        lp = U.empty((rows, d), dtype)
        dgam, dbet = U.empty(d, "f32"), U.empty(d, "f32")
        part = U.empty(A.atom_k_layernorm_bwd_part_floats(rows, d), "f32")
        A.atom_k_layernorm_bwd(U.dt_code(dtype), U.ptr(ddy), U.ptr(dx), U.ptr(mean), U.ptr(rs), U.ptr(dg_),
                               U.ptr(dres), U.ptr(lp), acc, U.ptr(dgam), U.ptr(dbet), U.ptr(part), rows, d, stream())
        U.sync()
        ref = dx_ref + (dres0 if acc else 0)
        assert U.rel_err(U.host(dres), ref) < 1e-4
        assert U.rel_err(U.host(lp), ref) < TOL_OUT[dtype]
        assert U.rel_err(U.host(dgam), dg_ref) < 1e-4
        assert U.rel_err(U.host(dbet), db_ref) < 1e-4


# ----------------------------------------------------------------- attention
# ragged T, T = 1, several heads and batches, and long loops (many key and
# query tiles through the two-stage pipelines) at both head sizes; B*H a
# multiple of 8 takes the per-XCD split of the heads in the work-item order
ATTN_CASES = [(2, 100, 2, 64), (1, 128, 3, 128), (1, 1, 1, 64), (2, 200, 1, 128), (1, 64, 2, 64), (1, 257, 1, 64),
              (1, 1000, 2, 128), (2, 600, 1, 64), (2, 300, 4, 64), (1, 520, 16, 128), (4, 130, 6, 64)]


def attn_inputs(B, T, H, dh, dtype, seed):
    r = U.rng(seed)
    d = H * dh
    qkv = U.rep(r.standard_normal((B * T, 3 * d)), dtype)
    do = U.rep(r.standard_normal((B * T, d)), dtype)
    return qkv, do


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("B,T,H,dh", ATTN_CASES)
def test_attention_fwd_bwd(dtype, B, T, H, dh):
    d = H * dh
    qkv, do = attn_inputs(B, T, H, dh, dtype, seed=B * 1000 + T + H + dh)
    o_ref, lse_ref = gpt.causal_attention(qkv.reshape(B, T, 3 * d).astype(np.float64), H)
    dqkv_ref = gpt.causal_attention_backward(do.reshape(B, T, d).astype(np.float64),
                                             qkv.reshape(B, T, 3 * d).astype(np.float64), H)
    dq = U.dev(qkv, dtype)
    o = U.empty((B * T, d), dtype)
    lse = U.empty((B, H, T), "f32")
    A.atom_k_attn_fwd(U.dt_code(dtype), U.ptr(dq), U.ptr(o), U.ptr(lse), B, T, H, dh, stream())
    U.sync()
    # bf16: P is rounded to bf16 before the P V product, then o is stored in bf16
    tol = 1.5e-2 if dtype == "bf16" else 1e-5
    assert U.rel_err(U.host(o), o_ref.reshape(B * T, d)) < tol
    assert np.max(np.abs(U.host(lse) - lse_ref)) < 1e-4 * max(1.0, np.max(np.abs(lse_ref)))
    ddo = U.dev(do, dtype)
    delta = U.empty((B, H, T), "f32")
    dqkv = U.empty((B * T, 3 * d), dtype)
    A.atom_k_attn_bwd(U.dt_code(dtype), U.ptr(dq), U.ptr(o), U.ptr(ddo), U.ptr(lse), U.ptr(delta), U.ptr(dqkv), B, T,
                      H, dh, stream())
    U.sync()
    got = U.host(dqkv).reshape(B, T, 3 * d)
    tol = 2e-2 if dtype == "bf16" else 1e-4
    for part in range(3):
        sl = slice(part * d, (part + 1) * d)
        assert U.rel_err(got[:, :, sl], dqkv_ref[:, :, sl]) < tol, part


# ------------------------------------------------------- cross-entropy etc.
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("rows,V,ld", [(33, 1000, 1024), (5, 50257, 50304), (1, 7, 128), (3, 4097, 4100), (4, 1003, 1003),
                                      (2, 65000, 65536)])
def test_cross_entropy_rows(dtype, rows, V, ld):
    r = U.rng(rows + V)
    z = np.zeros((rows, ld), np.float32)
    z[:, :V] = (r.standard_normal((rows, V)) * 3).astype(np.float32)
    y = r.integers(0, V, rows).astype(np.int32)
    scale = 1.0 / (rows * 4)
    loss_ref, dz_ref = gpt.cross_entropy_rows(z[:, :V].astype(np.float64), y, scale)
    dzt = U.dev_f32(z)
    dy = U.dev_i32(y)
    dz = U.dev(np.full((rows, ld), 7.0, np.float32), dtype)
    loss = U.empty(rows, "f32")
    A.atom_k_xent(U.dt_code(dtype), U.ptr(dzt), ld, U.ptr(dy), U.ptr(dz), ld, U.ptr(loss), rows, V, scale, stream())
    U.sync()
    assert U.rel_err(U.host(loss), loss_ref) < 1e-5
    g = U.host(dz)
    assert U.rel_err(g[:, :V], dz_ref) < TOL_OUT[dtype] + 1e-5
    assert np.all(g[:, V:] == 0)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_colsum(dtype):
    r = U.rng(3)
    for rows, cols in ((1000, 300), (64, 2304), (7, 5), (4100, 64), (130, 12292), (33, 1030)):
        x = U.rep(r.standard_normal((rows, cols)), dtype)
        dx = U.dev(x, dtype)
        out = U.empty(cols, "f32")
        part = U.empty(A.atom_k_colsum_part_floats(rows, cols), "f32")
        A.atom_k_colsum(U.dt_code(dtype), U.ptr(dx), rows, cols, U.ptr(out), U.ptr(part), stream())
        U.sync()
        assert U.rel_err(U.host(out), x.astype(np.float64).sum(axis=0)) < 1e-5


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_embedding_forward(dtype):
    r = U.rng(4)
    V, T, d, B = 300, 50, 128, 3
    wte = U.rep(r.standard_normal((V, d)), dtype)
    wpe = U.rep(r.standard_normal((T, d)), dtype)
    tok = r.integers(0, V, (B, T)).astype(np.int32)
    ref = gpt.embed_forward(tok, {"wte": wte, "wpe": wpe}).reshape(B * T, d)
    # every device buffer stays referenced until the kernel has finished
    dtok, dwte, dwpe = U.dev_i32(tok), U.dev(wte, dtype), U.dev(wpe, dtype)
    x = U.empty((B * T, d), "f32")
    A.atom_k_embed_fwd(U.dt_code(dtype), U.ptr(dtok), U.ptr(dwte), U.ptr(dwpe), U.ptr(x), B * T, T, V, d, stream())
    U.sync()
    assert U.rel_err(U.host(x), ref) < 1e-7
    # an id outside [0, V) yields a NaN row, never an out-of-range read
    bad = tok.copy()
    bad[1, 3] = V
    bad[2, 0] = -5
    dbad = U.dev_i32(bad)
    A.atom_k_embed_fwd(U.dt_code(dtype), U.ptr(dbad), U.ptr(dwte), U.ptr(dwpe), U.ptr(x), B * T, T, V, d, stream())
    U.sync()
    got = U.host(x).reshape(B, T, d)
    assert np.all(np.isnan(got[1, 3])) and np.all(np.isnan(got[2, 0]))
    assert np.array_equal(np.isnan(got).any(axis=2), (bad < 0) | (bad >= V))
