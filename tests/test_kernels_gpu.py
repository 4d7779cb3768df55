"""Per-kernel parity of the HIP path (through the C ABI) against the oracle.

Every case feeds the same bf16 inputs to the GPU entry point and to the
float64 oracle.  GEMM layout tests use small-integer inputs so that fp32
accumulation and bf16 rounding are exact: the GPU result must then equal
the oracle bit for bit.  Floating-point cases use the parity bar
max|gpu - ref| / max|ref| <= 2e-2 (activations) or 5e-2 (gradients).
Output buffers carry guard bands that must stay untouched.
"""

import numpy as np
import pytest
import torch

import oracle
from helpers import TOL_ACT, TOL_GRAD, announce, cuda, exact_equal, f64, guard_intact, guarded, max_rel
from paper_2408_03505_amd import binding as B
from paper_2408_03505_amd.synthetic import random_bf16, random_int_bf16, random_sparse_sign_bf16

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

# --------------------------------------------------------------------------- LayerNorm

LN_SHAPES = [(394, 192), (1000, 768), (97, 1280), (2048, 6144), (5, 16384), (3, 8), (1, 64)]


@pytest.mark.parametrize("rows,cols", LN_SHAPES)
def test_ln_fwd(rows, cols):
    announce(f"ln_fwd rows={rows} cols={cols}")
    x = random_bf16((rows, cols), 1, 2.0) + 0.5
    x = x.to(torch.bfloat16)
    g = (1 + random_bf16((cols,), 2, 0.2).float()).to(torch.bfloat16)
    b = random_bf16((cols,), 3, 0.2)
    y, ybuf = guarded((rows, cols), torch.bfloat16)
    mean, mbuf = guarded((rows,), torch.float32)
    rstd, rbuf = guarded((rows,), torch.float32)
    B.enc_ln_fwd(cuda(x), cuda(g), cuda(b), 1e-6, y=y, mean=mean, rstd=rstd)
    torch.cuda.synchronize()
    ry, rm, rr = oracle.layernorm_fwd(f64(x), f64(g), f64(b), 1e-6)
    assert max_rel(f64(y), ry) < TOL_ACT
    assert np.abs(f64(mean) - rm).max() < 1e-5 * max(1.0, np.abs(rm).max())
    assert np.abs(f64(rstd) / rr - 1).max() < 1e-5
    assert guard_intact(ybuf, rows * cols) and guard_intact(mbuf, rows) and guard_intact(rbuf, rows)


# widths cover one wave per row (1-4 chunks per thread), a block per row (3, 5
# and 8 chunks: the last without the next row loaded ahead), a single row and
# row counts that leave the last block short
@pytest.mark.parametrize("rows,cols", [(394, 192), (1000, 768), (300, 6144), (7, 1280), (260, 2048), (70, 16384),
                                       (33, 10240), (1, 8), (2049, 4104)])
@pytest.mark.parametrize("with_resid", [True, False])
def test_ln_bwd(rows, cols, with_resid):
    announce(f"ln_bwd rows={rows} cols={cols} resid={with_resid}")
    x = (random_bf16((rows, cols), 11, 1.5).float() - 0.3).to(torch.bfloat16)
    g = (1 + random_bf16((cols,), 12, 0.2).float()).to(torch.bfloat16)
    b = random_bf16((cols,), 13, 0.2)
    dy = random_bf16((rows, cols), 14)
    dres = random_bf16((rows, cols), 15) if with_resid else None
    _, mean, rstd = B.enc_ln_fwd(cuda(x), cuda(g), cuda(b), 1e-6)
    dx, dxbuf = guarded((rows, cols), torch.bfloat16)
    dg = torch.full((cols,), 0.25, device="cuda")
    db = torch.full((cols,), -0.5, device="cuda")
    B.enc_ln_bwd(cuda(dy), cuda(x), mean, rstd, cuda(g), dresid=cuda(dres) if dres is not None else None,
                 dx=dx, dgamma=dg, dbeta=db, accumulate=True)
    torch.cuda.synchronize()
    # the oracle's backward uses its own statistics of the same bf16 x
    _, rm, rr = oracle.layernorm_fwd(f64(x), f64(g), f64(b), 1e-6)
    rdx, rdg, rdb = oracle.layernorm_bwd(f64(dy), f64(x), rm, rr, f64(g))
    if dres is not None:
        rdx = rdx + f64(dres)
    assert max_rel(f64(dx), rdx) < TOL_GRAD
    assert max_rel(f64(dg) - 0.25, rdg) < TOL_GRAD
    assert max_rel(f64(db) + 0.5, rdb) < TOL_GRAD
    assert guard_intact(dxbuf, rows * cols)


# --------------------------------------------------------------------------- GEMM layouts (exact)

# (M, K_in, N_out) covering one tile, many tiles, ragged rows, K not a
# multiple of the 64-wide k-step (register-staged path), each tile
# configuration of the direct-to-LDS path (256x256, 256x192, 128x128), and
# both workgroup orders: one contiguous range per XCD (e.g. 16x18 tiles) and
# XCDs in two halves along M, including a short last group of row tiles
# (1536x1536: 12x12 tiles, 6 row tiles per half in groups of 4).
# The last three split their contraction (at most 32 output tiles of 256 x 256,
# K >= 1024), one with a ragged M.
FWD_SHAPES = [(394, 192, 576), (300, 200, 1280), (2048, 768, 2304), (2000, 72, 16384), (33, 8, 8),
              (2048, 256, 16384), (1000, 96, 4096), (2048, 128, 6144), (1536, 128, 1536), (2048, 64, 24576),
              (2048, 6144, 1024), (2048, 6144, 768), (1000, 2048, 512),
              # 256x192 tiles with a contraction past 8192: the uneven-ring kernel, ragged M
              (2000, 8256, 6144)]


def _sparse(shape, seed, density):
    return random_sparse_sign_bf16(shape, seed, density)


def _density(K):
    # keep |sum| well inside bf16's exact-integer range (<= 256)
    return min(0.5, float(np.sqrt(24.0 / K)))


@pytest.mark.parametrize("M,K,N", FWD_SHAPES)
def test_qkv_fwd_exact(M, K, N):
    announce(f"qkv_fwd exact M={M} K={K} N={N}")
    N3 = (N // 24) * 24 or 24  # 3A with A a multiple of 8
    d = _density(K)
    X, W = _sparse((M, K), 21, d), _sparse((N3, K), 22, d)
    b = random_int_bf16((N3,), 23, -3, 3)
    Y, buf = guarded((M, N3), torch.bfloat16)
    B.enc_qkv_fwd(cuda(X), cuda(W), cuda(b), qkv=Y)
    torch.cuda.synchronize()
    ok, err = exact_equal(Y, oracle.linear_fwd(f64(X), f64(W), f64(b)))
    assert ok, err
    assert guard_intact(buf, M * N3)


@pytest.mark.parametrize("M,K,N", FWD_SHAPES)
def test_oproj_and_mlp_down_fwd_exact(M, K, N):
    announce(f"oproj/mlp_down exact M={M} K={K} N={N}")
    d = _density(K)
    X, W = _sparse((M, K), 31, d), _sparse((N, K), 32, d)
    b = random_int_bf16((N,), 33, -3, 3)
    R = random_int_bf16((M, N), 34, -8, 8)
    want = oracle.linear_fwd(f64(X), f64(W), f64(b), resid=f64(R))
    Y, buf = guarded((M, N), torch.bfloat16)
    B.enc_oproj_fwd(cuda(X), cuda(W), cuda(b), cuda(R), h=Y)
    torch.cuda.synchronize()
    ok, err = exact_equal(Y, want)
    assert ok, err
    assert guard_intact(buf, M * N)
    Y2 = B.enc_mlp_down_fwd(cuda(X), cuda(W), cuda(b), cuda(R))
    torch.cuda.synchronize()
    ok, err = exact_equal(Y2, want)
    assert ok, err


@pytest.mark.parametrize("M,K,N", FWD_SHAPES[:4] + FWD_SHAPES[5:])
def test_mlp_up_fwd(M, K, N):
    announce(f"mlp_up exact M={M} K={K} N={N}")
    d = _density(K)
    X, W = _sparse((M, K), 41, d), _sparse((N, K), 42, d)
    b = random_int_bf16((N,), 43, -3, 3)
    u, ubuf = guarded((M, N), torch.bfloat16)
    g, gbuf = guarded((M, N), torch.bfloat16)
    B.enc_mlp_up_fwd(cuda(X), cuda(W), cuda(b), u=u, g=g)
    torch.cuda.synchronize()
    ru = oracle.linear_fwd(f64(X), f64(W), f64(b))
    ok, err = exact_equal(u, ru)
    assert ok, err
    rg = oracle.gelu(ru)
    # GELU is applied to the fp32 accumulator, then rounded to bf16
    assert np.abs(f64(g) - rg).max() <= np.abs(rg).max() * 2 ** -8 + 1e-6
    assert guard_intact(ubuf, M * N) and guard_intact(gbuf, M * N)


# dgrad: dX[M, K] = dY[M, N] W[N, K]
# The last three split their contraction (the ViT-22B shard's out-projection
# input gradient, a 32-tile output, a ragged M).
BWD_DATA_SHAPES = [(394, 576, 192), (300, 1280, 200), (2048, 2304, 768), (2000, 256, 16384), (9, 8, 8),
                   (2048, 96, 6144), (2048, 128, 6144), (2048, 6144, 768), (2048, 6144, 1024), (1000, 2048, 512),
                   # 256x192 tiles with a contraction past 20480: the ping-pong kernel, ragged M
                   (2000, 20544, 6144)]


@pytest.mark.parametrize("M,N,K", BWD_DATA_SHAPES)
def test_bwd_data_exact(M, N, K):
    announce(f"bwd_data exact M={M} N={N} K={K}")
    d = _density(N)
    dY, W = _sparse((M, N), 51, d), _sparse((N, K), 52, d)
    want = oracle.linear_bwd_data(f64(dY), f64(W))
    # MLP up: dy2[M, H] = du[M, F] W1[F, H]   (F = N, H = K)
    out, buf = guarded((M, K), torch.bfloat16)
    B.enc_mlp_up_bwd_data(cuda(dY), cuda(W), dy2=out)
    torch.cuda.synchronize()
    ok, err = exact_equal(out, want)
    assert ok, err
    assert guard_intact(buf, M * K)
    # output projection: dO[M, A] = dh[M, H] Wo[H, A]   (H = N, A = K)
    ok, err = exact_equal(B.enc_oproj_bwd_data(cuda(dY), cuda(W)), want)
    assert ok, err
    # MLP down with GELU'(u) == 1 exactly (u = 8): du = dout W2
    u = torch.full((M, K), 8.0, dtype=torch.bfloat16)
    ok, err = exact_equal(B.enc_mlp_down_bwd_data(cuda(dY), cuda(W), cuda(u)), want)
    assert ok, err
    if N % 3 == 0 and (N // 3) % 8 == 0:
        ok, err = exact_equal(B.enc_qkv_bwd_data(cuda(dY), cuda(W)), want)
        assert ok, err


SPLIT_PRODUCTS = [("qkv_fwd", 2048, 6144, 768), ("mlp_up_fwd", 2048, 6144, 1024), ("oproj_fwd", 1000, 2048, 512),
                  ("mlp_down_bwd_data", 2048, 6144, 1024), ("oproj_bwd_data", 2048, 6144, 768),
                  ("qkv_bwd_data", 2048, 2304, 1024)]


@pytest.mark.parametrize("kind,M,Kc,N", SPLIT_PRODUCTS)
def test_split_product_matches_unsplit(kind, M, Kc, N):
    # Output [M, N], contraction Kc.  The split path (workspace given) and the
    # unsplit kernel compute the same product and epilogue: both within bf16
    # rounding of float64, the split path bitwise repeatable.
    announce(f"split vs unsplit {kind} M={M} K={Kc} N={N}")
    assert B.linear_workspace_bytes(M, N, Kc) > 0
    X = cuda(random_bf16((M, Kc), 121))
    if kind.endswith("_fwd"):
        W = cuda(random_bf16((N, Kc), 122, 0.05))
        b = cuda(random_bf16((N,), 123, 0.1))
        R = cuda(random_bf16((M, N), 124))
        fn = {"qkv_fwd": lambda split: B.enc_qkv_fwd(X, W, b, split=split),
              "mlp_up_fwd": lambda split: B.enc_mlp_up_fwd(X, W, b, split=split),
              "oproj_fwd": lambda split: B.enc_oproj_fwd(X, W, b, R, split=split)}[kind]
        ref = oracle.linear_fwd(f64(X), f64(W), f64(b), resid=f64(R) if kind == "oproj_fwd" else None)
    else:
        W = cuda(random_bf16((Kc, N), 122, 0.05))
        U = cuda(random_bf16((M, N), 125, 1.5))
        fn = {"mlp_down_bwd_data": lambda split: B.enc_mlp_down_bwd_data(X, W, U, split=split),
              "oproj_bwd_data": lambda split: B.enc_oproj_bwd_data(X, W, split=split),
              "qkv_bwd_data": lambda split: B.enc_qkv_bwd_data(X, W, split=split)}[kind]
        ref = oracle.linear_bwd_data(f64(X), f64(W))
        if kind == "mlp_down_bwd_data":
            ref = ref * oracle.gelu_grad(f64(U))
    a, a2, u0 = fn(True), fn(True), fn(False)
    torch.cuda.synchronize()
    if kind == "mlp_up_fwd":  # (u, g): check u against the product, g against GELU(u)
        assert torch.equal(a[0], a2[0]) and torch.equal(a[1], a2[1])
        for got in (a, u0):
            assert max_rel(f64(got[0]), ref) < 1e-2
            assert max_rel(f64(got[1]), oracle.gelu(ref)) < 1e-2
    else:
        assert torch.equal(a, a2)
        for got in (a, u0):
            assert max_rel(f64(got), ref) < 1e-2


def _bf16_ulp(v):
    a = np.maximum(np.abs(v), 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(a)) - 7)


def test_gelu_epilogues_within_one_bf16_ulp():
    # u = bias exactly (zero activations), so g = GELU(u) and, with a unit
    # product, du = GELU'(u).  The epilogue's erf is a polynomial
    # approximation: both must be within one bf16 step of the exact float64
    # value for u >= -4, and within 1e-6 absolute over [-8, 8] (below -4 the
    # values are under 1.3e-4 and the approximation's absolute error governs).
    announce("GELU / GELU' epilogue accuracy")
    M, K, N = 64, 64, 4096
    b = torch.linspace(-8.0, 8.0, N).to(torch.bfloat16)
    X = torch.zeros((M, K), dtype=torch.bfloat16)
    W = random_bf16((N, K), 71)
    u, g = B.enc_mlp_up_fwd(cuda(X), cuda(W), cuda(b))
    # GELU': dout = e_0 rows and W2 row 0 = 1 give a product of exactly 1
    H = 64
    dout = torch.zeros((M, H), dtype=torch.bfloat16)
    dout[:, 0] = 1
    w2 = torch.zeros((H, N), dtype=torch.bfloat16)
    w2[0, :] = 1
    du = B.enc_mlp_down_bwd_data(cuda(dout), cuda(w2), cuda(b.expand(M, N).contiguous()))
    torch.cuda.synchronize()
    bu = f64(b)
    assert np.array_equal(f64(u), np.broadcast_to(bu, (M, N)))
    main = bu >= -4.0
    for got, exact in ((f64(g), oracle.gelu(bu)), (f64(du), oracle.gelu_grad(bu))):
        err = np.abs(got - exact)
        assert err.max() <= 1e-6 + np.abs(exact).max() * 2.0 ** -8, err.max()
        ref = f64(torch.from_numpy(exact).to(torch.bfloat16))
        assert np.all(np.abs(got - ref)[:, main] <= _bf16_ulp(ref)[main]), np.abs(got - ref)[:, main].max()
        assert np.all(err[:, ~main] <= 1e-6), err[:, ~main].max()


def test_mlp_down_bwd_data_gelu_grad():
    announce("mlp_down_bwd_data gelu' epilogue")
    M, H, F = 394, 192, 768
    dout = random_bf16((M, H), 61)
    w2 = random_bf16((H, F), 62, 0.05)
    u = random_bf16((M, F), 63, 1.5)
    du = B.enc_mlp_down_bwd_data(cuda(dout), cuda(w2), cuda(u))
    torch.cuda.synchronize()
    want = oracle.linear_bwd_data(f64(dout), f64(w2)) * oracle.gelu_grad(f64(u))
    assert max_rel(f64(du), want) < TOL_GRAD


# wgrad: dW[N, K] = dY[M, N]^T X[M, K], contraction over M tokens
# (6304, 768, 256), (2048, 1280, 200), (2000, 768, 256) ragged, (6304, 3072, 768)
# and (4112, 1280, 1280) split the token contraction (outputs of 3-36 tiles).
WGRAD_SHAPES = [(394, 576, 192), (130, 4096, 4096), (6304, 768, 256), (65, 8, 8), (2048, 1280, 200),
                (2048, 6144, 1536), (2000, 768, 256), (6304, 3072, 768), (4112, 1280, 1280)]


@pytest.mark.parametrize("M,N,K", WGRAD_SHAPES)
def test_linear_bwd_weight_exact(M, N, K):
    announce(f"bwd_weight exact M={M} N={N} K={K}")
    dY = random_int_bf16((M, N), 71, -3, 3)
    X = random_int_bf16((M, K), 72, -3, 3)
    rdW, rdb = oracle.linear_bwd_weight(f64(dY), f64(X))
    dW, wbuf = guarded((N, K), torch.float32)
    db, bbuf = guarded((N,), torch.float32)
    B.enc_linear_bwd_weight(cuda(dY), cuda(X), dW=dW, db=db)
    torch.cuda.synchronize()
    ok, err = exact_equal(dW, rdW)
    assert ok, err
    ok, err = exact_equal(db, rdb)
    assert ok, err
    assert guard_intact(wbuf, N * K) and guard_intact(bbuf, N)
    # accumulate adds onto the existing gradients
    B.enc_linear_bwd_weight(cuda(dY), cuda(X), dW=dW, db=db, accumulate=True)
    torch.cuda.synchronize()
    ok, err = exact_equal(dW, 2 * rdW)
    assert ok, err
    ok, err = exact_equal(db, 2 * rdb)
    assert ok, err


@pytest.mark.parametrize("M,N,K", [(6304, 768, 768), (2000, 768, 256), (4112, 1280, 1280)])
def test_linear_bwd_weight_split_matches_unsplit(M, N, K):
    # The split plan applies to these shapes; the unsplit kernel is the same
    # product summed in one pass.  Both within fp32 rounding of float64, and
    # the split path is run-to-run bitwise deterministic.
    assert B.linear_bwd_weight_workspace_bytes(M, N, K) > 0
    announce(f"bwd_weight split vs unsplit M={M} N={N} K={K}")
    dY, X = cuda(random_bf16((M, N), 111)), cuda(random_bf16((M, K), 112))
    w1, b1 = B.enc_linear_bwd_weight(dY, X)
    w2, b2 = B.enc_linear_bwd_weight(dY, X)
    w0, b0 = B.enc_linear_bwd_weight(dY, X, split=False)
    torch.cuda.synchronize()
    assert torch.equal(w1, w2) and torch.equal(b1, b2)
    rdW, rdb = oracle.linear_bwd_weight(f64(dY), f64(X))
    for got in (w1, w0):
        assert max_rel(f64(got), rdW) < 1e-5
    for got in (b1, b0):
        assert max_rel(f64(got), rdb) < 1e-5
    # a workspace one byte short is refused before anything runs
    need = B.linear_bwd_weight_workspace_bytes(M, N, K)
    short = torch.empty(need - 1, dtype=torch.uint8, device="cuda")
    with pytest.raises(B.EncError) as e:
        B.enc_linear_bwd_weight(dY, X, ws=short)
    assert e.value.status == B.ENC_ERR_WORKSPACE


def test_named_weight_gradients_match_generic():
    announce("named bwd_weight aliases")
    M, H, A, F = 394, 192, 192, 768
    dout, g = random_int_bf16((M, H), 81, -2, 2), random_int_bf16((M, F), 82, -2, 2)
    du, y2 = random_int_bf16((M, F), 83, -2, 2), random_int_bf16((M, H), 84, -2, 2)
    dh, o = random_int_bf16((M, H), 85, -2, 2), random_int_bf16((M, A), 86, -2, 2)
    dqkv, y1 = random_int_bf16((M, 3 * A), 87, -2, 2), random_int_bf16((M, H), 88, -2, 2)
    cases = [(B.enc_mlp_down_bwd_weight, dout, g), (B.enc_mlp_up_bwd_weight, du, y2),
             (B.enc_oproj_bwd_weight, dh, o), (B.enc_qkv_bwd_weight, dqkv, y1)]
    for fn, dY, X in cases:
        dW = torch.empty((dY.shape[1], X.shape[1]), device="cuda")
        db = torch.empty((dY.shape[1],), device="cuda")
        fn(cuda(dY), cuda(X), dW, db)
        torch.cuda.synchronize()
        rdW, rdb = oracle.linear_bwd_weight(f64(dY), f64(X))
        assert np.array_equal(f64(dW), rdW), fn.__name__
        assert np.array_equal(f64(db), rdb), fn.__name__


def test_linear_bwd_weight_without_db():
    announce("bwd_weight db=None")
    dY, X = random_int_bf16((100, 64), 91, -2, 2), random_int_bf16((100, 32), 92, -2, 2)
    dW, db = B.enc_linear_bwd_weight(cuda(dY), cuda(X), with_db=False)
    torch.cuda.synchronize()
    assert db is None
    assert np.array_equal(f64(dW), oracle.linear_bwd_weight(f64(dY), f64(X))[0])


# --------------------------------------------------------------------------- attention

# Grids of up to 256 workgroups take the small-grid launch shapes, larger
# ones (the last three cases: 384 forward / dQ workgroups each) the others.
ATTN_CASES = [(2, 197, 3, 64), (1, 257, 2, 80), (2, 256, 2, 128), (1, 1, 1, 64), (3, 7, 2, 80), (1, 65, 1, 128),
              (1, 129, 2, 64), (2, 300, 1, 80), (16, 197, 12, 64), (8, 257, 16, 80), (4, 256, 48, 128)]


def _attn_inputs(Bn, S, nh, d, seed, scale):
    return random_bf16((Bn * S, 3 * nh * d), seed, scale)


@pytest.mark.parametrize("Bn,S,nh,d", ATTN_CASES)
@pytest.mark.parametrize("scale", [1.0, 3.0])
def test_attn_fwd(Bn, S, nh, d, scale):
    announce(f"attn_fwd B={Bn} S={S} heads={nh} d={d} scale={scale}")
    qkv = _attn_inputs(Bn, S, nh, d, 101, scale)
    o, obuf = guarded((Bn * S, nh * d), torch.bfloat16)
    lse, lbuf = guarded((Bn, nh, S), torch.float32)
    B.enc_attn_fwd(Bn, S, nh, d, cuda(qkv), o=o, lse=lse)
    torch.cuda.synchronize()
    ro, rl = oracle.attention_fwd(f64(qkv), Bn, S, nh, d)
    assert max_rel(f64(o), ro) < TOL_ACT
    assert np.abs(f64(lse) - rl).max() < 2e-3 * max(1.0, np.abs(rl).max())
    assert guard_intact(obuf, o.numel()) and guard_intact(lbuf, lse.numel())


@pytest.mark.parametrize("Bn,S,nh,d", ATTN_CASES)
def test_attn_bwd(Bn, S, nh, d):
    announce(f"attn_bwd B={Bn} S={S} heads={nh} d={d}")
    qkv = _attn_inputs(Bn, S, nh, d, 111, 1.5)
    dO = random_bf16((Bn * S, nh * d), 112)
    o, lse = B.enc_attn_fwd(Bn, S, nh, d, cuda(qkv))
    dqkv, buf = guarded((Bn * S, 3 * nh * d), torch.bfloat16)
    B.enc_attn_bwd(Bn, S, nh, d, cuda(qkv), o, lse, cuda(dO), dqkv=dqkv)
    torch.cuda.synchronize()
    ref = oracle.attention_bwd(f64(qkv), f64(dO), Bn, S, nh, d)
    got = f64(dqkv)
    A = nh * d
    for part, sl in (("dq", slice(0, A)), ("dk", slice(A, 2 * A)), ("dv", slice(2 * A, 3 * A))):
        assert max_rel(got[:, sl], ref[:, sl]) < TOL_GRAD, part
    assert guard_intact(buf, dqkv.numel())


def _climbing_logits_qkv(Bn, S, nh, d, order, seed):
    """q and k whose logits climb across key tiles: along dimension 0 every
    query holds +8 (even queries) or -8 (odd queries) and key j holds a ramp
    r_j, so a query's running maximum grows by up to ~11 log2 units per
    32-key tile (ascending), only at the first tile (descending), or in
    uneven steps (zigzag).  Even and odd queries see opposite orders, so
    within one wave some queries grow while others do not.  The other
    dimensions hold small noise."""
    g = torch.Generator().manual_seed(seed)
    A = nh * d
    qkv = torch.randn(Bn * S, 3 * A, generator=g) * 0.3
    j = torch.arange(S, dtype=torch.float32)
    step = 0.35 / (8.0 * 1.4426950408889634 / d ** 0.5)  # log2 units per key, for |q0| = 8
    if order == "ascending":
        r = step * j
    elif order == "descending":
        r = step * (S - 1 - j)
    else:  # zigzag: tiles alternately climb and fall back, the maximum rising in uneven steps
        t = (j // 32).long()
        r = step * ((j % 32) * torch.where(t % 2 == 0, 1.0, 0.25) + 9.0 * t)
    sign = torch.where(torch.arange(S) % 2 == 0, 1.0, -1.0)
    for h in range(nh):
        qkv.view(Bn, S, 3 * A)[:, :, h * d] = 8.0 * sign
        qkv.view(Bn, S, 3 * A)[:, :, A + h * d] = r
    return qkv.to(torch.bfloat16)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("order", ["ascending", "descending", "zigzag"])
def test_attn_running_maximum_paths(order, d):
    """The forward rescales a query's accumulator only when its maximum grows
    by more than 2^8; random inputs rarely reach that after the first tile.
    Logits that climb across tiles drive the rescale path on every tile,
    never, or unevenly, with growing and non-growing queries in one wave."""
    Bn, S, nh = 2, 256, 2
    announce(f"attention running-maximum paths order={order} d={d}")
    qkv = _climbing_logits_qkv(Bn, S, nh, d, order, 141)
    dO = random_bf16((Bn * S, nh * d), 142)
    o, lse = B.enc_attn_fwd(Bn, S, nh, d, cuda(qkv))
    dqkv = B.enc_attn_bwd(Bn, S, nh, d, cuda(qkv), o, lse, cuda(dO))
    torch.cuda.synchronize()
    ro, rl = oracle.attention_fwd(f64(qkv), Bn, S, nh, d)
    assert max_rel(f64(o), ro) < TOL_ACT
    assert np.abs(f64(lse) - rl).max() < 2e-3 * max(1.0, np.abs(rl).max())
    ref = oracle.attention_bwd(f64(qkv), f64(dO), Bn, S, nh, d)
    assert max_rel(f64(dqkv), ref) < TOL_GRAD


def test_attn_bwd_is_deterministic():
    announce("attn_bwd determinism")
    Bn, S, nh, d = 2, 197, 3, 64
    qkv = cuda(_attn_inputs(Bn, S, nh, d, 121, 1.0))
    dO = cuda(random_bf16((Bn * S, nh * d), 122))
    o, lse = B.enc_attn_fwd(Bn, S, nh, d, qkv)
    a = B.enc_attn_bwd(Bn, S, nh, d, qkv, o, lse, dO)
    b = B.enc_attn_bwd(Bn, S, nh, d, qkv, o, lse, dO)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("S,d", [(100, 64), (197, 80), (70, 128), (256, 128)])
def test_attn_sequences_are_independent(S, d):
    """Tiles of the last keys of a sequence overhang into the next sequence;
    non-finite values there must not leak into this sequence's results."""
    announce(f"attn isolation S={S} d={d}")
    Bn, nh = 2, 2
    qkv = _attn_inputs(Bn, S, nh, d, 131, 1.0)
    dO = random_bf16((Bn * S, nh * d), 132)
    qkv[S:] = float("nan")
    dO[S:] = float("inf")
    o, lse = B.enc_attn_fwd(Bn, S, nh, d, cuda(qkv))
    dqkv = B.enc_attn_bwd(Bn, S, nh, d, cuda(qkv), o, lse, cuda(dO))
    torch.cuda.synchronize()
    ro, rl = oracle.attention_fwd(f64(qkv[:S]), 1, S, nh, d)
    assert max_rel(f64(o[:S]), ro) < TOL_ACT
    assert np.abs(f64(lse[:1]) - rl).max() < 2e-3 * max(1.0, np.abs(rl).max())
    ref = oracle.attention_bwd(f64(qkv[:S]), f64(dO[:S]), 1, S, nh, d)
    assert np.isfinite(f64(dqkv[:S])).all()
    assert max_rel(f64(dqkv[:S]), ref) < TOL_GRAD


# --------------------------------------------------------------------------- measurement helpers

def test_calibration_kernels():
    announce("calibration kernels")
    src = torch.randint(0, 256, (1 << 20,), dtype=torch.uint8, device="cuda")
    dst, buf = guarded((1 << 19,), torch.bfloat16)  # same byte size, guarded tail
    B.enc_calib_copy(src, dst.view(torch.uint8))
    out = B.enc_calib_mfma(8, 3)
    torch.cuda.synchronize()
    assert torch.equal(dst.view(torch.uint8), src)
    assert guard_intact(buf, dst.numel())
    assert torch.isfinite(out).all() and (out > 0).all()


# --------------------------------------------------------------------------- maximum sizes

def test_mlp_down_fwd_at_the_largest_accepted_operand():
    """g holds 2^31 - 8192 elements (4 GiB - 16 KiB), past the 32-bit byte
    offsets of the direct-to-LDS path: the register-staged kernel (64-bit
    row offsets) takes it.  Sampled rows against the oracle."""
    M, F, H = 87381, 24576, 64
    announce(f"mlp_down_fwd largest operand M={M} F={F} H={H}")
    gen = torch.Generator(device="cuda").manual_seed(7)
    g = torch.randn((M, F), generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    w2 = cuda(random_bf16((H, F), 8, 0.02))
    b2 = cuda(random_bf16((H,), 9, 0.02))
    resid = cuda(random_bf16((M, H), 10))
    out = B.enc_mlp_down_fwd(g, w2, b2, resid)
    torch.cuda.synchronize()
    rows = torch.tensor([0, 1, 40000, 87379, M - 1], device="cuda")
    ref = oracle.linear_fwd(f64(g[rows]), f64(w2), f64(b2), resid=f64(resid[rows]))
    assert max_rel(f64(out[rows]), ref) < TOL_ACT
    del g
