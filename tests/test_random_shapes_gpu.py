"""Seeded random shapes through the GEMM layouts, attention and LayerNorm
(through the C ABI), against the oracle.

Besides the hand-picked shapes of the per-kernel tests, these draw output
and contraction sizes at random (feature widths multiples of 8, any token
count): general ones, small outputs with long contractions so that the
library's split plans run, and grids large enough for 256-row tiles.  Inputs are small integers (sparse signs for the
bf16-output products) so that fp32 accumulation and bf16 rounding are
exact: every product must equal the oracle bit for bit, with and without a
workspace, and leave the guard band after each output untouched.  Attention
and LayerNorm draw sequence lengths, head counts, head dims, row counts and
widths at random and meet the parity bar of the per-kernel tests.
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


def _shapes():
    rng = np.random.default_rng(20240805)
    mk = []  # output [M, N], contraction K
    for _ in range(10):
        mk.append((int(rng.integers(1, 1600)), 8 * int(rng.integers(1, 257)), 8 * int(rng.integers(1, 385))))
    for _ in range(6):  # a few output tiles, a long contraction: split plans
        mk.append((int(rng.integers(200, 2049)), 8 * int(rng.integers(1, 65)), 64 * int(rng.integers(16, 64))))
    for _ in range(4):  # grids that fill the GPU: 256-row tiles
        mk.append((int(rng.integers(1800, 2049)), 8 * int(rng.integers(700, 801)), 64 * int(rng.integers(8, 17))))
    wg = []  # dW[N, K] over M tokens
    for _ in range(8):
        wg.append((int(rng.integers(1, 1600)), 8 * int(rng.integers(1, 257)), 8 * int(rng.integers(1, 257))))
    for _ in range(6):
        wg.append((int(rng.integers(1024, 3001)), 8 * int(rng.integers(1, 97)), 8 * int(rng.integers(1, 97))))
    for _ in range(3):
        wg.append((int(rng.integers(500, 2049)), 8 * int(rng.integers(300, 513)), 8 * int(rng.integers(300, 513))))
    at = []  # attention (batch, seq, heads, head_dim)
    for hi in (701, 701, 701, 701, 701, 100, 100, 100):
        at.append((int(rng.integers(1, 5)), int(rng.integers(1, hi)), int(rng.integers(1, 7)),
                   int(rng.choice([64, 80, 128]))))
    for _ in range(2):  # grids above 256 workgroups
        at.append((8, int(rng.integers(100, 401)), 16, int(rng.choice([64, 80, 128]))))
    ln = [(int(rng.integers(1, hi)), 8 * int(rng.integers(1, 1025))) for hi in (5001,) * 7 + (40,) * 3]
    return mk, wg, at, ln


MK, WG, AT, LN = _shapes()


def _density(K):
    return min(0.5, float(np.sqrt(24.0 / K)))


@pytest.mark.parametrize("M,N,K", MK)
def test_random_forward_and_input_gradient(M, N, K):
    for layout, name in ((B.LAYOUT_FWD, "fwd"), (B.LAYOUT_DGRAD, "dgrad")):
        announce(f"random {name} M={M} N={N} K={K} plan={B.linear_plan(layout, M, N, K)}")
    d = _density(K)
    X, W = random_sparse_sign_bf16((M, K), 301, d), random_sparse_sign_bf16((N, K), 302, d)
    b, R = random_int_bf16((N,), 303, -3, 3), random_int_bf16((M, N), 304, -8, 8)
    want = oracle.linear_fwd(f64(X), f64(W), f64(b), resid=f64(R))
    dY, Wd = random_sparse_sign_bf16((M, K), 305, d), random_sparse_sign_bf16((K, N), 306, d)
    want_d = oracle.linear_bwd_data(f64(dY), f64(Wd))
    for split in (True, False):
        Y, buf = guarded((M, N), torch.bfloat16)
        B.enc_oproj_fwd(cuda(X), cuda(W), cuda(b), cuda(R), h=Y, split=split)
        # MLP up input gradient: dy2[M, H] = du[M, F] w_1[F, H] with F = K, H = N
        Yd, bufd = guarded((M, N), torch.bfloat16)
        B.enc_mlp_up_bwd_data(cuda(dY), cuda(Wd), dy2=Yd, split=split)
        torch.cuda.synchronize()
        ok, err = exact_equal(Y, want)
        assert ok, ("fwd", split, err)
        ok, err = exact_equal(Yd, want_d)
        assert ok, ("dgrad", split, err)
        assert guard_intact(buf, M * N) and guard_intact(bufd, M * N)


@pytest.mark.parametrize("M,N,K", WG)
def test_random_weight_gradient(M, N, K):
    announce(f"random wgrad M={M} N={N} K={K} plan={B.linear_plan(B.LAYOUT_WGRAD, M, N, K)}")
    dY, X = random_int_bf16((M, N), 311, -3, 3), random_int_bf16((M, K), 312, -3, 3)
    rdW, rdb = oracle.linear_bwd_weight(f64(dY), f64(X))
    for split in (True, False):
        dW, wbuf = guarded((N, K), torch.float32)
        db, bbuf = guarded((N,), torch.float32)
        B.enc_linear_bwd_weight(cuda(dY), cuda(X), dW=dW, db=db, split=split)
        torch.cuda.synchronize()
        ok, err = exact_equal(dW, rdW)
        assert ok, ("dW", split, err)
        ok, err = exact_equal(db, rdb)
        assert ok, ("db", split, err)
        assert guard_intact(wbuf, N * K) and guard_intact(bbuf, N)


@pytest.mark.parametrize("Bn,S,nh,d", AT)
def test_random_attention(Bn, S, nh, d):
    announce(f"random attention B={Bn} S={S} heads={nh} d={d}")
    qkv = random_bf16((Bn * S, 3 * nh * d), 321, 1.5)
    dO = random_bf16((Bn * S, nh * d), 322)
    o, obuf = guarded((Bn * S, nh * d), torch.bfloat16)
    lse, lbuf = guarded((Bn, nh, S), torch.float32)
    B.enc_attn_fwd(Bn, S, nh, d, cuda(qkv), o=o, lse=lse)
    dqkv, dbuf = guarded((Bn * S, 3 * nh * d), torch.bfloat16)
    B.enc_attn_bwd(Bn, S, nh, d, cuda(qkv), o, lse, cuda(dO), dqkv=dqkv)
    torch.cuda.synchronize()
    ro, rl = oracle.attention_fwd(f64(qkv), Bn, S, nh, d)
    assert max_rel(f64(o), ro) < TOL_ACT
    assert np.abs(f64(lse) - rl).max() < 2e-3 * max(1.0, np.abs(rl).max())
    ref = oracle.attention_bwd(f64(qkv), f64(dO), Bn, S, nh, d)
    got, A = f64(dqkv), nh * d
    for part, sl in (("dq", slice(0, A)), ("dk", slice(A, 2 * A)), ("dv", slice(2 * A, 3 * A))):
        assert max_rel(got[:, sl], ref[:, sl]) < TOL_GRAD, part
    assert guard_intact(obuf, o.numel()) and guard_intact(lbuf, lse.numel()) and guard_intact(dbuf, dqkv.numel())


@pytest.mark.parametrize("rows,cols", LN)
def test_random_layernorm(rows, cols):
    announce(f"random layernorm rows={rows} cols={cols}")
    x = (random_bf16((rows, cols), 331, 1.5).float() + 0.4).to(torch.bfloat16)
    g = (1 + random_bf16((cols,), 332, 0.2).float()).to(torch.bfloat16)
    b = random_bf16((cols,), 333, 0.2)
    dy, dres = random_bf16((rows, cols), 334), random_bf16((rows, cols), 335)
    y, ybuf = guarded((rows, cols), torch.bfloat16)
    mean, mbuf = guarded((rows,), torch.float32)
    rstd, rbuf = guarded((rows,), torch.float32)
    B.enc_ln_fwd(cuda(x), cuda(g), cuda(b), 1e-6, y=y, mean=mean, rstd=rstd)
    dx, dxbuf = guarded((rows, cols), torch.bfloat16)
    dg, dgbuf = guarded((cols,), torch.float32)
    db, dbbuf = guarded((cols,), torch.float32)
    B.enc_ln_bwd(cuda(dy), cuda(x), mean, rstd, cuda(g), dresid=cuda(dres), dx=dx, dgamma=dg, dbeta=db)
    torch.cuda.synchronize()
    ry, rm, rr = oracle.layernorm_fwd(f64(x), f64(g), f64(b), 1e-6)
    assert max_rel(f64(y), ry) < TOL_ACT
    assert np.abs(f64(mean) - rm).max() < 1e-5 * max(1.0, np.abs(rm).max())
    assert np.abs(f64(rstd) / rr - 1).max() < 1e-5
    rdx, rdg, rdb = oracle.layernorm_bwd(f64(dy), f64(x), rm, rr, f64(g))
    assert max_rel(f64(dx), rdx + f64(dres)) < TOL_GRAD
    assert max_rel(f64(dg), rdg) < TOL_GRAD and max_rel(f64(db), rdb) < TOL_GRAD
    for buf, n in ((ybuf, rows * cols), (mbuf, rows), (rbuf, rows), (dxbuf, rows * cols), (dgbuf, cols),
                   (dbbuf, cols)):
        assert guard_intact(buf, n)
