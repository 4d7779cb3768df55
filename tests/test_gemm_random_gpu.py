"""Seeded random shapes through the three GEMM layouts (through the C ABI),
bit-exact against the oracle.

Besides the hand-picked shapes of the per-kernel tests, these draw output
and contraction sizes at random (feature widths multiples of 8, any token
count): general ones, small outputs with long contractions so that the
library's split plans run, and grids large enough for 256-row tiles.  Inputs are small integers (sparse signs for the
bf16-output products) so that fp32 accumulation and bf16 rounding are
exact: every product must equal the oracle bit for bit, with and without a
workspace, and leave the guard band after each output untouched.
"""

import numpy as np
import pytest
import torch

import oracle
from helpers import announce, cuda, exact_equal, f64, guard_intact, guarded
from paper_2408_03505_amd import binding as B
from paper_2408_03505_amd.synthetic import random_int_bf16, random_sparse_sign_bf16

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
    return mk, wg


MK, WG = _shapes()


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
