"""Pins of the float64 oracle against facts that do not come from the oracle.

Each check compares the oracle with something independent of it: the ViT
table of the paper (Appendix A), library routines the layer reduces to
(torch LayerNorm / linear / GELU / scaled-dot-product attention in float64),
closed forms and invariants, pure-Python brute force on tiny inputs, and
central finite differences of the oracle's own forward.  The mutation tests
at the end plant plausible mistakes in the oracle (on the CPU) and check that
at least one pin catches each.
"""

import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import encoder_layer as OL

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


def _tiny_cfg(**kw):
    cfg = dict(batch=2, seq=3, hidden=8, heads=2, head_dim=4, mlp=16, ln_eps=1e-6)
    cfg.update(kw)
    return cfg


def _params(cfg, rng, scale=0.5):
    shapes = oracle.param_shapes(cfg["hidden"], cfg["heads"], cfg["head_dim"], cfg["mlp"])
    p = {}
    for n in oracle.PARAM_NAMES:
        p[n] = rng.normal(size=shapes[n]) * scale
        if n in ("ln1_g", "ln2_g"):
            p[n] = 1.0 + p[n]
    return p


# ----------------------------------------------------------------- golden

def param_count_error(shapes_fn=None):
    """Largest relative gap between the layer's parameter count times depth
    and the counts printed in the paper's ViT table."""
    shapes_fn = shapes_fn or oracle.param_shapes
    data = json.load(open(os.path.join(GOLDEN, "vit_configs.json")))
    worst = 0.0
    for m in data["models"]:
        shapes = shapes_fn(m["width"], m["heads"], m["head_dim"], m["mlp"])
        per_layer = sum(int(np.prod(s)) for s in shapes.values())
        total_b = per_layer * m["depth"] / 1e9
        worst = max(worst, abs(total_b - m["params_printed_B"]) / m["params_printed_B"])
    return worst


def test_vit_table_heads_times_head_dim_is_width():
    data = json.load(open(os.path.join(GOLDEN, "vit_configs.json")))
    for m in data["models"]:
        assert m["heads"] * m["head_dim"] == m["width"], m["name"]


def test_vit_table_parameter_counts():
    # 48 * (4 H^2 + 2 H F) + biases/LN: 3.06B, 5.44B, 9.66B, 21.74B against
    # the printed 3B, 5.5B, 10B, 22B.
    assert param_count_error() < 0.04


# ----------------------------------------------------------------- LayerNorm

def layernorm_fwd_error(seed=0):
    rng = _rng(seed)
    x = rng.normal(size=(9, 96)) * 3.0 + 1.5
    g = 1.0 + 0.3 * rng.normal(size=96)
    b = 0.3 * rng.normal(size=96)
    eps = 1e-5
    y, mean, rstd = oracle.layernorm_fwd(x, g, b, eps)
    ref = F.layer_norm(torch.from_numpy(x), (96,), torch.from_numpy(g), torch.from_numpy(b), eps).numpy()
    return np.abs(y - ref).max()


def test_layernorm_matches_torch():
    assert layernorm_fwd_error() < 1e-12


def test_layernorm_invariants():
    rng = _rng(1)
    x = rng.normal(size=(7, 64)) * 2.0 - 0.7
    eps = 1e-6
    y, mean, rstd = oracle.layernorm_fwd(x, np.ones(64), np.zeros(64), eps)
    assert np.abs(y.mean(axis=1)).max() < 1e-12
    var = x.var(axis=1)  # numpy's biased variance
    np.testing.assert_allclose(y.var(axis=1), var / (var + eps), rtol=1e-12)
    np.testing.assert_allclose(mean, x.mean(axis=1), rtol=1e-12)
    np.testing.assert_allclose(rstd, 1.0 / np.sqrt(var + eps), rtol=1e-12)


def test_layernorm_constant_row_gives_beta():
    beta = np.arange(16, dtype=np.float64)
    y, _, _ = oracle.layernorm_fwd(np.full((3, 16), 2.5), np.full(16, 7.0), beta, 1e-6)
    np.testing.assert_allclose(y, np.broadcast_to(beta, (3, 16)), atol=1e-12)


def layernorm_bwd_error(seed=2):
    rng = _rng(seed)
    R, C = 5, 24
    x = rng.normal(size=(R, C)) * 2 + 0.5
    g = 1.0 + 0.3 * rng.normal(size=C)
    b = 0.3 * rng.normal(size=C)
    dy = rng.normal(size=(R, C))
    _, mean, rstd = oracle.layernorm_fwd(x, g, b, 1e-5)
    dx, dg, db = oracle.layernorm_bwd(dy, x, mean, rstd, g)
    tx, tg, tb = (torch.from_numpy(a).requires_grad_() for a in (x, g, b))
    F.layer_norm(tx, (C,), tg, tb, 1e-5).backward(torch.from_numpy(dy))
    return max(np.abs(dx - tx.grad.numpy()).max(), np.abs(dg - tg.grad.numpy()).max(),
               np.abs(db - tb.grad.numpy()).max())


def test_layernorm_bwd_matches_torch_autograd():
    assert layernorm_bwd_error() < 1e-12


# ----------------------------------------------------------------- Linear

def _brute_linear(X, W, b):
    M, K = len(X), len(X[0])
    N = len(W)
    return [[sum(X[m][k] * W[n][k] for k in range(K)) + b[n] for n in range(N)] for m in range(M)]


def test_linear_fwd_brute_force():
    rng = _rng(3)
    X = rng.integers(-4, 5, size=(3, 5)).astype(np.float64)
    W = rng.integers(-4, 5, size=(4, 5)).astype(np.float64)
    b = rng.integers(-4, 5, size=4).astype(np.float64)
    R = rng.integers(-4, 5, size=(3, 4)).astype(np.float64)
    Y = oracle.linear_fwd(X, W, b, resid=R)
    ref = np.array(_brute_linear(X.tolist(), W.tolist(), b.tolist())) + R
    assert np.array_equal(Y, ref)


def test_linear_bwd_brute_force():
    rng = _rng(4)
    M, N, K = 3, 4, 5
    dY = rng.integers(-4, 5, size=(M, N)).astype(np.float64)
    W = rng.integers(-4, 5, size=(N, K)).astype(np.float64)
    X = rng.integers(-4, 5, size=(M, K)).astype(np.float64)
    dX = oracle.linear_bwd_data(dY, W)
    dW, db = oracle.linear_bwd_weight(dY, X)
    for m in range(M):
        for k in range(K):
            assert dX[m, k] == sum(dY[m, n] * W[n, k] for n in range(N))
    for n in range(N):
        assert db[n] == sum(dY[m, n] for m in range(M))
        for k in range(K):
            assert dW[n, k] == sum(dY[m, n] * X[m, k] for m in range(M))


# ----------------------------------------------------------------- GELU

def gelu_error():
    u = np.linspace(-8, 8, 1601)
    ref = F.gelu(torch.from_numpy(u), approximate="none").numpy()
    return np.abs(oracle.gelu(u) - ref).max()


def gelu_grad_error():
    u = np.linspace(-6, 6, 241)
    h = 1e-5
    fd = (oracle.gelu(u + h) - oracle.gelu(u - h)) / (2 * h)
    return np.abs(oracle.gelu_grad(u) - fd).max()


def test_gelu_matches_torch_exact_gelu():
    assert gelu_error() < 1e-14


def test_gelu_closed_forms():
    assert oracle.gelu(np.array([0.0]))[0] == 0.0
    u = np.linspace(-5, 5, 101)
    np.testing.assert_allclose(oracle.gelu(u) - oracle.gelu(-u), u, atol=1e-14)
    assert abs(oracle.gelu_grad(np.array([0.0]))[0] - 0.5) < 1e-15
    # GELU(1) = Phi(1) = (1 + erf(1/sqrt2))/2
    assert abs(oracle.gelu(np.array([1.0]))[0] - 0.8413447460685429) < 1e-15


def test_gelu_grad_finite_difference():
    assert gelu_grad_error() < 1e-9


# ----------------------------------------------------------------- Attention

def _qkv(B, S, nh, d, rng, scale=1.0):
    return rng.normal(size=(B * S, 3 * nh * d)) * scale


def _torch_sdpa(qkv, B, S, nh, d):
    t = torch.from_numpy(qkv).view(B, S, 3, nh, d)
    q, k, v = (t[:, :, i].transpose(1, 2) for i in range(3))
    return F.scaled_dot_product_attention(q, k, v).transpose(1, 2).reshape(B * S, nh * d).numpy()


def attention_fwd_error(seed=5, B=2, S=7, nh=3, d=8):
    rng = _rng(seed)
    qkv = _qkv(B, S, nh, d, rng, 1.5)
    o, _ = oracle.attention_fwd(qkv, B, S, nh, d)
    return np.abs(o - _torch_sdpa(qkv, B, S, nh, d)).max()


def test_attention_matches_torch_sdpa():
    assert attention_fwd_error() < 1e-12
    assert attention_fwd_error(seed=6, B=1, S=20, nh=2, d=80) < 1e-12


def test_attention_softmax_rows_sum_to_one():
    rng = _rng(7)
    B, S, nh, d = 2, 9, 2, 16
    qkv = _qkv(B, S, nh, d, rng, 2.0)
    _, lse = oracle.attention_fwd(qkv, B, S, nh, d)
    t = qkv.reshape(B, S, 3, nh, d)
    for b in range(B):
        for h in range(nh):
            q, k = t[b, :, 0, h], t[b, :, 1, h]
            s = np.array([[float(np.dot(q[i], k[j])) for j in range(S)] for i in range(S)]) / math.sqrt(d)
            rows = np.exp(s - lse[b, h][:, None]).sum(axis=1)
            assert np.abs(rows - 1.0).max() < 1e-12


def test_attention_closed_forms():
    rng = _rng(8)
    B, S, nh, d = 2, 6, 2, 4
    qkv = _qkv(B, S, nh, d, rng)
    A = nh * d
    # Q = 0: uniform attention, O_i = mean over keys of V
    z = qkv.copy()
    z[:, :A] = 0.0
    o, lse = oracle.attention_fwd(z, B, S, nh, d)
    v = z[:, 2 * A:].reshape(B, S, A)
    np.testing.assert_allclose(o.reshape(B, S, A), np.broadcast_to(v.mean(axis=1, keepdims=True), (B, S, A)), atol=1e-14)
    np.testing.assert_allclose(lse, math.log(S), atol=1e-14)
    # S = 1: O = V
    one = _qkv(3, 1, nh, d, rng)
    o1, _ = oracle.attention_fwd(one, 3, 1, nh, d)
    np.testing.assert_allclose(o1, one[:, 2 * A:], atol=1e-15)
    # one dominant key: every query attends only to key 2
    dom = qkv.copy().reshape(B, S, 3, nh, d)
    dom[:, :, 0] = 1.0
    dom[:, :, 1] = 0.0
    dom[:, 2, 1] = 50.0
    o2, _ = oracle.attention_fwd(dom.reshape(B * S, 3 * A), B, S, nh, d)
    want = np.broadcast_to(dom[:, 2:3, 2].reshape(B, 1, A), (B, S, A))
    np.testing.assert_allclose(o2.reshape(B, S, A), want, atol=1e-12)


def test_attention_is_permutation_equivariant():
    rng = _rng(9)
    B, S, nh, d = 1, 8, 2, 4
    qkv = _qkv(B, S, nh, d, rng)
    perm = rng.permutation(S)
    o, _ = oracle.attention_fwd(qkv, B, S, nh, d)
    op, _ = oracle.attention_fwd(qkv[perm], B, S, nh, d)
    np.testing.assert_allclose(op, o[perm], atol=1e-13)


def attention_bwd_error(seed=10, B=2, S=5, nh=2, d=8):
    rng = _rng(seed)
    qkv = _qkv(B, S, nh, d, rng, 1.3)
    dO = rng.normal(size=(B * S, nh * d))
    got = oracle.attention_bwd(qkv, dO, B, S, nh, d)
    tq = torch.from_numpy(qkv).requires_grad_()
    t = tq.view(B, S, 3, nh, d)
    q, k, v = (t[:, :, i].transpose(1, 2) for i in range(3))
    o = F.scaled_dot_product_attention(q, k, v).transpose(1, 2).reshape(B * S, nh * d)
    o.backward(torch.from_numpy(dO))
    return np.abs(got - tq.grad.numpy()).max()


def test_attention_bwd_matches_torch_autograd():
    assert attention_bwd_error() < 1e-12


# ----------------------------------------------------------------- whole layer

def _loss(cfg, p, x, dout):
    out, _ = oracle.layer_fwd(cfg, p, x)
    return float((out * dout).sum())


def layer_fd_error(cfg, seed=11, h=1e-5):
    """Largest gap between the oracle's analytic gradients and central finite
    differences of L = <dout, out> over every element of x and every
    parameter, scaled by max(1, |gradient|)."""
    rng = _rng(seed)
    M = cfg["batch"] * cfg["seq"]
    x = rng.normal(size=(M, cfg["hidden"]))
    p = _params(cfg, rng)
    dout = rng.normal(size=(M, cfg["hidden"]))
    out, saved = oracle.layer_fwd(cfg, p, x)
    dx, grads, _ = oracle.layer_bwd(cfg, p, x, saved, dout)
    worst = 0.0
    targets = [("x", x, dx)] + [(n, p[n], grads[n]) for n in oracle.PARAM_NAMES]
    for name, arr, an in targets:
        flat = arr.reshape(-1)
        fd = np.empty(flat.size)
        for i in range(flat.size):
            keep = flat[i]
            flat[i] = keep + h
            lp = _loss(cfg, p, x, dout)
            flat[i] = keep - h
            lm = _loss(cfg, p, x, dout)
            flat[i] = keep
            fd[i] = (lp - lm) / (2 * h)
        scale = max(1.0, np.abs(an).max())
        worst = max(worst, np.abs(fd - an.reshape(-1)).max() / scale)
    return worst


def test_layer_gradients_finite_difference():
    assert layer_fd_error(_tiny_cfg()) < 1e-6


def test_layer_gradients_finite_difference_sharded_width():
    # heads*head_dim != hidden, as in one tensor-parallel shard
    assert layer_fd_error(_tiny_cfg(heads=1, head_dim=4, mlp=12, seq=4)) < 1e-6


def _torch_layer(cfg, p, x):
    B, S, H = cfg["batch"], cfg["seq"], cfg["hidden"]
    nh, d, eps = cfg["heads"], cfg["head_dim"], cfg["ln_eps"]
    y1 = F.layer_norm(x, (H,), p["ln1_g"], p["ln1_b"], eps)
    qkv = F.linear(y1, p["w_qkv"], p["b_qkv"]).view(B, S, 3, nh, d)
    q, k, v = (qkv[:, :, i].transpose(1, 2) for i in range(3))
    o = F.scaled_dot_product_attention(q, k, v).transpose(1, 2).reshape(B * S, nh * d)
    h = x + F.linear(o, p["w_o"], p["b_o"])
    y2 = F.layer_norm(h, (H,), p["ln2_g"], p["ln2_b"], eps)
    g = F.gelu(F.linear(y2, p["w_1"], p["b_1"]), approximate="none")
    return h + F.linear(g, p["w_2"], p["b_2"])


def layer_vs_torch_error(cfg, seed=12):
    rng = _rng(seed)
    M = cfg["batch"] * cfg["seq"]
    x = rng.normal(size=(M, cfg["hidden"]))
    p = _params(cfg, rng, scale=0.05)
    dout = rng.normal(size=(M, cfg["hidden"]))
    out, saved = oracle.layer_fwd(cfg, p, x)
    dx, grads, _ = oracle.layer_bwd(cfg, p, x, saved, dout)
    tx = torch.from_numpy(x).requires_grad_()
    tp = {n: torch.from_numpy(v).requires_grad_() for n, v in p.items()}
    tout = _torch_layer(cfg, tp, tx)
    tout.backward(torch.from_numpy(dout))
    errs = [np.abs(out - tout.detach().numpy()).max() / np.abs(out).max(),
            np.abs(dx - tx.grad.numpy()).max() / np.abs(dx).max()]
    for n in oracle.PARAM_NAMES:
        ref = tp[n].grad.numpy()
        errs.append(np.abs(grads[n] - ref).max() / max(np.abs(ref).max(), 1e-300))
    return max(errs)


def test_layer_matches_torch_composition_vit_tiny():
    cfg = dict(batch=2, seq=197, hidden=192, heads=3, head_dim=64, mlp=768, ln_eps=1e-6)
    assert layer_vs_torch_error(cfg) < 1e-10


def test_layer_matches_torch_composition_sharded_d80():
    cfg = dict(batch=2, seq=17, hidden=64, heads=2, head_dim=80, mlp=96, ln_eps=1e-6)
    assert layer_vs_torch_error(cfg) < 1e-10


def residual_wiring_error(cfg=None, seed=13):
    """All weights, biases and LayerNorm affines zero: the layer is the
    identity, dx = dout, db2 = dbo = column sums of dout, all else zero."""
    cfg = cfg or _tiny_cfg(seq=5)
    rng = _rng(seed)
    M, H = cfg["batch"] * cfg["seq"], cfg["hidden"]
    shapes = oracle.param_shapes(H, cfg["heads"], cfg["head_dim"], cfg["mlp"])
    p = {n: np.zeros(s) for n, s in shapes.items()}
    x = rng.normal(size=(M, H))
    dout = rng.normal(size=(M, H))
    out, saved = oracle.layer_fwd(cfg, p, x)
    dx, grads, _ = oracle.layer_bwd(cfg, p, x, saved, dout)
    errs = [np.abs(out - x).max(), np.abs(dx - dout).max(),
            np.abs(grads["b_2"] - dout.sum(0)).max(), np.abs(grads["b_o"] - dout.sum(0)).max()]
    for n in oracle.PARAM_NAMES:
        if n not in ("b_2", "b_o"):
            errs.append(np.abs(grads[n]).max())
    return max(errs)


def test_layer_residual_wiring():
    assert residual_wiring_error() < 1e-13


def test_layer_sequences_independent_and_permutation_equivariant():
    cfg = _tiny_cfg(batch=2, seq=6)
    rng = _rng(14)
    M, H = 12, cfg["hidden"]
    x = rng.normal(size=(M, H))
    p = _params(cfg, rng)
    out, _ = oracle.layer_fwd(cfg, p, x)
    # swap the two sequences and permute tokens inside the first one
    perm = np.concatenate([6 + rng.permutation(6), rng.permutation(6)])
    outp, _ = oracle.layer_fwd(cfg, p, x[perm])
    np.testing.assert_allclose(outp, out[perm], atol=1e-12)


def test_layer_flops_formula():
    # ViT-22B layer, micro-batch 8 of 256 tokens: 4 projections + attention
    cfg = dict(batch=8, seq=256, hidden=6144, heads=48, head_dim=128, mlp=24576)
    assert oracle.layer_flops(cfg) == 2 * 2048 * (3 * 6144 * 6144 + 6144 * 6144 + 2 * 6144 * 24576) \
        + 4 * 8 * 48 * 256 * 256 * 128


# ----------------------------------------------------------------- mutants
# Plant plausible mistakes in the oracle and check that a pin catches each.

def test_mutant_ln_bwd_dropped_term_is_caught(monkeypatch):
    def bad(dy, x, mean, rstd, gamma):
        xhat = (x - mean[:, None]) * rstd[:, None]
        ghat = dy * gamma
        dx = rstd[:, None] * (ghat - ghat.mean(axis=1, keepdims=True))
        return dx, (dy * xhat).sum(axis=0), dy.sum(axis=0)
    monkeypatch.setattr(OL, "layernorm_bwd", bad)
    monkeypatch.setattr(oracle, "layernorm_bwd", bad)
    assert layernorm_bwd_error() > 1e-3
    assert layer_fd_error(_tiny_cfg()) > 1e-3


def test_mutant_ln_unbiased_variance_is_caught(monkeypatch):
    def bad(x, gamma, beta, eps):
        mean = x.mean(axis=-1)
        c = x - mean[..., None]
        rstd = 1.0 / np.sqrt((c * c).sum(axis=-1) / (x.shape[-1] - 1) + eps)
        return c * rstd[..., None] * gamma + beta, mean, rstd
    monkeypatch.setattr(oracle, "layernorm_fwd", bad)
    assert layernorm_fwd_error() > 1e-3


def test_mutant_attention_bwd_missing_rowsum_is_caught(monkeypatch):
    def bad(qkv, dO, B, S, heads, d):
        q, k, v = OL._split_heads(qkv, B, S, heads, d)
        do = dO.reshape(B, S, heads, d).transpose(0, 2, 1, 3)
        sc = 1.0 / math.sqrt(d)
        P = OL._softmax_rows((q @ k.transpose(0, 1, 3, 2)) * sc)
        dv = P.transpose(0, 1, 3, 2) @ do
        dS = P * (do @ v.transpose(0, 1, 3, 2))
        out = np.stack([OL._merge_heads(t, B, S, heads, d)
                        for t in ((dS @ k) * sc, (dS.transpose(0, 1, 3, 2) @ q) * sc, dv)], axis=1)
        return out.reshape(B * S, 3 * heads * d)
    monkeypatch.setattr(OL, "attention_bwd", bad)
    monkeypatch.setattr(oracle, "attention_bwd", bad)
    assert attention_bwd_error() > 1e-3
    assert layer_fd_error(_tiny_cfg()) > 1e-3


def test_mutant_attention_wrong_scale_is_caught(monkeypatch):
    def bad(qkv, B, S, heads, d):
        q, k, v = OL._split_heads(qkv, B, S, heads, d)
        s = (q @ k.transpose(0, 1, 3, 2)) / d
        m = s.max(axis=-1)
        lse = m + np.log(np.exp(s - m[..., None]).sum(axis=-1))
        return OL._merge_heads(OL._softmax_rows(s) @ v, B, S, heads, d), lse
    monkeypatch.setattr(OL, "attention_fwd", bad)
    monkeypatch.setattr(oracle, "attention_fwd", bad)
    assert attention_fwd_error() > 1e-3
    assert layer_fd_error(_tiny_cfg()) > 1e-3


def test_mutant_gelu_grad_dropped_term_is_caught(monkeypatch):
    def bad(u):
        return 0.5 * (1.0 + OL._erf(u / math.sqrt(2.0)))
    monkeypatch.setattr(OL, "gelu_grad", bad)
    monkeypatch.setattr(oracle, "gelu_grad", bad)
    assert gelu_grad_error() > 1e-3
    assert layer_fd_error(_tiny_cfg()) > 1e-3


def test_mutant_tanh_gelu_is_caught(monkeypatch):
    def bad(u):
        return 0.5 * u * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (u + 0.044715 * u ** 3)))
    monkeypatch.setattr(oracle, "gelu", bad)
    assert gelu_error() > 1e-5


def test_mutant_dropped_residual_is_caught(monkeypatch):
    real = OL.layer_fwd

    def bad(cfg, p, x):
        out, saved = real(cfg, p, x)
        return out - saved["h"] + (saved["h"] - x), saved
    monkeypatch.setattr(OL, "layer_fwd", bad)
    monkeypatch.setattr(oracle, "layer_fwd", bad)
    assert residual_wiring_error() > 1e-3


def test_mutant_swapped_wgrad_operands_is_caught(monkeypatch):
    def bad(dY, X):
        return (X.T @ dY).T[:, ::-1], dY.sum(axis=0)
    monkeypatch.setattr(OL, "linear_bwd_weight", bad)
    monkeypatch.setattr(oracle, "linear_bwd_weight", bad)
    assert layer_fd_error(_tiny_cfg()) > 1e-3


def test_mutant_block_structure_is_caught():
    # A gated (three-matrix) MLP or a missing output projection would not
    # reproduce the paper's parameter counts.
    def gated(H, nh, d, F_):
        s = oracle.param_shapes(H, nh, d, F_)
        s["w_gate"] = (F_, H)
        return s

    def no_out_proj(H, nh, d, F_):
        s = oracle.param_shapes(H, nh, d, F_)
        del s["w_o"]
        return s
    assert param_count_error(gated) > 0.04
    assert param_count_error(no_out_proj) > 0.04
