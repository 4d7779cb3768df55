"""Pins of the ViT-22B-style parallel block oracle (oracle.parallel_layer).

The block is pinned against facts outside the oracle: fp64 finite
differences of L = <dout, out> for every parameter and for x, fp64 torch
autograd of the same block written with torch's own layer_norm and
scaled-dot-product attention, the identity with every parameter zero, the
additivity of the two branches, and the QK-normalisation invariants.
Planted mistakes (the MLP fed by the attention output as in the sequential
block, the QK-norm backward dropped, normalisation over all heads at once,
values normalised too) must each fail a pin.
"""

import numpy as np
import torch
import torch.nn.functional as F

import oracle
from oracle import parallel_layer as PL


def _rng(seed):
    return np.random.default_rng(seed)


def _tiny_cfg(**kw):
    cfg = dict(batch=2, seq=3, hidden=8, heads=2, head_dim=4, mlp=16, ln_eps=1e-6)
    cfg.update(kw)
    return cfg


def _params(cfg, rng, scale=0.5):
    shapes = oracle.parallel_param_shapes(cfg["hidden"], cfg["heads"], cfg["head_dim"], cfg["mlp"])
    p = {}
    for n in oracle.PARALLEL_PARAM_NAMES:
        p[n] = rng.normal(size=shapes[n]) * scale
        if n in ("ln_g", "qn_g", "kn_g"):
            p[n] = 1.0 + p[n]
    return p


def _loss(cfg, p, x, dout):
    out, _ = oracle.parallel_layer_fwd(cfg, p, x)
    return float((out * dout).sum())


def fd_error(cfg, seed=21, h=1e-5):
    rng = _rng(seed)
    M = cfg["batch"] * cfg["seq"]
    x = rng.normal(size=(M, cfg["hidden"]))
    p = _params(cfg, rng)
    dout = rng.normal(size=(M, cfg["hidden"]))
    out, saved = oracle.parallel_layer_fwd(cfg, p, x)
    dx, grads, _ = oracle.parallel_layer_bwd(cfg, p, x, saved, dout)
    worst = 0.0
    for name, arr, an in [("x", x, dx)] + [(n, p[n], grads[n]) for n in oracle.PARALLEL_PARAM_NAMES]:
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
        worst = max(worst, np.abs(fd - an.reshape(-1)).max() / max(1.0, np.abs(an).max()))
    return worst


def test_gradients_finite_difference():
    assert fd_error(_tiny_cfg()) < 1e-6


def test_gradients_finite_difference_sharded_width():
    assert fd_error(_tiny_cfg(heads=1, head_dim=8, mlp=12, seq=4)) < 1e-6


def _torch_block(cfg, p, x):
    B, S, H = cfg["batch"], cfg["seq"], cfg["hidden"]
    nh, d, eps = cfg["heads"], cfg["head_dim"], cfg["ln_eps"]
    y = F.layer_norm(x, (H,), p["ln_g"], p["ln_b"], eps)
    qkv = F.linear(y, p["w_qkv"]).view(B, S, 3, nh, d)
    q = F.layer_norm(qkv[:, :, 0], (d,), p["qn_g"], p["qn_b"], eps).transpose(1, 2)
    k = F.layer_norm(qkv[:, :, 1], (d,), p["kn_g"], p["kn_b"], eps).transpose(1, 2)
    v = qkv[:, :, 2].transpose(1, 2)
    o = F.scaled_dot_product_attention(q, k, v).transpose(1, 2).reshape(B * S, nh * d)
    g = F.gelu(F.linear(y, p["w_1"], p["b_1"]), approximate="none")
    return x + F.linear(o, p["w_o"], p["b_o"]) + F.linear(g, p["w_2"], p["b_2"])


def torch_error(cfg, seed=22):
    rng = _rng(seed)
    M = cfg["batch"] * cfg["seq"]
    x = rng.normal(size=(M, cfg["hidden"]))
    p = _params(cfg, rng, scale=0.1)
    dout = rng.normal(size=(M, cfg["hidden"]))
    out, saved = oracle.parallel_layer_fwd(cfg, p, x)
    dx, grads, _ = oracle.parallel_layer_bwd(cfg, p, x, saved, dout)
    tx = torch.from_numpy(x).requires_grad_()
    tp = {n: torch.from_numpy(v).requires_grad_() for n, v in p.items()}
    tout = _torch_block(cfg, tp, tx)
    tout.backward(torch.from_numpy(dout))
    errs = [np.abs(out - tout.detach().numpy()).max() / np.abs(out).max(),
            np.abs(dx - tx.grad.numpy()).max() / np.abs(dx).max()]
    for n in oracle.PARALLEL_PARAM_NAMES:
        ref = tp[n].grad.numpy()
        if n == "kn_b":  # identically zero (see test_key_norm_bias_gradient_vanishes): compare absolutely
            errs.append(np.abs(grads[n] - ref).max() / np.abs(grads["kn_g"]).max())
            continue
        errs.append(np.abs(grads[n] - ref).max() / max(np.abs(ref).max(), 1e-300))
    return max(errs)


def test_key_norm_bias_gradient_vanishes():
    # adding one vector to every key shifts each query's logits by a constant,
    # which the softmax ignores: the key-norm bias has zero gradient
    cfg = _tiny_cfg(seq=5)
    rng = _rng(26)
    M = cfg["batch"] * cfg["seq"]
    x, dout = rng.normal(size=(M, cfg["hidden"])), rng.normal(size=(M, cfg["hidden"]))
    p = _params(cfg, rng)
    out, saved = oracle.parallel_layer_fwd(cfg, p, x)
    _, grads, _ = oracle.parallel_layer_bwd(cfg, p, x, saved, dout)
    assert np.abs(grads["kn_b"]).max() < 1e-12 * np.abs(grads["kn_g"]).max() + 1e-14
    assert np.abs(grads["qn_b"]).max() > 1e-3


def test_matches_torch_composition():
    assert torch_error(dict(batch=2, seq=19, hidden=64, heads=2, head_dim=32, mlp=96, ln_eps=1e-6)) < 1e-10


def test_matches_torch_composition_d80():
    assert torch_error(dict(batch=1, seq=11, hidden=48, heads=2, head_dim=80, mlp=64, ln_eps=1e-6)) < 1e-10


def test_zero_parameters_give_the_identity():
    cfg = _tiny_cfg(seq=5)
    rng = _rng(23)
    M, H = cfg["batch"] * cfg["seq"], cfg["hidden"]
    shapes = oracle.parallel_param_shapes(H, cfg["heads"], cfg["head_dim"], cfg["mlp"])
    p = {n: np.zeros(s) for n, s in shapes.items()}
    x, dout = rng.normal(size=(M, H)), rng.normal(size=(M, H))
    out, saved = oracle.parallel_layer_fwd(cfg, p, x)
    dx, grads, _ = oracle.parallel_layer_bwd(cfg, p, x, saved, dout)
    assert np.abs(out - x).max() < 1e-14 and np.abs(dx - dout).max() < 1e-14
    assert np.abs(grads["b_o"] - dout.sum(0)).max() < 1e-12
    assert np.abs(grads["b_2"] - dout.sum(0)).max() < 1e-12
    for n in oracle.PARALLEL_PARAM_NAMES:
        if n not in ("b_o", "b_2"):
            assert np.abs(grads[n]).max() < 1e-14, n


def test_branches_add():
    cfg = _tiny_cfg(seq=4)
    rng = _rng(24)
    x = rng.normal(size=(cfg["batch"] * cfg["seq"], cfg["hidden"]))
    p = _params(cfg, rng)
    full, _ = oracle.parallel_layer_fwd(cfg, p, x)
    pa = dict(p, w_2=np.zeros_like(p["w_2"]), b_2=np.zeros_like(p["b_2"]))   # attention branch alone
    pm = dict(p, w_o=np.zeros_like(p["w_o"]), b_o=np.zeros_like(p["b_o"]))   # MLP branch alone
    oa, _ = oracle.parallel_layer_fwd(cfg, pa, x)
    om, _ = oracle.parallel_layer_fwd(cfg, pm, x)
    assert np.abs((full - x) - ((oa - x) + (om - x))).max() < 1e-12


def test_qk_norm_invariants():
    rng = _rng(25)
    M, nh, d, eps = 7, 3, 16, 1e-6
    qkv = rng.normal(size=(M, 3 * nh * d)) * 3.0 + 1.5
    one, zero = np.ones(d), np.zeros(d)
    qkvn, st = oracle.qk_norm_fwd(qkv, nh, d, one, zero, one, zero, eps)
    A = nh * d
    for part, sl in (("q", slice(0, A)), ("k", slice(A, 2 * A))):
        t = qkvn[:, sl].reshape(M, nh, d)
        raw = qkv[:, sl].reshape(M, nh, d)
        var = raw.var(axis=-1)
        assert np.abs(t.mean(axis=-1)).max() < 1e-12, part
        assert np.abs(t.var(axis=-1) - var / (var + eps)).max() < 1e-12, part
    assert np.array_equal(qkvn[:, 2 * A:], qkv[:, 2 * A:])   # values untouched


# ---- planted mistakes

def test_mutant_sequential_mlp_input_is_caught(monkeypatch):
    real = PL.parallel_layer_fwd

    def bad(cfg, p, x):
        out, s = real(cfg, p, x)
        y2 = oracle.layernorm_fwd(s["h"], p["ln_g"], p["ln_b"], cfg["ln_eps"])[0]
        g = oracle.gelu(oracle.linear_fwd(y2, p["w_1"], p["b_1"]))
        return oracle.linear_fwd(g, p["w_2"], p["b_2"], resid=s["h"]), s
    monkeypatch.setattr(oracle, "parallel_layer_fwd", bad)
    assert torch_error(dict(batch=1, seq=7, hidden=32, heads=2, head_dim=16, mlp=48, ln_eps=1e-6)) > 1e-3


def test_mutant_dropped_qk_norm_backward_is_caught(monkeypatch):
    def bad(dqkvn, qkv, stats, heads, d, qg, kg):
        z = np.zeros(d)
        return dqkvn.copy(), {"qn_g": z, "qn_b": z, "kn_g": z, "kn_b": z}
    monkeypatch.setattr(PL, "qk_norm_bwd", bad)
    assert fd_error(_tiny_cfg()) > 1e-3


def test_mutant_joint_head_normalisation_is_caught(monkeypatch):
    def bad(qkv, heads, d, qg, qb, kg, kb, eps):
        M, A = qkv.shape[0], heads * d
        q, qm, qr = oracle.layernorm_fwd(qkv[:, :A], np.tile(qg, heads), np.tile(qb, heads), eps)
        k, km, kr = oracle.layernorm_fwd(qkv[:, A:2 * A], np.tile(kg, heads), np.tile(kb, heads), eps)
        st = dict(qmean=np.repeat(qm[:, None], heads, 1), qrstd=np.repeat(qr[:, None], heads, 1),
                  kmean=np.repeat(km[:, None], heads, 1), krstd=np.repeat(kr[:, None], heads, 1))
        return np.concatenate([q, k, qkv[:, 2 * A:]], axis=1), st
    monkeypatch.setattr(PL, "qk_norm_fwd", bad)
    assert torch_error(dict(batch=1, seq=7, hidden=32, heads=2, head_dim=16, mlp=48, ln_eps=1e-6)) > 1e-3


def test_mutant_normalised_values_are_caught(monkeypatch):
    real = PL.qk_norm_fwd

    def bad(qkv, heads, d, qg, qb, kg, kb, eps):
        qkvn, st = real(qkv, heads, d, qg, qb, kg, kb, eps)
        M, A = qkv.shape[0], heads * d
        v = oracle.layernorm_fwd(qkv[:, 2 * A:].reshape(M * heads, d), np.ones(d), np.zeros(d), eps)[0]
        qkvn[:, 2 * A:] = v.reshape(M, A)
        return qkvn, st
    monkeypatch.setattr(PL, "qk_norm_fwd", bad)
    assert torch_error(dict(batch=1, seq=7, hidden=32, heads=2, head_dim=16, mlp=48, ln_eps=1e-6)) > 1e-3
