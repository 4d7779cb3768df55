"""Parity of the ViT-22B-style parallel block's HIP path (through the C ABI)
against its oracle: QK normalisation forward and backward, the bias-free QKV
projection and the input gradient with addend (integer-exact), the whole
block element by element at small shapes, and the full ViT-22B width on
sampled rows / heads with every step fed the GPU's own inputs."""

import numpy as np
import pytest
import torch

import oracle
from helpers import TOL_ACT, TOL_GRAD, announce, cuda, f64, max_rel
from paper_2408_03505_amd import binding as B
from paper_2408_03505_amd.synthetic import (CONFIGS, PPARAM_ORDER, parallel_block_inputs, random_bf16,
                                            random_int_bf16, random_sparse_sign_bf16)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

SMALL = {
    "tiny_d64": dict(batch=2, seq=197, hidden=192, heads=3, head_dim=64, mlp=768, ln_eps=1e-6),
    "d80": dict(batch=2, seq=65, hidden=256, heads=2, head_dim=80, mlp=320, ln_eps=1e-6),
    "d128_ragged": dict(batch=3, seq=33, hidden=384, heads=2, head_dim=128, mlp=1024, ln_eps=1e-5),
}


def _affine(d, seed):
    g = 1.0 + 0.3 * random_bf16((d,), seed).float()
    return g.to(torch.bfloat16), (0.3 * random_bf16((d,), seed + 1).float()).to(torch.bfloat16)


@pytest.mark.parametrize("M,nh,d", [(197, 3, 64), (65, 2, 80), (33, 4, 128), (1, 1, 64), (300, 48, 128)])
def test_qk_norm_fwd(M, nh, d):
    announce(f"qk_norm_fwd M={M} heads={nh} d={d}")
    qkv = (random_bf16((M, 3 * nh * d), 31, 2.0).float() + 0.7).to(torch.bfloat16)
    qg, qb = _affine(d, 32)
    kg, kb = _affine(d, 34)
    qkvn, st = B.enc_qk_norm_fwd(nh, d, cuda(qkv), cuda(qg), cuda(qb), cuda(kg), cuda(kb), 1e-6)
    torch.cuda.synchronize()
    rq, rst = oracle.qk_norm_fwd(f64(qkv), nh, d, f64(qg), f64(qb), f64(kg), f64(kb), 1e-6)
    A = nh * d
    assert max_rel(f64(qkvn[:, :2 * A]), rq[:, :2 * A]) < TOL_ACT
    assert torch.equal(qkvn[:, 2 * A:].cpu().view(torch.int16), qkv[:, 2 * A:].view(torch.int16))
    gst = f64(st)
    for i, k in enumerate(("qmean", "qrstd", "kmean", "krstd")):
        assert max_rel(gst[:, :, i], rst[k]) < 1e-4, k


@pytest.mark.parametrize("M,nh,d", [(197, 3, 64), (65, 2, 80), (33, 4, 128), (300, 48, 128)])
def test_qk_norm_bwd(M, nh, d):
    announce(f"qk_norm_bwd M={M} heads={nh} d={d}")
    qkv = (random_bf16((M, 3 * nh * d), 41, 2.0).float() - 0.4).to(torch.bfloat16)
    dqkvn = random_bf16((M, 3 * nh * d), 42)
    qg, qb = _affine(d, 43)
    kg, kb = _affine(d, 45)
    _, st = B.enc_qk_norm_fwd(nh, d, cuda(qkv), cuda(qg), cuda(qb), cuda(kg), cuda(kb), 1e-6)
    dqkv, grads = B.enc_qk_norm_bwd(nh, d, cuda(dqkvn), cuda(qkv), st, cuda(qg), cuda(kg))
    torch.cuda.synchronize()
    _, rst = oracle.qk_norm_fwd(f64(qkv), nh, d, f64(qg), f64(qb), f64(kg), f64(kb), 1e-6)
    rdq, rg = oracle.qk_norm_bwd(f64(dqkvn), f64(qkv), rst, nh, d, f64(qg), f64(kg))
    A = nh * d
    assert max_rel(f64(dqkv[:, :2 * A]), rdq[:, :2 * A]) < TOL_GRAD
    assert torch.equal(dqkv[:, 2 * A:].cpu().view(torch.int16), dqkvn[:, 2 * A:].view(torch.int16))
    for n in ("qn_g", "qn_b", "kn_g", "kn_b"):
        assert max_rel(f64(grads[n]), rg[n]) < TOL_GRAD, n
    # accumulate adds the same fixed-order sums: exactly twice the first result
    first = {n: grads[n].clone() for n in grads}
    B.enc_qk_norm_bwd(nh, d, cuda(dqkvn), cuda(qkv), st, cuda(qg), cuda(kg), grads=grads, accumulate=True)
    torch.cuda.synchronize()
    for n in grads:
        assert torch.equal(grads[n], 2 * first[n]), n


@pytest.mark.parametrize("M,K,N", [(394, 192, 576), (2048, 6144, 2304), (130, 256, 384)])
def test_qkv_fwd_without_bias_exact(M, K, N):
    announce(f"qkv_fwd no bias M={M} K={K} N={N}")
    X = random_sparse_sign_bf16((M, K), 51, 0.02 if K > 1024 else 0.2)
    W = random_sparse_sign_bf16((N, K), 52, 0.5)
    Y = B.enc_qkv_fwd(cuda(X), cuda(W), None)
    torch.cuda.synchronize()
    assert np.array_equal(f64(Y), oracle.linear_fwd(f64(X), f64(W)))


@pytest.mark.parametrize("M,N3,H", [(394, 576, 192), (2048, 2304, 6144), (130, 384, 256)])
def test_qkv_bwd_data_add_exact(M, N3, H):
    announce(f"qkv_bwd_data_add M={M} 3A={N3} H={H}")
    dY = random_sparse_sign_bf16((M, N3), 53, 0.05 if N3 > 1024 else 0.2)
    W = random_sparse_sign_bf16((N3, H), 54, 0.5)
    R = random_int_bf16((M, H), 55, -4, 4)
    dy = B.enc_qkv_bwd_data_add(cuda(dY), cuda(W), cuda(R))
    torch.cuda.synchronize()
    assert np.array_equal(f64(dy), oracle.linear_bwd_data(f64(dY), f64(W)) + f64(R))


def _gpu(params):
    return {n: cuda(params[n]) for n in PPARAM_ORDER}


def _run(cfg, x, gp, dout):
    out, saved = B.encoder_parallel_fwd(cfg, gp, x)
    dx, grads = B.encoder_parallel_bwd(cfg, gp, x, saved, dout)
    torch.cuda.synchronize()
    return out, saved, dx, grads


def _grad_errors(grads, rgrads, dx, rdx):
    errs = {"dx": max_rel(f64(dx), rdx)}
    for n in PPARAM_ORDER:
        if n == "kn_b":  # identically zero in exact arithmetic: compare against the key-norm scale's gradient
            errs[n] = np.abs(f64(grads[n]) - rgrads[n]).max() / np.abs(rgrads["kn_g"]).max()
        else:
            errs[n] = max_rel(f64(grads[n]), rgrads[n])
    return errs


@pytest.mark.parametrize("name", list(SMALL))
def test_parallel_block_matches_oracle_elementwise(name):
    cfg = SMALL[name]
    announce(f"parallel block fwd+bwd {name} {cfg}")
    x, params, dout = parallel_block_inputs(cfg, seed=0)
    out, saved, dx, grads = _run(cfg, cuda(x), _gpu(params), cuda(dout))
    p64 = {n: f64(params[n]) for n in PPARAM_ORDER}
    rout, rs = oracle.parallel_layer_fwd(cfg, p64, f64(x))
    rdx, rgrads, _ = oracle.parallel_layer_bwd(cfg, p64, f64(x), rs, f64(dout))
    v = B.parallel_saved_views(cfg, saved)
    errs = {"out": max_rel(f64(out), rout)}
    for k in ("y", "qkv", "qkvn", "o", "h", "u", "g", "mean", "rstd", "lse"):
        errs[k] = max_rel(f64(v[k]), rs[k])
    st = f64(v["qkstats"])
    for i, k in enumerate(("qmean", "qrstd", "kmean", "krstd")):
        errs[k] = max_rel(st[:, :, i], rs[k])
    for k, e in errs.items():
        assert e < TOL_ACT, (k, e)
    gerrs = _grad_errors(grads, rgrads, dx, rdx)
    for k, e in gerrs.items():
        assert e < TOL_GRAD, (k, e)
    print(f"[parity] parallel {name}: act {max(errs.values()):.3e}, grad {max(gerrs.values()):.3e}")


def test_parallel_block_is_deterministic_and_accumulates():
    cfg = SMALL["d128_ragged"]
    announce("parallel block determinism + accumulate")
    x, params, dout = parallel_block_inputs(cfg, seed=5)
    gp, gx, gd = _gpu(params), cuda(x), cuda(dout)
    out1, saved1, dx1, g1 = _run(cfg, gx, gp, gd)
    out2, saved2, dx2, g2 = _run(cfg, gx, gp, gd)
    assert torch.equal(out1.view(torch.int16), out2.view(torch.int16))
    assert torch.equal(dx1.view(torch.int16), dx2.view(torch.int16))
    for n in PPARAM_ORDER:
        assert torch.equal(g1[n], g2[n]), n
    B.encoder_parallel_bwd(cfg, gp, gx, saved1, gd, grads=g2, accumulate=True)
    torch.cuda.synchronize()
    for n in PPARAM_ORDER:
        assert torch.equal(g2[n], 2 * g1[n]), n


def _parallel_chain_by_kernels(cfg, x, p, dout):
    """The parallel block through the per-kernel entry points, in the
    composite's order, with every product unsplit as the block's composites
    run them; returns every step's output."""
    Bn, S, nh, d, eps = cfg["batch"], cfg["seq"], cfg["heads"], cfg["head_dim"], cfg["ln_eps"]
    t = {}
    t["y"], t["mean"], t["rstd"] = B.enc_ln_fwd(x, p["ln_g"], p["ln_b"], eps)
    t["qkv"] = B.enc_qkv_fwd(t["y"], p["w_qkv"], None, split=False)
    t["qkvn"], t["qkstats"] = B.enc_qk_norm_fwd(nh, d, t["qkv"], p["qn_g"], p["qn_b"], p["kn_g"], p["kn_b"], eps)
    t["o"], t["lse"] = B.enc_attn_fwd(Bn, S, nh, d, t["qkvn"])
    t["h"] = B.enc_oproj_fwd(t["o"], p["w_o"], p["b_o"], x, split=False)
    t["u"], t["g"] = B.enc_mlp_up_fwd(t["y"], p["w_1"], p["b_1"], split=False)
    t["out"] = B.enc_mlp_down_fwd(t["g"], p["w_2"], p["b_2"], t["h"], split=False)
    t["du"] = B.enc_mlp_down_bwd_data(dout, p["w_2"], t["u"], split=False)
    t["dw_2"], t["db_2"] = B.enc_linear_bwd_weight(dout, t["g"], split=False)
    t["dy_mlp"] = B.enc_mlp_up_bwd_data(t["du"], p["w_1"], split=False)
    t["dw_1"], t["db_1"] = B.enc_linear_bwd_weight(t["du"], t["y"], split=False)
    t["do"] = B.enc_oproj_bwd_data(dout, p["w_o"], split=False)
    t["dw_o"], t["db_o"] = B.enc_linear_bwd_weight(dout, t["o"], split=False)
    t["dqkvn"] = B.enc_attn_bwd(Bn, S, nh, d, t["qkvn"], t["o"], t["lse"], t["do"])
    t["dqkv"], qg = B.enc_qk_norm_bwd(nh, d, t["dqkvn"], t["qkv"], t["qkstats"], p["qn_g"], p["kn_g"])
    t.update({"d" + n: v for n, v in qg.items()})
    t["dw_qkv"], _ = B.enc_linear_bwd_weight(t["dqkv"], t["y"], with_db=False, split=False)
    t["dy"] = B.enc_qkv_bwd_data_add(t["dqkv"], p["w_qkv"], t["dy_mlp"], split=False)
    t["dx"], t["dln_g"], t["dln_b"] = B.enc_ln_bwd(t["dy"], x, t["mean"], t["rstd"], p["ln_g"], dresid=dout)
    torch.cuda.synchronize()
    return t


def _rows(M, n, seed):
    rng = np.random.default_rng(seed)
    r = set(rng.choice(M, size=min(n, M), replace=False).tolist()) | {0, M - 1}
    return np.array(sorted(r))


@pytest.mark.parametrize("name", ["vit22b_tp8", "vit22b"])
def test_parallel_full_size_sampled(name):
    cfg = CONFIGS[name]
    announce(f"parallel block full size {name} {cfg}")
    Bn, S, H, nh, d = cfg["batch"], cfg["seq"], cfg["hidden"], cfg["heads"], cfg["head_dim"]
    M, eps = Bn * S, cfg["ln_eps"]
    x, params, dout = parallel_block_inputs(cfg, seed=0)
    gp, gx, gd = _gpu(params), cuda(x), cuda(dout)
    t = _parallel_chain_by_kernels(cfg, gx, gp, gd)
    out, saved, dx, grads = _run(cfg, gx, gp, gd)
    v = B.parallel_saved_views(cfg, saved)
    assert torch.equal(out.view(torch.int16), t["out"].view(torch.int16))
    for k in ("y", "qkv", "qkvn", "o", "h", "u", "g", "mean", "rstd", "lse", "qkstats"):
        assert torch.equal(v[k].contiguous().view(-1).view(torch.uint8), t[k].contiguous().view(-1).view(torch.uint8)), k
    assert torch.equal(dx.view(torch.int16), t["dx"].view(torch.int16))
    for n in PPARAM_ORDER:
        assert torch.equal(grads[n], t["d" + n]), n
    del out, saved, dx, grads, v

    rows = _rows(M, 12, 7)
    ridx = torch.as_tensor(rows, device="cuda")
    R = lambda k: f64(t[k][ridx])  # noqa: E731
    P = lambda n: f64(params[n])  # noqa: E731
    X = f64(x[torch.as_tensor(rows)])
    errs = {"ln": max_rel(R("y"), oracle.layernorm_fwd(X, P("ln_g"), P("ln_b"), eps)[0]),
            "qkv": max_rel(R("qkv"), oracle.linear_fwd(R("y"), P("w_qkv"))),
            "qk_norm": max_rel(R("qkvn"), oracle.qk_norm_fwd(R("qkv"), nh, d, P("qn_g"), P("qn_b"), P("kn_g"),
                                                             P("kn_b"), eps)[0]),
            "oproj": max_rel(R("h"), oracle.linear_fwd(R("o"), P("w_o"), P("b_o"), resid=X))}
    ru = oracle.linear_fwd(R("y"), P("w_1"), P("b_1"))
    errs["mlp_up"] = max(max_rel(R("u"), ru), max_rel(R("g"), oracle.gelu(ru)))
    errs["mlp_down"] = max_rel(R("out"), oracle.linear_fwd(R("g"), P("w_2"), P("b_2"), resid=R("h")))
    for (b, hh) in ((0, 0), (Bn - 1, nh - 1)):
        seq = f64(t["qkvn"][b * S:(b + 1) * S]).reshape(S, 3, nh, d)[:, :, hh].reshape(S, 3 * d)
        ro, _ = oracle.attention_fwd(seq, 1, S, 1, d)
        errs[f"attn[{b},{hh}]"] = max_rel(f64(t["o"][b * S:(b + 1) * S, hh * d:(hh + 1) * d]), ro)
    for k, e in errs.items():
        assert e < TOL_ACT, (k, e)
    dO = f64(gd[ridx])
    gerrs = {"du": max_rel(R("du"), oracle.linear_bwd_data(dO, P("w_2")) * oracle.gelu_grad(R("u"))),
             "dy_mlp": max_rel(R("dy_mlp"), oracle.linear_bwd_data(R("du"), P("w_1"))),
             "do": max_rel(R("do"), oracle.linear_bwd_data(dO, P("w_o"))),
             "dy": max_rel(R("dy"), oracle.linear_bwd_data(R("dqkv"), P("w_qkv")) + R("dy_mlp"))}
    st = {k: f64(t["qkstats"][ridx])[:, :, i] for i, k in enumerate(("qmean", "qrstd", "kmean", "krstd"))}
    rdq, _ = oracle.qk_norm_bwd(R("dqkvn"), R("qkv"), st, nh, d, P("qn_g"), P("kn_g"))
    gerrs["qk_norm_bwd"] = max_rel(R("dqkv"), rdq)
    for k, e in gerrs.items():
        assert e < TOL_GRAD, (k, e)
    print(f"[parity] parallel {name} sampled: act {max(errs.values()):.3e}, grad {max(gerrs.values()):.3e}")
