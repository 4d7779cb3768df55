"""Whole-layer parity of the HIP chain (through the C ABI) against the oracle.

Small configurations are compared element by element: the layer output, every
saved intermediate, dx and all twelve parameter gradients.  The full-size
workloads (ViT-Base, ViT-Huge, the ViT-22B tensor-parallel shard and the full
ViT-22B layer) run the chain kernel by kernel through the per-kernel entry
points, check each step's output on sampled rows / heads against the oracle
step fed with the GPU's own inputs, and check that the composite entry points
reproduce the step-by-step chain bit for bit.  Also: run-to-run determinism,
gradient accumulation and HIP-graph capture.
"""

import numpy as np
import pytest
import torch

import oracle
from helpers import TOL_ACT, TOL_GRAD, announce, cuda, f64, max_rel
from paper_2408_03505_amd import binding as B
from paper_2408_03505_amd.synthetic import CONFIGS, PARAM_ORDER, layer_inputs

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

SMALL_CONFIGS = {
    "vit_tiny": CONFIGS["vit_tiny"],
    "shard_d80": dict(batch=2, seq=65, hidden=256, heads=2, head_dim=80, mlp=320, ln_eps=1e-6),
    "huge_one_seq": dict(batch=1, seq=257, hidden=1280, heads=16, head_dim=80, mlp=5120, ln_eps=1e-6),
    "d128_ragged": dict(batch=3, seq=33, hidden=384, heads=2, head_dim=128, mlp=1024, ln_eps=1e-5),
}

def _gpu_params(params):
    return {n: cuda(params[n]) for n in PARAM_ORDER}


def run_layer(cfg, x, params, dout):
    out, saved = B.encoder_layer_fwd(cfg, params, x)
    dx, grads = B.encoder_layer_bwd(cfg, params, x, saved, dout)
    torch.cuda.synchronize()
    return out, saved, dx, grads


@pytest.mark.parametrize("name", list(SMALL_CONFIGS))
def test_layer_matches_oracle_elementwise(name):
    cfg = SMALL_CONFIGS[name]
    announce(f"layer fwd+bwd elementwise {name} {cfg}")
    x, params, dout = layer_inputs(cfg, seed=0)
    gp = _gpu_params(params)
    out, saved, dx, grads = run_layer(cfg, cuda(x), gp, cuda(dout))
    p64 = {n: f64(params[n]) for n in PARAM_ORDER}
    rout, rsaved = oracle.layer_fwd(cfg, p64, f64(x))
    rdx, rgrads, _ = oracle.layer_bwd(cfg, p64, f64(x), rsaved, f64(dout))
    views = B.saved_views(cfg, saved)
    errs = {"out": max_rel(f64(out), rout)}
    for k in ("y1", "qkv", "o", "h", "y2", "u", "g"):
        errs[k] = max_rel(f64(views[k]), rsaved[k])
    for k in ("mean1", "rstd1", "mean2", "rstd2", "lse"):
        errs[k] = max_rel(f64(views[k]), rsaved[k])
    for k, e in errs.items():
        assert e < TOL_ACT, (k, e, errs)
    gerrs = {"dx": max_rel(f64(dx), rdx)}
    for n in PARAM_ORDER:
        gerrs[n] = max_rel(f64(grads[n]), rgrads[n])
    for k, e in gerrs.items():
        assert e < TOL_GRAD, (k, e, gerrs)
    print(f"[parity] {name} max act err {max(errs.values()):.3e}, max grad err {max(gerrs.values()):.3e}")


def test_layer_is_deterministic_and_accumulates():
    cfg = SMALL_CONFIGS["vit_tiny"]
    announce("layer determinism + accumulate")
    x, params, dout = layer_inputs(cfg, seed=3)
    gp = _gpu_params(params)
    x, dout = cuda(x), cuda(dout)
    out1, saved1, dx1, g1 = run_layer(cfg, x, gp, dout)
    out2, saved2, dx2, g2 = run_layer(cfg, x, gp, dout)
    assert torch.equal(out1.view(torch.int16), out2.view(torch.int16))
    v1, v2 = B.saved_views(cfg, saved1), B.saved_views(cfg, saved2)
    for k in v1:  # the alignment padding between saved tensors is never written
        assert torch.equal(v1[k].contiguous().view(torch.uint8), v2[k].contiguous().view(torch.uint8)), k
    assert torch.equal(dx1.view(torch.int16), dx2.view(torch.int16))
    for n in PARAM_ORDER:
        assert torch.equal(g1[n], g2[n]), n
    acc = {n: g1[n].clone() for n in PARAM_ORDER}
    B.encoder_layer_bwd(cfg, gp, x, saved1, dout, grads=acc, accumulate=True)
    torch.cuda.synchronize()
    for n in PARAM_ORDER:
        assert torch.equal(acc[n], 2 * g1[n]), n


def test_layer_graph_capture_replays_match_eager():
    cfg = SMALL_CONFIGS["shard_d80"]
    announce("layer graph capture")
    x, params, dout = layer_inputs(cfg, seed=4)
    gp = _gpu_params(params)
    x, dout = cuda(x), cuda(dout)
    out_e, saved_e, dx_e, g_e = run_layer(cfg, x, gp, dout)
    M, H = x.shape
    out = torch.empty_like(out_e)
    saved = torch.empty_like(saved_e)
    dx = torch.empty_like(dx_e)
    grads = {n: torch.empty_like(g_e[n]) for n in PARAM_ORDER}
    ws = torch.empty(B.layer_workspace_bytes(cfg), dtype=torch.uint8, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):  # warm up on the capture stream
        B.encoder_layer_fwd(cfg, gp, x, out=out, saved=saved)
        B.encoder_layer_bwd(cfg, gp, x, saved, dout, grads=grads, dx=dx, ws=ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        B.encoder_layer_fwd(cfg, gp, x, out=out, saved=saved)
        B.encoder_layer_bwd(cfg, gp, x, saved, dout, grads=grads, dx=dx, ws=ws)
    for rep in range(3):
        out.zero_(); dx.zero_()
        for n in PARAM_ORDER:
            grads[n].fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), out_e.view(torch.int16)), rep
        assert torch.equal(dx.view(torch.int16), dx_e.view(torch.int16)), rep
        for n in PARAM_ORDER:
            assert torch.equal(grads[n], g_e[n]), (rep, n)
        # unrelated eager work between replays
        _ = run_layer(cfg, x, gp, dout)


# --------------------------------------------------------------------------- full-size workloads

def _sample_rows(M, n, seed):
    rng = np.random.default_rng(seed)
    rows = set(rng.choice(M, size=min(n, M), replace=False).tolist())
    rows.update({0, M - 1})
    return np.array(sorted(rows))


def _chain_by_kernels(cfg, x, p, dout):
    """Run the layer through the per-kernel entry points in the composite's
    order; return every step's output."""
    Bn, S, H, nh, d, F = cfg["batch"], cfg["seq"], cfg["hidden"], cfg["heads"], cfg["head_dim"], cfg["mlp"]
    eps = cfg["ln_eps"]
    t = {}
    t["y1"], t["mean1"], t["rstd1"] = B.enc_ln_fwd(x, p["ln1_g"], p["ln1_b"], eps)
    t["qkv"] = B.enc_qkv_fwd(t["y1"], p["w_qkv"], p["b_qkv"])
    t["o"], t["lse"] = B.enc_attn_fwd(Bn, S, nh, d, t["qkv"])
    t["h"] = B.enc_oproj_fwd(t["o"], p["w_o"], p["b_o"], x)
    t["y2"], t["mean2"], t["rstd2"] = B.enc_ln_fwd(t["h"], p["ln2_g"], p["ln2_b"], eps)
    t["u"], t["g"] = B.enc_mlp_up_fwd(t["y2"], p["w_1"], p["b_1"])
    t["out"] = B.enc_mlp_down_fwd(t["g"], p["w_2"], p["b_2"], t["h"])
    t["du"] = B.enc_mlp_down_bwd_data(dout, p["w_2"], t["u"])
    t["dw_2"], t["db_2"] = B.enc_linear_bwd_weight(dout, t["g"])
    t["dy2"] = B.enc_mlp_up_bwd_data(t["du"], p["w_1"])
    t["dw_1"], t["db_1"] = B.enc_linear_bwd_weight(t["du"], t["y2"])
    t["dh"], t["dln2_g"], t["dln2_b"] = B.enc_ln_bwd(t["dy2"], t["h"], t["mean2"], t["rstd2"], p["ln2_g"], dresid=dout)
    t["do"] = B.enc_oproj_bwd_data(t["dh"], p["w_o"])
    t["dw_o"], t["db_o"] = B.enc_linear_bwd_weight(t["dh"], t["o"])
    t["dqkv"] = B.enc_attn_bwd(Bn, S, nh, d, t["qkv"], t["o"], t["lse"], t["do"])
    t["dy1"] = B.enc_qkv_bwd_data(t["dqkv"], p["w_qkv"])
    t["dw_qkv"], t["db_qkv"] = B.enc_linear_bwd_weight(t["dqkv"], t["y1"])
    t["dx"], t["dln1_g"], t["dln1_b"] = B.enc_ln_bwd(t["dy1"], x, t["mean1"], t["rstd1"], p["ln1_g"], dresid=t["dh"])
    torch.cuda.synchronize()
    return t


@pytest.mark.parametrize("name", ["vit_base", "vit_huge", "vit22b_tp8", "vit22b"])
def test_full_size_chain_sampled(name):
    cfg = CONFIGS[name]
    announce(f"full-size chain {name} {cfg}")
    Bn, S, H, nh, d, F = cfg["batch"], cfg["seq"], cfg["hidden"], cfg["heads"], cfg["head_dim"], cfg["mlp"]
    M, A, eps = Bn * S, nh * d, cfg["ln_eps"]
    x, params, dout = layer_inputs(cfg, seed=0)
    gp = _gpu_params(params)
    gx, gd = cuda(x), cuda(dout)
    t = _chain_by_kernels(cfg, gx, gp, gd)

    # The composite entry points run the same kernels: bitwise equal.
    out, saved, dx, grads = run_layer(cfg, gx, gp, gd)
    views = B.saved_views(cfg, saved)
    assert torch.equal(out.view(torch.int16), t["out"].view(torch.int16))
    for k in ("y1", "qkv", "o", "h", "y2", "u", "g", "mean1", "rstd1", "mean2", "rstd2", "lse"):
        assert torch.equal(views[k].contiguous().view(-1).view(torch.uint8),
                           t[k].contiguous().view(-1).view(torch.uint8)), k
    assert torch.equal(dx.view(torch.int16), t["dx"].view(torch.int16))
    gmap = {"w_2": "dw_2", "b_2": "db_2", "w_1": "dw_1", "b_1": "db_1", "w_o": "dw_o", "b_o": "db_o",
            "w_qkv": "dw_qkv", "b_qkv": "db_qkv", "ln1_g": "dln1_g", "ln1_b": "dln1_b", "ln2_g": "dln2_g",
            "ln2_b": "dln2_b"}
    for n, k in gmap.items():
        assert torch.equal(grads[n], t[k]), n
    del out, saved, dx, grads, views

    # Each step against the oracle step fed with the GPU's own inputs.
    rows = _sample_rows(M, 12, 7)
    lse_all = f64(t["lse"])
    rowsof = lambda k: f64(t[k][torch.as_tensor(rows, device="cuda")])  # noqa: E731
    P = lambda n: f64(params[n])  # noqa: E731
    X = f64(x[torch.as_tensor(rows)])
    errs = {}
    ry, rm, rr = oracle.layernorm_fwd(X, P("ln1_g"), P("ln1_b"), eps)
    errs["ln1"] = max_rel(rowsof("y1"), ry)
    errs["qkv"] = max_rel(rowsof("qkv"), oracle.linear_fwd(rowsof("y1"), P("w_qkv"), P("b_qkv")))
    errs["oproj"] = max_rel(rowsof("h"), oracle.linear_fwd(rowsof("o"), P("w_o"), P("b_o"), resid=X))
    ry2, _, _ = oracle.layernorm_fwd(rowsof("h"), P("ln2_g"), P("ln2_b"), eps)
    errs["ln2"] = max_rel(rowsof("y2"), ry2)
    ru = oracle.linear_fwd(rowsof("y2"), P("w_1"), P("b_1"))
    errs["mlp_up.u"] = max_rel(rowsof("u"), ru)
    errs["mlp_up.g"] = max_rel(rowsof("g"), oracle.gelu(ru))
    errs["mlp_down"] = max_rel(rowsof("out"), oracle.linear_fwd(rowsof("g"), P("w_2"), P("b_2"), resid=rowsof("h")))
    # attention: a few whole (sequence, head) pairs
    qkv_all = t["qkv"]
    rng = np.random.default_rng(9)
    pairs = {(0, 0), (Bn - 1, nh - 1)} | {(int(rng.integers(Bn)), int(rng.integers(nh))) for _ in range(2)}
    for (b, hh) in sorted(pairs):
        seq = f64(qkv_all[b * S:(b + 1) * S]).reshape(S, 3, nh, d)[:, :, hh].reshape(S, 3 * d)
        ro, rl = oracle.attention_fwd(seq, 1, S, 1, d)
        go = f64(t["o"][b * S:(b + 1) * S, hh * d:(hh + 1) * d])
        errs[f"attn_fwd[{b},{hh}]"] = max_rel(go, ro)
        errs[f"lse[{b},{hh}]"] = max_rel(lse_all[b, hh], rl[0, 0])
        dO = f64(t["do"][b * S:(b + 1) * S, hh * d:(hh + 1) * d])
        rdq = oracle.attention_bwd(seq, dO, 1, S, 1, d)
        gdq = f64(t["dqkv"][b * S:(b + 1) * S]).reshape(S, 3, nh, d)[:, :, hh].reshape(S, 3 * d)
        for i, part in enumerate(("dq", "dk", "dv")):
            errs[f"attn_bwd.{part}[{b},{hh}]"] = max_rel(gdq[:, i * d:(i + 1) * d], rdq[:, i * d:(i + 1) * d])
    for k, e in errs.items():
        tol = TOL_GRAD if k.startswith("attn_bwd") else TOL_ACT
        assert e < tol, (k, e)

    gerrs = {}
    dout_rows = f64(gd[torch.as_tensor(rows, device="cuda")])
    gerrs["mlp_down_bwd_data"] = max_rel(
        rowsof("du"), oracle.linear_bwd_data(dout_rows, P("w_2")) * oracle.gelu_grad(rowsof("u")))
    gerrs["mlp_up_bwd_data"] = max_rel(rowsof("dy2"), oracle.linear_bwd_data(rowsof("du"), P("w_1")))
    gerrs["oproj_bwd_data"] = max_rel(rowsof("do"), oracle.linear_bwd_data(rowsof("dh"), P("w_o")))
    gerrs["qkv_bwd_data"] = max_rel(rowsof("dy1"), oracle.linear_bwd_data(rowsof("dqkv"), P("w_qkv")))
    # LayerNorm backward: dx on sampled rows, dgamma/dbeta over all rows
    for ln, dy, xin, mean, rstd, gam, dres, dxk in (
            ("ln2", "dy2", "h", "mean2", "rstd2", "ln2_g", None, "dh"),
            ("ln1", "dy1", None, "mean1", "rstd1", "ln1_g", "dh", "dx")):
        xin_all = f64(t[xin]) if xin else f64(x)
        _, m_ref, r_ref = oracle.layernorm_fwd(xin_all, P(gam), np.zeros(H), eps)
        rdx, rdg, rdb = oracle.layernorm_bwd(f64(t[dy]), xin_all, m_ref, r_ref, P(gam))
        rdx = rdx + (f64(t[dres]) if dres else f64(dout))
        gerrs[f"{ln}_bwd.dx"] = max_rel(f64(t[dxk])[rows], rdx[rows])
        gerrs[f"{ln}_bwd.dgamma"] = max_rel(f64(t["d" + gam]), rdg)
        gerrs[f"{ln}_bwd.dbeta"] = max_rel(f64(t["d" + gam[:-1] + "b"]), rdb)
    # weight gradients on sampled output rows (all columns), bias grads whole
    for dwk, dbk, dyk, xk in (("dw_2", "db_2", None, "g"), ("dw_1", "db_1", "du", "y2"),
                              ("dw_o", "db_o", "dh", "o"), ("dw_qkv", "db_qkv", "dqkv", "y1")):
        dY = t[dyk] if dyk else gd
        N = dY.shape[1]
        nrows = _sample_rows(N, 8, 11)
        ridx = torch.as_tensor(nrows, device="cuda")
        rdW, rdb = oracle.linear_bwd_weight(f64(dY[:, ridx]), f64(t[xk]))
        gerrs[dwk] = max_rel(f64(t[dwk][ridx]), rdW)
        gerrs[dbk] = max_rel(f64(t[dbk]), oracle.linear_bwd_weight(f64(dY), np.zeros((M, 8)))[1])
    for k, e in gerrs.items():
        assert e < TOL_GRAD, (k, e)
    print(f"[parity] {name} max step act err {max(errs.values()):.3e}, grad err {max(gerrs.values()):.3e}")
