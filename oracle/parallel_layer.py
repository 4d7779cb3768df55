"""Float64 CPU oracle of the ViT-22B-style encoder block (test infrastructure only).

Only the tests, the smoke check and the CPU-baseline leg of the benchmark
import this module; the product library never does.

The paper trains ViT-22B as its largest encoder (Appendix A, ViT table) but
does not write the layer out.  The architecture of the cited ViT-22B work
differs from the sequential pre-LN block in three ways, and this block takes
them as its reading:
  - parallel branches: attention and MLP both read one LayerNorm of the
    input, and both outputs are added to the residual,
        y   = LN(x)
        out = x + Attn(y) Wo^T + bo + GELU(y W1^T + b1) W2^T + b2
  - QK normalisation: queries and keys are layer-normalised over head_dim,
    per token and head, before the dot product, with affine parameters of
    length head_dim shared by all heads (qn_g, qn_b for queries, kn_g, kn_b
    for keys); values are not normalised;
  - no bias on the QKV projection.
LayerNorms keep their bias (read from the cited ViT-22B architecture); every
other convention (scale 1/sqrt(d), exact-erf GELU, [3][heads][d] packing,
epsilon = ln_eps for all LayerNorms) is that of the sequential block.
"""

import numpy as np

from .encoder_layer import (attention_bwd, attention_fwd, gelu, gelu_grad, layernorm_bwd, layernorm_fwd,
                            linear_bwd_data, linear_bwd_weight, linear_fwd)

__all__ = ["PARALLEL_PARAM_NAMES", "parallel_param_shapes", "qk_norm_fwd", "qk_norm_bwd",
           "parallel_layer_fwd", "parallel_layer_bwd"]

PARALLEL_PARAM_NAMES = ("ln_g", "ln_b", "w_qkv", "qn_g", "qn_b", "kn_g", "kn_b",
                        "w_o", "b_o", "w_1", "b_1", "w_2", "b_2")


def parallel_param_shapes(hidden, heads, head_dim, mlp):
    A = heads * head_dim
    return {"ln_g": (hidden,), "ln_b": (hidden,), "w_qkv": (3 * A, hidden),
            "qn_g": (head_dim,), "qn_b": (head_dim,), "kn_g": (head_dim,), "kn_b": (head_dim,),
            "w_o": (hidden, A), "b_o": (hidden,), "w_1": (mlp, hidden), "b_1": (mlp,),
            "w_2": (hidden, mlp), "b_2": (hidden,)}


def qk_norm_fwd(qkv, heads, d, qg, qb, kg, kb, eps):
    """LayerNorm of every (token, head) query and key vector over head_dim.

    Returns (qkvn, stats): qkvn has the qkv packing with q and k normalised
    and v unchanged; stats holds qmean, qrstd, kmean, krstd of shape [M, heads].
    """
    M, A = qkv.shape[0], heads * d
    q = qkv[:, :A].reshape(M * heads, d)
    k = qkv[:, A:2 * A].reshape(M * heads, d)
    qn, qmean, qrstd = layernorm_fwd(q, qg, qb, eps)
    kn, kmean, krstd = layernorm_fwd(k, kg, kb, eps)
    qkvn = np.concatenate([qn.reshape(M, A), kn.reshape(M, A), qkv[:, 2 * A:]], axis=1)
    stats = dict(qmean=qmean.reshape(M, heads), qrstd=qrstd.reshape(M, heads),
                 kmean=kmean.reshape(M, heads), krstd=krstd.reshape(M, heads))
    return qkvn, stats


def qk_norm_bwd(dqkvn, qkv, stats, heads, d, qg, kg):
    """Gradient of qk_norm_fwd: returns (dqkv, grads of qn_g, qn_b, kn_g, kn_b)."""
    M, A = qkv.shape[0], heads * d
    dq, dqg, dqb = layernorm_bwd(dqkvn[:, :A].reshape(M * heads, d), qkv[:, :A].reshape(M * heads, d),
                                 stats["qmean"].reshape(-1), stats["qrstd"].reshape(-1), qg)
    dk, dkg, dkb = layernorm_bwd(dqkvn[:, A:2 * A].reshape(M * heads, d), qkv[:, A:2 * A].reshape(M * heads, d),
                                 stats["kmean"].reshape(-1), stats["krstd"].reshape(-1), kg)
    dqkv = np.concatenate([dq.reshape(M, A), dk.reshape(M, A), dqkvn[:, 2 * A:]], axis=1)
    return dqkv, {"qn_g": dqg, "qn_b": dqb, "kn_g": dkg, "kn_b": dkb}


def parallel_layer_fwd(cfg, p, x):
    """Forward of the parallel block.  Returns (out, saved) with saved holding
    y, mean, rstd, qkv, qkvn, the QK-norm statistics, o, lse, h, u, g, where
    h = x + o Wo^T + bo is the residual plus the attention branch."""
    B, S = cfg["batch"], cfg["seq"]
    nh, d, eps = cfg["heads"], cfg["head_dim"], cfg["ln_eps"]
    y, mean, rstd = layernorm_fwd(x, p["ln_g"], p["ln_b"], eps)
    qkv = linear_fwd(y, p["w_qkv"])
    qkvn, st = qk_norm_fwd(qkv, nh, d, p["qn_g"], p["qn_b"], p["kn_g"], p["kn_b"], eps)
    o, lse = attention_fwd(qkvn, B, S, nh, d)
    h = linear_fwd(o, p["w_o"], p["b_o"], resid=x)
    u = linear_fwd(y, p["w_1"], p["b_1"])
    g = gelu(u)
    out = linear_fwd(g, p["w_2"], p["b_2"], resid=h)
    saved = dict(y=y, mean=mean, rstd=rstd, qkv=qkv, qkvn=qkvn, o=o, lse=lse, h=h, u=u, g=g, **st)
    return out, saved


def parallel_layer_bwd(cfg, p, x, saved, dout):
    """Backward of parallel_layer_fwd.  Returns (dx, grads, inter) with inter
    holding du, dy_mlp, do, dqkvn, dqkv, dy_attn and dy = dy_attn + dy_mlp."""
    B, S = cfg["batch"], cfg["seq"]
    nh, d = cfg["heads"], cfg["head_dim"]
    s = saved
    gr = {}
    # MLP branch: out += GELU(y W1^T + b1) W2^T + b2
    gr["w_2"], gr["b_2"] = linear_bwd_weight(dout, s["g"])
    du = linear_bwd_data(dout, p["w_2"]) * gelu_grad(s["u"])
    gr["w_1"], gr["b_1"] = linear_bwd_weight(du, s["y"])
    dy_mlp = linear_bwd_data(du, p["w_1"])
    # attention branch: out += o Wo^T + bo, o = Attn(QKnorm(y Wqkv^T))
    gr["w_o"], gr["b_o"] = linear_bwd_weight(dout, s["o"])
    do = linear_bwd_data(dout, p["w_o"])
    dqkvn = attention_bwd(s["qkvn"], do, B, S, nh, d)
    dqkv, gq = qk_norm_bwd(dqkvn, s["qkv"], s, nh, d, p["qn_g"], p["kn_g"])
    gr.update(gq)
    gr["w_qkv"], _ = linear_bwd_weight(dqkv, s["y"])
    dy_attn = linear_bwd_data(dqkv, p["w_qkv"])
    # both branches read y = LN(x); x also feeds the residual
    dy = dy_attn + dy_mlp
    dx_ln, gr["ln_g"], gr["ln_b"] = layernorm_bwd(dy, x, s["mean"], s["rstd"], p["ln_g"])
    dx = dout + dx_ln
    inter = dict(du=du, dy_mlp=dy_mlp, do=do, dqkvn=dqkvn, dqkv=dqkv, dy_attn=dy_attn, dy=dy)
    return dx, gr, inter
