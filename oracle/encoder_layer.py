"""CPU oracle for one ViT encoder layer, forward and backward, in float64.

TEST INFRASTRUCTURE ONLY.  Nothing in the product library imports, links or
calls this module; only the test suite, the smoke check and the CPU-baseline
leg of the benchmark use it.  It shares no code with the HIP path.

What is computed.  The paper (Optimus, arXiv 2408.03505) splits the encoder
layer's forward and backward into a chain of kernels so that the pieces fit
sub-millisecond LLM bubbles (abstract; §1 third challenge; §3.1 design
decision 3; §4.2, the ScheduleKernels step).  The decomposition only changes
*when* work runs, never *what* is computed, so the oracle is the plain
definition of one encoder layer and its exact gradient.  The paper names the
encoders (ViT-3B/5B/10B/22B: width, MLP dimension, heads, head dimension;
Appendix A, table of ViT configurations) but does not write the block out;
the reading used here is the standard pre-LayerNorm ViT block:

    h   = x + Attn(LN1(x)) Wo^T + bo
    out = h + GELU(LN2(h) W1^T + b1) W2^T + b2

with one fused QKV projection whose output columns are packed
[3][heads][head_dim], bidirectional softmax attention scaled by
1/sqrt(head_dim), no mask, no dropout, LayerNorm with biased variance and
eps inside the square root, and the exact (erf) GELU.  The parameter counts
this gives reproduce the ViT table of Appendix A (tests/golden).  Parameter
gradients are full sums over all token rows, returned in float64; the GPU
path keeps them in fp32 because the paper's training keeps parameters in
bf16 and their gradients in fp32 (§4.5, memory analysis, k = 6 bytes per
parameter).

Every array is a numpy float64 array, row-major.  Token rows are M = B*S,
ordered sequence-major (row r = b*S + s).  Weights are stored [out, in].

Each function is written from its mathematical definition with numpy's
matmul and scipy's erf as the only library primitives; nothing is blocked,
fused or reordered.
"""

import math

import numpy as np
import scipy.special

__all__ = [
    "layernorm_fwd",
    "layernorm_bwd",
    "linear_fwd",
    "linear_bwd_data",
    "linear_bwd_weight",
    "gelu",
    "gelu_grad",
    "attention_fwd",
    "attention_bwd",
    "layer_fwd",
    "layer_bwd",
    "PARAM_NAMES",
    "param_shapes",
    "layer_flops",
]

# Parameter order of the layer (also the order the input generator draws them).
PARAM_NAMES = (
    "ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
    "ln2_g", "ln2_b", "w_1", "b_1", "w_2", "b_2",
)


def param_shapes(hidden, heads, head_dim, mlp):
    """Shapes of the twelve layer parameters, weights stored [out, in].

    A = heads*head_dim may differ from hidden (a tensor-parallel shard keeps
    the full LayerNorm width but only some heads and part of the MLP).
    """
    A = heads * head_dim
    return {
        "ln1_g": (hidden,), "ln1_b": (hidden,),
        "w_qkv": (3 * A, hidden), "b_qkv": (3 * A,),
        "w_o": (hidden, A), "b_o": (hidden,),
        "ln2_g": (hidden,), "ln2_b": (hidden,),
        "w_1": (mlp, hidden), "b_1": (mlp,),
        "w_2": (hidden, mlp), "b_2": (hidden,),
    }


# ---------------------------------------------------------------- LayerNorm

def layernorm_fwd(x, gamma, beta, eps):
    """LayerNorm over the last axis.

    mean_r = (1/C) sum_c x_rc;  var_r = (1/C) sum_c (x_rc - mean_r)^2
    (biased, two-pass);  rstd_r = 1/sqrt(var_r + eps);
    xhat = (x - mean) * rstd;  y = xhat * gamma + beta.
    Returns (y, mean, rstd); mean and rstd have one entry per row.
    """
    mean = x.mean(axis=-1)
    centered = x - mean[..., None]
    var = (centered * centered).mean(axis=-1)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = centered * rstd[..., None]
    return xhat * gamma + beta, mean, rstd


def layernorm_bwd(dy, x, mean, rstd, gamma):
    """Exact gradient of layernorm_fwd with respect to x, gamma and beta.

    With xhat = (x - mean) * rstd and ghat = dy * gamma, differentiating
    y = xhat*gamma + beta through mean and rstd gives, per row,
        dx = rstd * (ghat - mean_c(ghat) - xhat * mean_c(ghat * xhat)),
    and the affine gradients are column sums over all rows:
        dgamma = sum_r dy * xhat,   dbeta = sum_r dy.
    Returns (dx, dgamma, dbeta).
    """
    xhat = (x - mean[:, None]) * rstd[:, None]
    ghat = dy * gamma
    c1 = ghat.mean(axis=1, keepdims=True)
    c2 = (ghat * xhat).mean(axis=1, keepdims=True)
    dx = rstd[:, None] * (ghat - c1 - xhat * c2)
    return dx, (dy * xhat).sum(axis=0), dy.sum(axis=0)


# ---------------------------------------------------------------- Linear

def linear_fwd(X, W, b=None, resid=None):
    """Y[m, n] = sum_k X[m, k] * W[n, k] + b[n] (+ resid[m, n])."""
    Y = X @ W.T
    if b is not None:
        Y = Y + b
    if resid is not None:
        Y = Y + resid
    return Y


def linear_bwd_data(dY, W):
    """Input gradient of linear_fwd: dX[m, k] = sum_n dY[m, n] * W[n, k]."""
    return dY @ W


def linear_bwd_weight(dY, X):
    """Parameter gradients of linear_fwd, summed over all rows m:
    dW[n, k] = sum_m dY[m, n] * X[m, k];  db[n] = sum_m dY[m, n]."""
    return dY.T @ X, dY.sum(axis=0)


# ---------------------------------------------------------------- GELU

# The error function, element-wise in float64 (scipy's vectorised erf; agrees
# with math.erf to within 5e-16 relative).
_erf = scipy.special.erf


def gelu(u):
    """Exact GELU: u * Phi(u), Phi the standard normal CDF = (1 + erf(u/sqrt 2))/2."""
    return 0.5 * u * (1.0 + _erf(u / math.sqrt(2.0)))


def gelu_grad(u):
    """d GELU / du = Phi(u) + u * phi(u), phi(u) = exp(-u^2/2)/sqrt(2 pi)."""
    Phi = 0.5 * (1.0 + _erf(u / math.sqrt(2.0)))
    phi = np.exp(-0.5 * u * u) / math.sqrt(2.0 * math.pi)
    return Phi + u * phi


# ---------------------------------------------------------------- Attention

def _split_heads(qkv, B, S, heads, d):
    """qkv[M, 3A] with columns [3][heads][d] -> q, k, v each [B, heads, S, d]."""
    t = qkv.reshape(B, S, 3, heads, d)
    return (t[:, :, 0].transpose(0, 2, 1, 3),
            t[:, :, 1].transpose(0, 2, 1, 3),
            t[:, :, 2].transpose(0, 2, 1, 3))


def _merge_heads(o, B, S, heads, d):
    """[B, heads, S, d] -> [M, heads*d] with columns [heads][d]."""
    return o.transpose(0, 2, 1, 3).reshape(B * S, heads * d)


def _softmax_rows(s):
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


def attention_fwd(qkv, B, S, heads, d):
    """Bidirectional multi-head softmax attention of every sequence.

    For each sequence b and head h: s_ij = q_i . k_j / sqrt(d);
    P = softmax over j; O_i = sum_j P_ij v_j.  Also returns the per-row
    log-sum-exp of the scaled logits, lse_i = log sum_j exp(s_ij), shape
    [B, heads, S] (the softmax normaliser the backward pass can reuse).
    Returns (O [M, heads*d], lse).
    """
    q, k, v = _split_heads(qkv, B, S, heads, d)
    s = (q @ k.transpose(0, 1, 3, 2)) / math.sqrt(d)
    m = s.max(axis=-1)
    lse = m + np.log(np.exp(s - m[..., None]).sum(axis=-1))
    P = _softmax_rows(s)
    return _merge_heads(P @ v, B, S, heads, d), lse


def attention_bwd(qkv, dO, B, S, heads, d):
    """Exact gradient of attention_fwd with respect to qkv.

    P is recomputed from its definition.  dV = P^T dO; dP = dO V^T; the
    softmax Jacobian gives dS_ij = P_ij (dP_ij - sum_k P_ik dP_ik); the
    1/sqrt(d) scale then gives dQ = dS K / sqrt(d), dK = dS^T Q / sqrt(d).
    Returns dqkv [M, 3A] packed like qkv.
    """
    q, k, v = _split_heads(qkv, B, S, heads, d)
    do = dO.reshape(B, S, heads, d).transpose(0, 2, 1, 3)
    scale = 1.0 / math.sqrt(d)
    P = _softmax_rows((q @ k.transpose(0, 1, 3, 2)) * scale)
    dv = P.transpose(0, 1, 3, 2) @ do
    dP = do @ v.transpose(0, 1, 3, 2)
    dS = P * (dP - (P * dP).sum(axis=-1, keepdims=True))
    dq = (dS @ k) * scale
    dk = (dS.transpose(0, 1, 3, 2) @ q) * scale
    out = np.stack([_merge_heads(t, B, S, heads, d) for t in (dq, dk, dv)], axis=1)
    return out.reshape(B * S, 3 * heads * d)


# ---------------------------------------------------------------- Layer

def layer_fwd(cfg, p, x):
    """Forward of one pre-LN encoder layer on one micro-batch.

    cfg: dict with batch, seq, hidden, heads, head_dim, mlp, ln_eps.
    p:   dict of the twelve parameters (PARAM_NAMES), float64.
    x:   [M, hidden] input tokens, M = batch*seq.
    Returns (out, saved) where saved holds every intermediate of the chain:
    y1, mean1, rstd1, qkv, o, lse, h, y2, mean2, rstd2, u, g.
    """
    B, S = cfg["batch"], cfg["seq"]
    nh, d, eps = cfg["heads"], cfg["head_dim"], cfg["ln_eps"]
    y1, mean1, rstd1 = layernorm_fwd(x, p["ln1_g"], p["ln1_b"], eps)
    qkv = linear_fwd(y1, p["w_qkv"], p["b_qkv"])
    o, lse = attention_fwd(qkv, B, S, nh, d)
    h = linear_fwd(o, p["w_o"], p["b_o"], resid=x)
    y2, mean2, rstd2 = layernorm_fwd(h, p["ln2_g"], p["ln2_b"], eps)
    u = linear_fwd(y2, p["w_1"], p["b_1"])
    g = gelu(u)
    out = linear_fwd(g, p["w_2"], p["b_2"], resid=h)
    saved = dict(y1=y1, mean1=mean1, rstd1=rstd1, qkv=qkv, o=o, lse=lse, h=h,
                 y2=y2, mean2=mean2, rstd2=rstd2, u=u, g=g)
    return out, saved


def layer_bwd(cfg, p, x, saved, dout):
    """Backward of layer_fwd given the upstream gradient dout [M, hidden].

    Returns (dx, grads, inter): grads[name] is the gradient of parameter
    name (PARAM_NAMES), inter holds the intermediate gradients du, dy2, dh,
    do, dqkv and dy1 of the chain.
    """
    B, S = cfg["batch"], cfg["seq"]
    nh, d = cfg["heads"], cfg["head_dim"]
    s = saved
    gr = {}
    # out = h + g W2^T + b2
    gr["w_2"], gr["b_2"] = linear_bwd_weight(dout, s["g"])
    dg = linear_bwd_data(dout, p["w_2"])
    # g = GELU(u), u = y2 W1^T + b1
    du = dg * gelu_grad(s["u"])
    gr["w_1"], gr["b_1"] = linear_bwd_weight(du, s["y2"])
    dy2 = linear_bwd_data(du, p["w_1"])
    # y2 = LN2(h); h also feeds the residual into out
    dh_ln, gr["ln2_g"], gr["ln2_b"] = layernorm_bwd(dy2, s["h"], s["mean2"], s["rstd2"], p["ln2_g"])
    dh = dout + dh_ln
    # h = x + o Wo^T + bo
    gr["w_o"], gr["b_o"] = linear_bwd_weight(dh, s["o"])
    do = linear_bwd_data(dh, p["w_o"])
    dqkv = attention_bwd(s["qkv"], do, B, S, nh, d)
    # qkv = y1 Wqkv^T + bqkv
    gr["w_qkv"], gr["b_qkv"] = linear_bwd_weight(dqkv, s["y1"])
    dy1 = linear_bwd_data(dqkv, p["w_qkv"])
    # y1 = LN1(x); x also feeds the residual into h
    dx_ln, gr["ln1_g"], gr["ln1_b"] = layernorm_bwd(dy1, x, s["mean1"], s["rstd1"], p["ln1_g"])
    dx = dh + dx_ln
    inter = dict(du=du, dy2=dy2, dh=dh, do=do, dqkv=dqkv, dy1=dy1)
    return dx, gr, inter


def layer_flops(cfg):
    """Algorithmic flops of one forward pass (multiply-add = 2 flops):
    four projections 2*M*(3*H*A + A*H + 2*H*F) plus attention 4*B*heads*S^2*d.
    The backward pass is twice this (input and parameter gradients of every
    product; four products in attention), so forward+backward is 3x."""
    B, S, H = cfg["batch"], cfg["seq"], cfg["hidden"]
    A, F = cfg["heads"] * cfg["head_dim"], cfg["mlp"]
    M = B * S
    return 2 * M * (3 * H * A + A * H + 2 * H * F) + 4 * B * cfg["heads"] * S * S * cfg["head_dim"]
