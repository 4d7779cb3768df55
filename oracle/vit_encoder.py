"""Float64 CPU oracle of a whole ViT encoder on one micro-batch (test
infrastructure only): patch embedding, a stack of encoder layers and a final
LayerNorm.

Only the tests, the smoke check and the CPU-baseline leg of the benchmark
import this module; the product library never does.

The paper's encoders are ViTs (Appendix A, ViT table: width, depth, MLP
width, heads); an image of side `img` is cut into non-overlapping p x p
patches (the sequence lengths of the workloads follow: 224/16 = 14, 14^2 + 1
class token = 197; 224/14 = 16, 16^2 = 256 patches, +1 with a class token).
Reading: the patch embedding is the usual stride-p convolution written as a
matrix product -- patch vector order (channel, row, column), weight
[hidden, C*p*p] -- plus a bias; an optional class token is prepended and a
learned position embedding [seq, hidden] is added; layers are the
sequential pre-LN blocks of encoder_layer; a final LayerNorm follows.
"""

import numpy as np

from .encoder_layer import layer_bwd, layer_fwd, layernorm_bwd, layernorm_fwd, linear_bwd_weight, linear_fwd

__all__ = ["patchify", "patch_embed_fwd", "patch_embed_bwd", "encoder_fwd", "encoder_bwd"]


def patchify(images, p):
    """[B, C, Hi, Wi] -> [B*N, C*p*p]: patches in row-major grid order, each
    flattened in (channel, row, column) order."""
    B, C, Hi, Wi = images.shape
    gh, gw = Hi // p, Wi // p
    t = images.reshape(B, C, gh, p, gw, p).transpose(0, 2, 4, 1, 3, 5)
    return t.reshape(B * gh * gw, C * p * p)


def patch_embed_fwd(images, p, w_pe, b_pe, cls, pos):
    """x0 [B*S, H]: patch tokens (patches w_pe^T + b_pe), the class token
    first when cls is not None, plus pos [S, H] for every sequence."""
    B = images.shape[0]
    patches = patchify(images, p)
    tok = linear_fwd(patches, w_pe, b_pe)
    N, H = tok.shape[0] // B, tok.shape[1]
    tok = tok.reshape(B, N, H)
    if cls is not None:
        tok = np.concatenate([np.broadcast_to(cls, (B, 1, H)), tok], axis=1)
    x0 = tok + pos[None]
    return x0.reshape(-1, H), patches


def patch_embed_bwd(dx0, patches, B, has_cls):
    """Gradients of patch_embed_fwd's parameters: (dw_pe, db_pe, dcls or None, dpos)."""
    H = dx0.shape[1]
    d = dx0.reshape(B, -1, H)
    dpos = d.sum(axis=0)
    dcls = d[:, 0].sum(axis=0) if has_cls else None
    dtok = (d[:, 1:] if has_cls else d).reshape(-1, H)
    dw, db = linear_bwd_weight(dtok, patches)
    return dw, db, dcls, dpos


def encoder_fwd(cfg, pe, layers, ln_f, images):
    """Whole encoder.  pe: dict w_pe, b_pe, cls (or None), pos, patch; layers:
    list of per-layer parameter dicts; ln_f: (gamma, beta).  Returns (out, saved)."""
    x, patches = patch_embed_fwd(images, pe["patch"], pe["w_pe"], pe["b_pe"], pe["cls"], pe["pos"])
    xs, saves = [x], []
    for p in layers:
        x, s = layer_fwd(cfg, p, x)
        xs.append(x)
        saves.append(s)
    out, mean, rstd = layernorm_fwd(x, ln_f[0], ln_f[1], cfg["ln_eps"])
    return out, dict(patches=patches, xs=xs, layers=saves, mean=mean, rstd=rstd)


def encoder_bwd(cfg, pe, layers, ln_f, images, saved, dout):
    """Returns (grads_pe, grads_layers, (dln_f_g, dln_f_b)); the images get no gradient."""
    dx, dg, dbeta = layernorm_bwd(dout, saved["xs"][-1], saved["mean"], saved["rstd"], ln_f[0])
    glayers = [None] * len(layers)
    for i in range(len(layers) - 1, -1, -1):
        dx, glayers[i], _ = layer_bwd(cfg, layers[i], saved["xs"][i], saved["layers"][i], dx)
    dw, db, dcls, dpos = patch_embed_bwd(dx, saved["patches"], images.shape[0], pe["cls"] is not None)
    return dict(w_pe=dw, b_pe=db, cls=dcls, pos=dpos), glayers, (dg, dbeta)
