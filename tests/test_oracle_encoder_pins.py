"""Pins of the whole-encoder oracle (oracle.vit_encoder): the patch embedding
against torch's stride-p Conv2d, the whole encoder (patch embedding, layers,
final LayerNorm; with and without a class token) against fp64 torch autograd
of an independent composition, finite differences of the embedding
parameters, and planted mistakes."""

import numpy as np
import torch
import torch.nn.functional as F

import oracle
from oracle import vit_encoder as V
from test_oracle_pins import _params, _torch_layer


def _rng(seed):
    return np.random.default_rng(seed)


def _setup(cfg, layers, img, p, C, has_cls, seed):
    rng = _rng(seed)
    B, H = cfg["batch"], cfg["hidden"]
    N = (img // p) ** 2
    S = N + (1 if has_cls else 0)
    assert S == cfg["seq"]
    images = rng.normal(size=(B, C, img, img))
    pe = dict(patch=p, w_pe=rng.normal(size=(H, C * p * p)) * 0.2, b_pe=rng.normal(size=H) * 0.1,
              cls=rng.normal(size=H) if has_cls else None, pos=rng.normal(size=(S, H)) * 0.1)
    lp = [_params(cfg, rng, scale=0.1) for _ in range(layers)]
    ln_f = (1.0 + 0.1 * rng.normal(size=H), 0.1 * rng.normal(size=H))
    dout = rng.normal(size=(B * S, H))
    return images, pe, lp, ln_f, dout


def _torch_encoder(cfg, images, pe, lp, ln_f):
    B, H = cfg["batch"], cfg["hidden"]
    p = pe["patch"]
    C = images.shape[1]
    tok = F.conv2d(images, pe["w_pe"].reshape(H, C, p, p), pe["b_pe"], stride=p)  # [B, H, gh, gw]
    tok = tok.flatten(2).transpose(1, 2)                                          # [B, N, H]
    if pe["cls"] is not None:
        tok = torch.cat([pe["cls"].expand(B, 1, H), tok], dim=1)
    x = (tok + pe["pos"]).reshape(-1, H)
    for q in lp:
        x = _torch_layer(cfg, q, x)
    return F.layer_norm(x, (H,), ln_f[0], ln_f[1], cfg["ln_eps"])


def encoder_vs_torch_error(has_cls, seed=31):
    S = 16 + (1 if has_cls else 0)
    cfg = dict(batch=2, seq=S, hidden=32, heads=2, head_dim=16, mlp=64, ln_eps=1e-6)
    images, pe, lp, ln_f, dout = _setup(cfg, 2, 8, 2, 3, has_cls, seed)
    out, saved = oracle.vit_encoder.encoder_fwd(cfg, pe, lp, ln_f, images)
    gpe, gl, gln = oracle.vit_encoder.encoder_bwd(cfg, pe, lp, ln_f, images, saved, dout)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).requires_grad_()  # noqa: E731
    tpe = {k: (T(v) if isinstance(v, np.ndarray) else v) for k, v in pe.items()}
    tlp = [{k: T(v) for k, v in q.items()} for q in lp]
    tln = (T(ln_f[0]), T(ln_f[1]))
    tout = _torch_encoder(cfg, torch.from_numpy(images), tpe, tlp, tln)
    tout.backward(torch.from_numpy(dout))
    rel = lambda a, b: np.abs(a - b).max() / max(np.abs(b).max(), 1e-300)  # noqa: E731
    errs = [rel(out, tout.detach().numpy()), rel(gln[0], tln[0].grad.numpy()), rel(gln[1], tln[1].grad.numpy())]
    for k in ("w_pe", "b_pe", "pos") + (("cls",) if has_cls else ()):
        errs.append(rel(gpe[k], tpe[k].grad.numpy()))
    for q, tq in zip(gl, tlp):
        errs += [rel(q[n], tq[n].grad.numpy()) for n in oracle.PARAM_NAMES]
    return max(errs)


def test_patch_embedding_is_a_strided_convolution():
    rng = _rng(30)
    B, C, img, p, H = 2, 3, 12, 4, 10
    images = rng.normal(size=(B, C, img, img))
    w, b = rng.normal(size=(H, C * p * p)), rng.normal(size=H)
    pos = rng.normal(size=((img // p) ** 2, H))
    x0, _ = V.patch_embed_fwd(images, p, w, b, None, pos)
    ref = F.conv2d(torch.from_numpy(images), torch.from_numpy(w).reshape(H, C, p, p), torch.from_numpy(b), stride=p)
    ref = (ref.flatten(2).transpose(1, 2) + torch.from_numpy(pos)).reshape(-1, H).numpy()
    assert np.abs(x0 - ref).max() < 1e-12


def test_encoder_matches_torch_with_class_token():
    assert encoder_vs_torch_error(True) < 1e-10


def test_encoder_matches_torch_without_class_token():
    assert encoder_vs_torch_error(False) < 1e-10


def test_embedding_gradients_finite_difference():
    cfg = dict(batch=2, seq=5, hidden=8, heads=2, head_dim=4, mlp=16, ln_eps=1e-6)
    images, pe, lp, ln_f, dout = _setup(cfg, 1, 4, 2, 2, True, 32)
    out, saved = V.encoder_fwd(cfg, pe, lp, ln_f, images)
    gpe, _, gln = V.encoder_bwd(cfg, pe, lp, ln_f, images, saved, dout)
    loss = lambda: float((V.encoder_fwd(cfg, pe, lp, ln_f, images)[0] * dout).sum())  # noqa: E731
    h, worst = 1e-5, 0.0
    for arr, an in ((pe["w_pe"], gpe["w_pe"]), (pe["b_pe"], gpe["b_pe"]), (pe["cls"], gpe["cls"]),
                    (pe["pos"], gpe["pos"]), (ln_f[0], gln[0]), (ln_f[1], gln[1])):
        flat = arr.reshape(-1)
        fd = np.empty(flat.size)
        for i in range(flat.size):
            keep = flat[i]
            flat[i] = keep + h
            lp_ = loss()
            flat[i] = keep - h
            lm = loss()
            flat[i] = keep
            fd[i] = (lp_ - lm) / (2 * h)
        worst = max(worst, np.abs(fd - an.reshape(-1)).max() / max(1.0, np.abs(an).max()))
    assert worst < 1e-6


# ---- planted mistakes

def test_mutant_patch_flatten_order_is_caught(monkeypatch):
    def bad(images, p):
        B, C, Hi, Wi = images.shape
        t = images.reshape(B, C, Hi // p, p, Wi // p, p).transpose(0, 2, 4, 3, 5, 1)  # (row, col, channel)
        return t.reshape(B * (Hi // p) * (Wi // p), C * p * p)
    monkeypatch.setattr(V, "patchify", bad)
    assert encoder_vs_torch_error(True) > 1e-3


def test_mutant_position_embedding_misaligned_is_caught(monkeypatch):
    real = V.patch_embed_fwd

    def bad(images, p, w_pe, b_pe, cls, pos):
        x0, patches = real(images, p, w_pe, b_pe, cls, np.roll(pos, 1, axis=0))
        return x0, patches
    monkeypatch.setattr(V, "patch_embed_fwd", bad)
    assert encoder_vs_torch_error(True) > 1e-3


def test_mutant_class_token_gradient_is_caught(monkeypatch):
    real = V.patch_embed_bwd

    def bad(dx0, patches, B, has_cls):
        dw, db, dcls, dpos = real(dx0, patches, B, has_cls)
        return dw, db, (dx0.reshape(B, -1, dx0.shape[1])[0, 0] if has_cls else None), dpos
    monkeypatch.setattr(V, "patch_embed_bwd", bad)
    assert encoder_vs_torch_error(True) > 1e-3
