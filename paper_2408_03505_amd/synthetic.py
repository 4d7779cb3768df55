"""Seeded synthetic inputs for one encoder layer.

This module only draws random numbers: it holds none of the layer's
arithmetic.  The same draws, rounded once to bfloat16, feed both the HIP
path and the float64 oracle, so the two see bit-identical inputs.

Recipe (one torch CPU generator, seeded, drawn in this fixed order):
  x     ~ N(0, 1)                     [M, hidden]
  ln*_g = 1 + N(0, std)               [hidden]
  ln*_b, every weight and bias ~ N(0, std)   (std = 0.02)
  dout  ~ N(0, 1)                     [M, hidden]
Parameters are drawn in the order ln1_g, ln1_b, w_qkv, b_qkv, w_o, b_o,
ln2_g, ln2_b, w_1, b_1, w_2, b_2 (weights stored [out, in]).  Everything is
drawn in float32 and rounded to bfloat16 (round to nearest even) once.
"""

import torch

PARAM_ORDER = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
               "ln2_g", "ln2_b", "w_1", "b_1", "w_2", "b_2")


def layer_param_shapes(hidden, heads, head_dim, mlp):
    a = heads * head_dim
    return {
        "ln1_g": (hidden,), "ln1_b": (hidden,),
        "w_qkv": (3 * a, hidden), "b_qkv": (3 * a,),
        "w_o": (hidden, a), "b_o": (hidden,),
        "ln2_g": (hidden,), "ln2_b": (hidden,),
        "w_1": (mlp, hidden), "b_1": (mlp,),
        "w_2": (hidden, mlp), "b_2": (hidden,),
    }


def layer_inputs(cfg, seed=0, std=0.02, with_dout=True):
    """Return (x, params, dout) as bfloat16 CPU tensors for config cfg
    (a dict with batch, seq, hidden, heads, head_dim, mlp)."""
    g = torch.Generator().manual_seed(seed)
    M = cfg["batch"] * cfg["seq"]
    H = cfg["hidden"]

    def normal(shape, s=1.0, mean=0.0):
        t = torch.randn(shape, generator=g, dtype=torch.float32)
        if s != 1.0:
            t.mul_(s)
        if mean != 0.0:
            t.add_(mean)
        return t.to(torch.bfloat16)

    x = normal((M, H))
    shapes = layer_param_shapes(H, cfg["heads"], cfg["head_dim"], cfg["mlp"])
    params = {}
    for name in PARAM_ORDER:
        mean = 1.0 if name in ("ln1_g", "ln2_g") else 0.0
        params[name] = normal(shapes[name], std, mean)
    dout = normal((M, H)) if with_dout else None
    return x, params, dout


PPARAM_ORDER = ("ln_g", "ln_b", "w_qkv", "qn_g", "qn_b", "kn_g", "kn_b", "w_o", "b_o", "w_1", "b_1", "w_2", "b_2")


def parallel_param_shapes(hidden, heads, head_dim, mlp):
    A = heads * head_dim
    return {"ln_g": (hidden,), "ln_b": (hidden,), "w_qkv": (3 * A, hidden), "qn_g": (head_dim,),
            "qn_b": (head_dim,), "kn_g": (head_dim,), "kn_b": (head_dim,), "w_o": (hidden, A), "b_o": (hidden,),
            "w_1": (mlp, hidden), "b_1": (mlp,), "w_2": (hidden, mlp), "b_2": (hidden,)}


def parallel_block_inputs(cfg, seed=0, std=0.02):
    """(x, params, dout) for the ViT-22B-style block, bfloat16 CPU tensors,
    drawn like layer_inputs: x, then the parameters in PPARAM_ORDER (the
    three LayerNorm scales 1 + N(0, std^2), everything else N(0, std^2)),
    then dout."""
    g = torch.Generator().manual_seed(seed)
    M, H = cfg["batch"] * cfg["seq"], cfg["hidden"]

    def normal(shape, s=1.0, mean=0.0):
        t = torch.randn(shape, generator=g, dtype=torch.float32)
        return (t * s + mean).to(torch.bfloat16)

    x = normal((M, H))
    shapes = parallel_param_shapes(H, cfg["heads"], cfg["head_dim"], cfg["mlp"])
    params = {n: normal(shapes[n], std, 1.0 if n in ("ln_g", "qn_g", "kn_g") else 0.0) for n in PPARAM_ORDER}
    dout = normal((M, H))
    return x, params, dout


def random_bf16(shape, seed, scale=1.0):
    """A seeded N(0, scale^2) tensor rounded to bfloat16 (CPU)."""
    g = torch.Generator().manual_seed(seed)
    t = torch.randn(shape, generator=g, dtype=torch.float32)
    if scale != 1.0:
        t.mul_(scale)
    return t.to(torch.bfloat16)


def random_int_bf16(shape, seed, lo=-2, hi=2):
    """A seeded tensor of small integers in [lo, hi], stored as bfloat16
    (exactly representable), for exact-arithmetic layout tests."""
    g = torch.Generator().manual_seed(seed)
    return torch.randint(lo, hi + 1, shape, generator=g, dtype=torch.int32).to(torch.bfloat16)


# The five workloads: a ViT-Tiny, ViT-Base and ViT-Huge layer, one GPU's
# 1/8 tensor-parallel shard of a ViT-22B layer, and a full ViT-22B layer.
CONFIGS = {
    "vit_tiny": dict(batch=2, seq=197, hidden=192, heads=3, head_dim=64, mlp=768, ln_eps=1e-6),
    "vit_base": dict(batch=32, seq=197, hidden=768, heads=12, head_dim=64, mlp=3072, ln_eps=1e-6),
    "vit_huge": dict(batch=16, seq=257, hidden=1280, heads=16, head_dim=80, mlp=5120, ln_eps=1e-6),
    "vit22b_tp8": dict(batch=8, seq=256, hidden=6144, heads=6, head_dim=128, mlp=3072, ln_eps=1e-6),
    "vit22b": dict(batch=8, seq=256, hidden=6144, heads=48, head_dim=128, mlp=24576, ln_eps=1e-6),
}


def random_sparse_sign_bf16(shape, seed, density=0.1):
    """A seeded tensor with entries in {-1, 0, 1}, each non-zero with
    probability `density` (sign uniform), stored as bfloat16.  Products of
    such matrices stay small integers, so fp32 accumulation and bf16 outputs
    are exact for layout tests."""
    g = torch.Generator().manual_seed(seed)
    keep = torch.rand(shape, generator=g) < density
    sign = torch.randint(0, 2, shape, generator=g, dtype=torch.int32) * 2 - 1
    return (sign * keep.to(torch.int32)).to(torch.bfloat16)
