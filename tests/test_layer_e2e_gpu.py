"""End-to-end parity of the composite layer entry points at full size.

For each full-size workload (ViT-Base, ViT-Huge, one tensor-parallel 1/8
shard of a ViT-22B layer, a full ViT-22B layer), `encoder_layer_fwd` and
`encoder_layer_bwd` run on the seeded bf16 inputs, and the float64 oracle
runs the same layer from the same inputs.  Every element of the output,
of the twelve saved intermediates, of dx and of the twelve parameter
gradients is compared, so the error built up over the whole chain of
kernels is bounded against the plain definition of the layer: splitting
the layer into kernels changes when work runs, never what it computes
(the paper's kernel-level decomposition, §3.1 design decision 3, and the
kernel packing of §4.2).

Bar, per tensor: max|gpu - ref| / max|ref| <= 2e-2 for activations and
saved statistics, <= 5e-2 for dx and the parameter gradients.
"""

import json
import os

import numpy as np
import pytest
import torch

import oracle
from helpers import TOL_ACT, TOL_GRAD, announce, cuda, f64, max_rel
from paper_2408_03505_amd import binding as B
from paper_2408_03505_amd.synthetic import CONFIGS, PARAM_ORDER, layer_inputs

pytestmark = [pytest.mark.gpu, pytest.mark.slow,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

SAVED = ("y1", "mean1", "rstd1", "qkv", "o", "lse", "h", "y2", "mean2", "rstd2", "u", "g")


def _record(name, errs, gerrs):
    """Print the measured errors, and append them as one JSON line to the
    file OPTIMUS_PARITY_LOG names, if set."""
    line = {"config": name, "act": errs, "grad": gerrs}
    print("[parity-e2e] " + json.dumps(line), flush=True)
    path = os.environ.get("OPTIMUS_PARITY_LOG")
    if path:
        with open(path, "a") as f:
            f.write(json.dumps(line) + "\n")


@pytest.mark.parametrize("name", ["vit_base", "vit_huge", "vit22b_tp8", "vit22b"])
def test_layer_end_to_end(name):
    cfg = CONFIGS[name]
    announce(f"end-to-end layer fwd+bwd {name} {cfg}")
    x, params, dout = layer_inputs(cfg, seed=0)
    gp = {n: cuda(params[n]) for n in PARAM_ORDER}
    gx, gd = cuda(x), cuda(dout)
    out, saved = B.encoder_layer_fwd(cfg, gp, gx)
    dx, grads = B.encoder_layer_bwd(cfg, gp, gx, saved, gd)
    torch.cuda.synchronize()
    # Move every result to the host now and free the device copies.
    views = B.saved_views(cfg, saved)
    got = {"out": f64(out), "dx": f64(dx)}
    for k in SAVED:
        got[k] = f64(views[k])
    for n in PARAM_ORDER:
        got["d" + n] = f64(grads[n])
    del out, saved, dx, grads, views, gp, gx, gd
    torch.cuda.empty_cache()

    p64 = {n: f64(params[n]) for n in PARAM_ORDER}
    X = f64(x)
    rout, rsaved = oracle.layer_fwd(cfg, p64, X)
    errs = {"out": max_rel(got["out"], rout)}
    del rout
    for k in SAVED:
        errs[k] = max_rel(got[k], rsaved[k])
    rdx, rgrads, _ = oracle.layer_bwd(cfg, p64, X, rsaved, f64(dout))
    del rsaved
    gerrs = {"dx": max_rel(got["dx"], rdx)}
    for n in PARAM_ORDER:
        gerrs["d" + n] = max_rel(got["d" + n], rgrads[n])
    _record(name, errs, gerrs)
    bad = {k: e for k, e in errs.items() if not e <= TOL_ACT}
    bad.update({k: e for k, e in gerrs.items() if not e <= TOL_GRAD})
    assert not bad, bad
