"""Host-only cases run against the sanitizer build of the C ABI.

Not collected by default: tests/test_host_sanitizers.py runs this file, with
the library's host code built under AddressSanitizer and
UndefinedBehaviorSanitizer and linked against stand-in launchers, so every
entry point runs its argument checks, buffer layouts and whole composite
chains (several layers for the stack) on fake device pointers without any
device code.  Refuses to run against any other library: the product library
would launch kernels on these pointers.
"""

import ctypes

import pytest

from paper_2408_03505_amd import binding as B

L = B.lib()
if not hasattr(L, "enc_host_stub_build"):
    raise RuntimeError("host_san_cases.py runs only against the host-only sanitizer build (OPTIMUS_ENC_LIB)")

P = ctypes.c_void_p(0x10000)
S0 = ctypes.c_void_p(0)
CFGS = [dict(batch=8, seq=256, hidden=6144, heads=48, head_dim=128, mlp=24576, ln_eps=1e-6),
        dict(batch=32, seq=197, hidden=768, heads=12, head_dim=64, mlp=3072, ln_eps=1e-6),
        dict(batch=2, seq=197, hidden=192, heads=3, head_dim=64, mlp=768, ln_eps=1e-6),
        dict(batch=3, seq=33, hidden=256, heads=2, head_dim=80, mlp=320, ln_eps=1e-5)]


def _ok(name, *args):
    st = getattr(L, name)(*args)
    assert st == B.ENC_OK, (name, st, L.enc_last_error())


@pytest.mark.parametrize("cfg", CFGS)
def test_layer_composites_run_their_chain(cfg):
    c = B.make_cfg(cfg)
    params = B.EncParams(*[0x10000] * 12)
    grads = B.EncGrads(*[0x20000] * 12)
    ws = B.layer_workspace_bytes(cfg)
    _ok("encoder_layer_fwd", ctypes.byref(c), ctypes.byref(params), P, P, P, P, ws, S0)
    for acc in (0, 1):
        _ok("encoder_layer_bwd", ctypes.byref(c), ctypes.byref(params), P, P, P, P, ctypes.byref(grads), acc, P, ws,
            S0)
    pp = B.EncPParams(*[0x10000] * 13)
    pg = B.EncPGrads(*[0x20000] * 13)
    _ok("encoder_parallel_fwd", ctypes.byref(c), ctypes.byref(pp), P, P, P, S0)
    _ok("encoder_parallel_bwd", ctypes.byref(c), ctypes.byref(pp), P, P, P, P, ctypes.byref(pg), 1, P,
        B.parallel_workspace_bytes(cfg), S0)


@pytest.mark.parametrize("layers", [1, 3])
def test_stack_composites_run_every_layer(layers):
    cfg = CFGS[1]
    c = B.make_cfg(cfg)
    params = (B.EncParams * layers)(*[B.EncParams(*[0x10000] * 12) for _ in range(layers)])
    grads = (B.EncGrads * layers)(*[B.EncGrads(*[0x20000] * 12) for _ in range(layers)])
    _ok("encoder_stack_fwd", ctypes.byref(c), layers, params, P, P, P, P, P, S0)
    _ok("encoder_stack_bwd", ctypes.byref(c), layers, params, P, P, P, P, P, grads, P, P, 0, P,
        B.stack_workspace_bytes(cfg, layers), S0)


def test_per_kernel_entry_points_run():
    M, H, A, F = 394, 192, 192, 768
    f = ctypes.c_float(1e-6)
    _ok("enc_ln_fwd", M, H, P, P, P, f, P, P, P, S0)
    _ok("enc_qkv_fwd", M, H, A, P, P, P, P, S0, 0, S0)
    _ok("enc_qkv_fwd", M, H, A, P, P, S0, P, S0, 0, S0)  # no bias
    _ok("enc_attn_fwd", 2, 197, 3, 64, P, P, P, S0)
    _ok("enc_oproj_fwd", M, A, H, P, P, P, P, P, S0, 0, S0)
    _ok("enc_mlp_up_fwd", M, H, F, P, P, P, P, P, S0, 0, S0)
    _ok("enc_mlp_down_fwd", M, F, H, P, P, P, P, P, S0, 0, S0)
    _ok("enc_mlp_down_bwd_data", M, F, H, P, P, P, P, S0, 0, S0)
    _ok("enc_mlp_up_bwd_data", M, H, F, P, P, P, S0, 0, S0)
    _ok("enc_oproj_bwd_data", M, A, H, P, P, P, S0, 0, S0)
    _ok("enc_qkv_bwd_data", M, H, A, P, P, P, S0, 0, S0)
    _ok("enc_linear_bwd_weight", M, F, H, P, P, P, P, 1, S0, 0, S0)
    _ok("enc_linear_bwd_weight", M, F, H, P, P, P, S0, 0, S0, 0, S0)  # no bias gradient
    # a split weight gradient (small output, many tokens) with its workspace
    need = B.linear_bwd_weight_workspace_bytes(6304, 768, 768)
    _ok("enc_linear_bwd_weight", 6304, 768, 768, P, P, P, P, 1, P, need, S0)
    for name, n, k in (("enc_mlp_down_bwd_weight", F, H), ("enc_mlp_up_bwd_weight", H, F),
                       ("enc_oproj_bwd_weight", A, H), ("enc_qkv_bwd_weight", H, A)):
        _ok(name, M, n, k, P, P, P, P, 0, S0, 0, S0)
    _ok("enc_ln_bwd", M, H, P, P, P, P, P, S0, P, P, P, 0, P, B.ln_bwd_workspace_bytes(M, H), S0)
    _ok("enc_attn_bwd", 2, 197, 3, 64, P, P, P, P, P, P, B.attn_bwd_workspace_bytes(2, 197, 3, 64), S0)
    _ok("enc_attn_bwd_noalloc", 2, 197, 3, 64, P, P, P, P, P, S0)
    _ok("enc_qk_norm_fwd", M, 3, 64, P, P, P, P, P, f, P, P, S0)
    _ok("enc_qk_norm_bwd", M, 3, 64, P, P, P, P, P, P, P, P, P, P, 0, P, B.qk_norm_bwd_workspace_bytes(M, 3, 64),
        S0)
    _ok("enc_qkv_bwd_data_add", M, H, A, P, P, P, P, S0, 0, S0)
    # split forward and input-gradient products with their workspaces
    need = B.linear_workspace_bytes(2048, 1024, 6144)
    assert need > 0
    _ok("enc_mlp_up_fwd", 2048, 6144, 1024, P, P, P, P, P, P, need, S0)
    _ok("enc_mlp_down_bwd_data", 2048, 1024, 6144, P, P, P, P, P, need, S0)
    need = B.linear_workspace_bytes(2048, 768, 6144)
    _ok("enc_oproj_bwd_data", 2048, 768, 6144, P, P, P, P, need, S0)
    for cls in (0, 1):
        ws = B.patch_embed_workspace_bytes(2, 3, 224, 224, 14, 192, bool(cls))
        _ok("enc_patch_embed_fwd", 2, 3, 224, 224, 14, 192, cls, P, P, P, P if cls else S0, P, P, P,
            P if cls else S0, ws, S0)
        _ok("enc_patch_embed_bwd", 2, 3, 224, 224, 14, 192, cls, P, P, P, P, P if cls else S0, P, 1,
            P if cls else S0, ws, S0)
    _ok("enc_calib_mfma", 4, 10, P, S0)
    _ok("enc_calib_copy", P, ctypes.c_void_p(0x10000 + (1 << 20)), 4096, S0)


def test_linear_plan_queries():
    r, c, sp = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    for layout in (B.LAYOUT_FWD, B.LAYOUT_DGRAD, B.LAYOUT_WGRAD):
        for M, N, K in ((2048, 24576, 6144), (6304, 768, 768), (300, 200, 200), (1, 8, 8), (8192, 8192, 8200)):
            _ok("enc_linear_plan", layout, M, N, K, ctypes.byref(r), ctypes.byref(c), ctypes.byref(sp))
            assert r.value in (128, 256) and c.value in (128, 192, 256) and 1 <= sp.value <= 16
    assert L.enc_linear_plan(9, 16, 8, 8, ctypes.byref(r), ctypes.byref(c), ctypes.byref(sp)) == B.ENC_ERR_INVALID
