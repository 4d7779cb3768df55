"""Host-side checks of the C-ABI library: it loads, exports every entry point
the header declares, sizes buffers consistently, and rejects bad arguments
with the documented status codes before launching anything.

These tests never launch a kernel.  The argument-error cases pass fake,
never-dereferenced pointers, so they are skipped whenever a GPU is visible.
"""

import ctypes
import os
import re

import pytest
import torch

from paper_2408_03505_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "optimus_enc.h")

no_gpu_only = pytest.mark.skipif(torch.cuda.is_available(), reason="fake-pointer cases run only without a GPU")

VIT22B = dict(batch=8, seq=256, hidden=6144, heads=48, head_dim=128, mlp=24576, ln_eps=1e-6)
VIT_TINY = dict(batch=2, seq=197, hidden=192, heads=3, head_dim=64, mlp=768, ln_eps=1e-6)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)
    return sorted(set(n for n in names if n not in ("if", "defined")))


def test_header_declares_the_chain():
    names = declared_functions()
    for want in ("encoder_layer_fwd", "encoder_layer_bwd", "enc_ln_fwd", "enc_qkv_fwd", "enc_attn_fwd",
                 "enc_oproj_fwd", "enc_mlp_up_fwd", "enc_mlp_down_fwd", "enc_mlp_down_bwd_data",
                 "enc_linear_bwd_weight", "enc_mlp_up_bwd_data", "enc_ln_bwd", "enc_oproj_bwd_data",
                 "enc_attn_bwd", "enc_qkv_bwd_data"):
        assert want in names


def test_library_exports_every_declared_symbol():
    L = B.lib()
    missing = [n for n in declared_functions() if not hasattr(L, n)]
    assert not missing, missing
    # the binding covers every declared entry point as well
    covered = set(B._SIGS) | {"enc_status_string", "enc_last_error"}
    assert set(declared_functions()) <= covered


def test_abi_version_and_status_strings():
    L = B.lib()
    assert L.enc_abi_version() == 2
    for code in (0, -1, -2, -3, -4, -5):
        assert len(L.enc_status_string(code)) > 0
    assert L.enc_status_string(7) == b"unknown status"


@pytest.mark.parametrize("cfg", [VIT22B, VIT_TINY, dict(VIT22B, heads=6, mlp=3072)])
def test_saved_layout_is_aligned_and_disjoint(cfg):
    lay = B.saved_layout(cfg)
    M = cfg["batch"] * cfg["seq"]
    H, A, F = cfg["hidden"], cfg["heads"] * cfg["head_dim"], cfg["mlp"]
    sizes = {"y1": M * H * 2, "mean1": M * 4, "rstd1": M * 4, "qkv": M * 3 * A * 2, "o": M * A * 2,
             "lse": cfg["batch"] * cfg["heads"] * cfg["seq"] * 4, "h": M * H * 2, "y2": M * H * 2,
             "mean2": M * 4, "rstd2": M * 4, "u": M * F * 2, "g": M * F * 2}
    spans = sorted((lay[n], lay[n] + s) for n, s in sizes.items())
    for n in sizes:
        assert lay[n] % 256 == 0
    for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
        assert a1 <= b0
    assert spans[-1][1] <= lay["total"]


@pytest.mark.parametrize("cfg", [VIT22B, VIT_TINY])
def test_parallel_saved_layout_is_aligned_and_disjoint(cfg):
    lay = B.parallel_saved_layout(cfg)
    M, nh = cfg["batch"] * cfg["seq"], cfg["heads"]
    H, A, F = cfg["hidden"], nh * cfg["head_dim"], cfg["mlp"]
    sizes = {"y": M * H * 2, "mean": M * 4, "rstd": M * 4, "qkv": M * 3 * A * 2, "qkvn": M * 3 * A * 2,
             "qkstats": M * nh * 16, "o": M * A * 2, "lse": cfg["batch"] * nh * cfg["seq"] * 4, "h": M * H * 2,
             "u": M * F * 2, "g": M * F * 2}
    spans = sorted((lay[n], lay[n] + s) for n, s in sizes.items())
    assert all(lay[n] % 256 == 0 for n in sizes)
    assert all(a1 <= b0 for (_, a1), (b0, _) in zip(spans, spans[1:]))
    assert spans[-1][1] <= lay["total"]
    assert B.parallel_workspace_bytes(cfg) > 0
    assert B.qk_norm_bwd_workspace_bytes(M, nh, cfg["head_dim"]) % (4 * 4 * cfg["head_dim"]) == 0


def test_weight_gradient_split_plan_sizes():
    # outputs that fill the GPU never split; small outputs with many tokens do
    assert B.linear_bwd_weight_workspace_bytes(2048, 24576, 6144) == 0
    assert B.linear_bwd_weight_workspace_bytes(2048, 6144, 18432) == 0
    assert B.linear_bwd_weight_workspace_bytes(394, 576, 192) == 0
    # ViT-Base's out-projection: a 768 x 768 output over 6304 tokens; one fp32
    # partial of dW and db per split, two or more splits
    need = B.linear_bwd_weight_workspace_bytes(6304, 768, 768)
    assert need % (768 * 768 * 4 + 768 * 4) == 0 and need // (768 * 768 * 4 + 768 * 4) >= 2
    # the layer workspace holds the largest of the four weight gradients' partials
    base = dict(batch=32, seq=197, hidden=768, heads=12, head_dim=64, mlp=3072, ln_eps=1e-6)
    M = 32 * 197
    wg = max(B.linear_bwd_weight_workspace_bytes(M, n, k) for n, k in ((768, 3072), (3072, 768), (768, 768),
                                                                        (2304, 768)))
    assert wg > 0 and B.layer_workspace_bytes(base) >= wg


def test_linear_plan_matches_the_workspace_queries():
    # a plan splits exactly when the workspace query asks for partials, and
    # the workspace holds one fp32 partial per split
    r256 = lambda x: (x + 255) // 256 * 256
    for M, N, K in ((2048, 768, 6144), (2048, 24576, 6144), (1000, 2048, 512), (300, 200, 1280),
                    (2048, 2304, 6144), (6304, 768, 3072)):
        for layout in (B.LAYOUT_FWD, B.LAYOUT_DGRAD):
            bm, bn, sp = B.linear_plan(layout, M, N, K)
            ws = B.linear_workspace_bytes(M, N, K)
            assert (sp > 1) == (ws > 0), (M, N, K, layout)
            if sp > 1:
                assert ws == r256(sp * M * N * 4) and (bm, bn) == (128, 128)
    for M, N, K in ((6304, 768, 768), (6304, 3072, 768), (4112, 1280, 1280), (2048, 24576, 6144),
                    (2048, 6144, 768), (2000, 768, 256)):
        bm, bn, sp = B.linear_plan(B.LAYOUT_WGRAD, M, N, K)
        ws = B.linear_bwd_weight_workspace_bytes(M, N, K)
        assert (sp > 1) == (ws > 0), (M, N, K)
        if sp > 1:
            assert ws == r256(sp * N * K * 4) + r256(sp * N * 4)
            # every split covers at least 512 tokens but the last
            assert (M + sp - 1) // sp >= 512


def test_linear_plan_tiles():
    # ViT-22B layer (2048 tokens): 256x256 tiles where the grid fills whole
    # rounds of the 256 CUs, 256x192 where 256x256 would leave CUs idle
    assert B.linear_plan(B.LAYOUT_FWD, 2048, 24576, 6144) == (256, 256, 1)
    assert B.linear_plan(B.LAYOUT_FWD, 2048, 18432, 6144) == (256, 192, 1)
    assert B.linear_plan(B.LAYOUT_DGRAD, 2048, 6144, 24576) == (256, 192, 1)
    assert B.linear_plan(B.LAYOUT_WGRAD, 2048, 24576, 6144) == (256, 256, 1)
    assert B.linear_plan(B.LAYOUT_WGRAD, 2048, 6144, 24576) == (256, 256, 1)
    # a contiguous contraction that is not a multiple of 64 takes the
    # register-staged kernel's tiles, unsplit
    assert B.linear_plan(B.LAYOUT_FWD, 300, 200, 200) == (128, 128, 1)
    assert B.linear_plan(B.LAYOUT_FWD, 8192, 8192, 8200) == (256, 128, 1)
    # arguments are checked like the entry points'
    for args, code in (((7, 2048, 768, 768), B.ENC_ERR_INVALID), ((B.LAYOUT_FWD, 0, 768, 768), B.ENC_ERR_INVALID),
                       ((B.LAYOUT_FWD, 16, 770, 768), B.ENC_ERR_UNSUPPORTED)):
        with pytest.raises(B.EncError) as e:
            B.linear_plan(*args)
        assert e.value.status == code
    L = B.lib()
    i = ctypes.c_int()
    assert L.enc_linear_plan(B.LAYOUT_FWD, 16, 64, 64, None, ctypes.byref(i), ctypes.byref(i)) == B.ENC_ERR_INVALID


def test_workspace_sizes():
    assert B.layer_workspace_bytes(VIT22B) > 0
    for rows, cols in ((2048, 6144), (10, 192), (6304, 768), (1, 8)):
        ws = B.ln_bwd_workspace_bytes(rows, cols)
        # whole fp32 partial rows for dgamma and dbeta, at most one pair per row
        assert ws > 0 and ws % (cols * 8) == 0 and ws <= rows * cols * 8
    assert B.attn_bwd_workspace_bytes(8, 256, 48, 128) == 8 * 48 * 256 * 4


def _status(name, *args):
    L = B.lib()
    return getattr(L, name)(*args)


def test_bad_configs_are_rejected():
    for bad, code in ((dict(VIT22B, head_dim=96), B.ENC_ERR_UNSUPPORTED),
                      (dict(VIT22B, hidden=6145), B.ENC_ERR_UNSUPPORTED),
                      (dict(VIT22B, mlp=100), B.ENC_ERR_UNSUPPORTED),
                      (dict(VIT22B, batch=0), B.ENC_ERR_INVALID),
                      (dict(VIT22B, seq=-3), B.ENC_ERR_INVALID),
                      (dict(VIT22B, hidden=32768), B.ENC_ERR_UNSUPPORTED),
                      (dict(VIT22B, batch=4096), B.ENC_ERR_UNSUPPORTED)):
        with pytest.raises(B.EncError) as e:
            B.layer_workspace_bytes(bad)
        assert e.value.status == code


FAKE = 0x10000  # aligned, never dereferenced

# Every tensor under 2^31 elements (M * 3A = 2147481600), but qkv plus the
# attention kernels' one-tile overhang past the 4 GiB of 32-bit byte offsets.
NEAR_LIMIT = dict(batch=1, seq=5592400, hidden=8, heads=1, head_dim=128, mlp=8, ln_eps=1e-6)


def test_attention_address_limit_is_a_cfg_check():
    for query in (B.layer_workspace_bytes, B.saved_layout, B.parallel_workspace_bytes, B.parallel_saved_layout):
        with pytest.raises(B.EncError) as e:
            query(NEAR_LIMIT)
        assert e.value.status == B.ENC_ERR_UNSUPPORTED and "4 GiB" in str(e.value), query
    # one fewer token of overhang room fits
    ok = dict(NEAR_LIMIT, seq=NEAR_LIMIT["seq"] - 64)
    assert B.layer_workspace_bytes(ok) > 0


@no_gpu_only
def test_composites_refuse_before_launching():
    # The composites validate every kernel's shape limits before the first
    # launch; with fake pointers a launch would fault, so a clean
    # ENC_ERR_UNSUPPORTED shows that nothing was enqueued.
    p, s = ctypes.c_void_p(FAKE), ctypes.c_void_p(0)
    cfg = B.make_cfg(NEAR_LIMIT)
    params = B.EncParams(*[FAKE] * 12)
    grads = B.EncGrads(*[FAKE] * 12)
    assert _status("encoder_layer_fwd", ctypes.byref(cfg), ctypes.byref(params), p, p, p, p, 0, s) \
        == B.ENC_ERR_UNSUPPORTED
    assert _status("encoder_layer_bwd", ctypes.byref(cfg), ctypes.byref(params), p, p, p, p, ctypes.byref(grads),
                   1, p, 1 << 40, s) == B.ENC_ERR_UNSUPPORTED
    assert _status("encoder_stack_fwd", ctypes.byref(cfg), 2, (B.EncParams * 2)(params, params), p, p, p, p, p, s) \
        == B.ENC_ERR_UNSUPPORTED
    pp = B.EncPParams(*[FAKE] * 13)
    pg = B.EncPGrads(*[FAKE] * 13)
    assert _status("encoder_parallel_fwd", ctypes.byref(cfg), ctypes.byref(pp), p, p, p, s) == B.ENC_ERR_UNSUPPORTED
    assert _status("encoder_parallel_bwd", ctypes.byref(cfg), ctypes.byref(pp), p, p, p, p, ctypes.byref(pg), 1, p,
                   1 << 40, s) == B.ENC_ERR_UNSUPPORTED
    assert b"4 GiB" in B.lib().enc_last_error()


@no_gpu_only
def test_null_and_misaligned_pointers_are_rejected():
    p, z = ctypes.c_void_p(FAKE), ctypes.c_void_p(0)
    s = ctypes.c_void_p(0)
    assert _status("enc_ln_fwd", 4, 64, z, p, p, ctypes.c_float(1e-6), p, p, p, s) == B.ENC_ERR_INVALID
    assert _status("enc_ln_fwd", 4, 64, ctypes.c_void_p(FAKE + 2), p, p, ctypes.c_float(1e-6), p, p, p, s) \
        == B.ENC_ERR_ALIGN
    assert b"not 16-byte aligned" in B.lib().enc_last_error()
    # b_qkv may be NULL, qkv not
    assert _status("enc_qkv_fwd", 8, 64, 64, p, p, p, z, z, 0, s) == B.ENC_ERR_INVALID
    assert _status("enc_qkv_fwd", 8, 64, 64, p, p, ctypes.c_void_p(FAKE + 4), p, z, 0, s) == B.ENC_ERR_ALIGN
    # a product workspace is optional; a given one must be aligned and large enough
    need = B.linear_workspace_bytes(2048, 1024, 6144)
    assert need > 0
    assert _status("enc_mlp_up_fwd", 2048, 6144, 1024, p, p, p, p, p, ctypes.c_void_p(FAKE + 8), need, s) \
        == B.ENC_ERR_ALIGN
    assert _status("enc_mlp_up_fwd", 2048, 6144, 1024, p, p, p, p, p, p, need - 1, s) == B.ENC_ERR_WORKSPACE
    assert _status("enc_qk_norm_fwd", 4, 2, 64, p, p, p, z, p, ctypes.c_float(1e-6), p, p, s) == B.ENC_ERR_INVALID
    assert _status("enc_qk_norm_fwd", 4, 2, 96, p, p, p, p, p, ctypes.c_float(1e-6), p, p, s) \
        == B.ENC_ERR_UNSUPPORTED
    assert _status("enc_qkv_bwd_data_add", 8, 64, 64, p, p, z, p, ctypes.c_void_p(0), 0, s) == B.ENC_ERR_INVALID
    assert _status("enc_attn_fwd", 1, 8, 1, 64, p, z, p, s) == B.ENC_ERR_INVALID
    assert _status("enc_linear_bwd_weight", 8, 64, 64, p, p, z, z, 0, z, 0, s) == B.ENC_ERR_INVALID
    # db may be NULL, but a misaligned db is an error
    assert _status("enc_linear_bwd_weight", 8, 64, 64, p, p, p, ctypes.c_void_p(FAKE + 4), 0, z, 0, s) \
        == B.ENC_ERR_ALIGN
    # a workspace is optional, but a given one must be aligned and large enough
    need = B.linear_bwd_weight_workspace_bytes(6304, 768, 768)
    assert need > 0
    assert _status("enc_linear_bwd_weight", 6304, 768, 768, p, p, p, p, 0, ctypes.c_void_p(FAKE + 8), need, s) \
        == B.ENC_ERR_ALIGN
    assert _status("enc_linear_bwd_weight", 6304, 768, 768, p, p, p, p, 0, p, need - 1, s) == B.ENC_ERR_WORKSPACE


@no_gpu_only
def test_bad_shapes_are_rejected():
    p, s = ctypes.c_void_p(FAKE), ctypes.c_void_p(0)
    assert _status("enc_ln_fwd", 4, 60, p, p, p, ctypes.c_float(1e-6), p, p, p, s) == B.ENC_ERR_UNSUPPORTED
    assert _status("enc_ln_fwd", 0, 64, p, p, p, ctypes.c_float(1e-6), p, p, p, s) == B.ENC_ERR_INVALID
    assert _status("enc_ln_fwd", 4, 64, p, p, p, ctypes.c_float(-1.0), p, p, p, s) == B.ENC_ERR_INVALID
    assert _status("enc_attn_fwd", 1, 8, 1, 96, p, p, p, s) == B.ENC_ERR_UNSUPPORTED
    # qkv just under 2^31 elements but past the attention kernels' 32-bit byte offsets
    assert _status("enc_attn_fwd", 1, 116500, 48, 128, p, p, p, s) == B.ENC_ERR_UNSUPPORTED
    assert b"4 GiB" in B.lib().enc_last_error()
    # per-kernel GEMM operands at 2^31 elements are refused
    assert _status("enc_mlp_down_fwd", 87382, 24576, 64, p, p, p, p, p, ctypes.c_void_p(0), 0, s) == B.ENC_ERR_UNSUPPORTED
    assert _status("enc_qkv_fwd", 8, 60, 64, p, p, p, p, ctypes.c_void_p(0), 0, s) == B.ENC_ERR_UNSUPPORTED
    assert _status("enc_mlp_up_fwd", -1, 64, 64, p, p, p, p, p, ctypes.c_void_p(0), 0, s) == B.ENC_ERR_INVALID


@no_gpu_only
def test_noalloc_attention_backward_checks_its_limit():
    p, z, s = ctypes.c_void_p(FAKE), ctypes.c_void_p(0), ctypes.c_void_p(0)
    # batch*heads*seq past the 2^20 rows of the static scratch
    assert _status("enc_attn_bwd_noalloc", 256, 257, 16, 64, p, p, p, p, p, s) == B.ENC_ERR_UNSUPPORTED
    assert b"static scratch" in B.lib().enc_last_error()
    assert _status("enc_attn_bwd_noalloc", 1, 8, 1, 96, p, p, p, p, p, s) == B.ENC_ERR_UNSUPPORTED
    assert _status("enc_attn_bwd_noalloc", 1, 8, 1, 64, p, p, p, p, z, s) == B.ENC_ERR_INVALID
    assert _status("enc_attn_bwd_noalloc", 1, 8, 1, 64, p, p, ctypes.c_void_p(FAKE + 4), p, p, s) == B.ENC_ERR_ALIGN


@no_gpu_only
def test_calibration_arguments_are_checked():
    p, s = ctypes.c_void_p(FAKE), ctypes.c_void_p(0)
    assert _status("enc_calib_mfma", 0, 10, p, s) == B.ENC_ERR_INVALID
    assert _status("enc_calib_mfma", 4, -1, p, s) == B.ENC_ERR_INVALID
    assert _status("enc_calib_mfma", 4, 10, ctypes.c_void_p(0), s) == B.ENC_ERR_INVALID
    q = ctypes.c_void_p(FAKE + (1 << 20))
    assert _status("enc_calib_copy", p, q, 0, s) == B.ENC_ERR_INVALID
    assert _status("enc_calib_copy", p, q, 24, s) == B.ENC_ERR_INVALID
    assert _status("enc_calib_copy", ctypes.c_void_p(FAKE + 8), q, 32, s) == B.ENC_ERR_ALIGN
    assert _status("enc_calib_copy", p, ctypes.c_void_p(FAKE + 16), 64, s) == B.ENC_ERR_INVALID  # overlap
    assert b"overlap" in B.lib().enc_last_error()


@no_gpu_only
def test_patch_and_stack_arguments_are_checked():
    p, z, s = ctypes.c_void_p(FAKE), ctypes.c_void_p(0), ctypes.c_void_p(0)
    # image side not a multiple of the patch
    assert _status("enc_patch_embed_fwd", 1, 3, 30, 28, 14, 64, 0, p, p, p, z, p, p, p, z, 0, s) \
        == B.ENC_ERR_UNSUPPORTED
    assert _status("enc_patch_embed_fwd", 1, 3, 28, 28, 14, 64, 2, p, p, p, p, p, p, p, p, 1 << 20, s) \
        == B.ENC_ERR_INVALID
    # a class token needs cls and a workspace
    assert _status("enc_patch_embed_fwd", 1, 3, 28, 28, 14, 64, 1, p, p, p, z, p, p, p, p, 1 << 20, s) \
        == B.ENC_ERR_INVALID
    assert _status("enc_patch_embed_fwd", 1, 3, 28, 28, 14, 64, 1, p, p, p, p, p, p, p, p, 16, s) \
        == B.ENC_ERR_WORKSPACE
    assert B.patch_embed_workspace_bytes(2, 3, 224, 224, 16, 192, False) == 0
    assert B.patch_embed_workspace_bytes(2, 3, 224, 224, 16, 192, True) == 2 * 196 * 192 * 2
    assert B.patch_kp(3, 14) == 592 and B.patch_kp(3, 16) == 768
    cfg = B.make_cfg(VIT_TINY)
    assert _status("encoder_stack_fwd", ctypes.byref(cfg), 0, p, p, p, p, p, p, s) == B.ENC_ERR_INVALID
    one = B.stack_saved_bytes(VIT_TINY, 1)
    assert B.stack_saved_bytes(VIT_TINY, 4) > 3 * one and B.stack_workspace_bytes(VIT_TINY, 4) > 0


@no_gpu_only
def test_small_workspace_is_rejected():
    p, s = ctypes.c_void_p(FAKE), ctypes.c_void_p(0)
    need = B.ln_bwd_workspace_bytes(16, 64)
    assert _status("enc_ln_bwd", 16, 64, p, p, p, p, p, ctypes.c_void_p(0), p, p, p, 0, p, need - 1, s) \
        == B.ENC_ERR_WORKSPACE
    need = B.attn_bwd_workspace_bytes(1, 8, 1, 64)
    assert _status("enc_attn_bwd", 1, 8, 1, 64, p, p, p, p, p, p, need - 1, s) == B.ENC_ERR_WORKSPACE
    cfg = B.make_cfg(VIT_TINY)
    params = B.EncParams(*[FAKE] * 12)
    grads = B.EncGrads(*[FAKE] * 12)
    need = B.layer_workspace_bytes(VIT_TINY)
    assert _status("encoder_layer_bwd", ctypes.byref(cfg), ctypes.byref(params), p, p, p, p, ctypes.byref(grads),
                   0, p, need - 1, s) == B.ENC_ERR_WORKSPACE
    params.w_o = 0
    assert _status("encoder_layer_fwd", ctypes.byref(cfg), ctypes.byref(params), p, p, p, p, 0, s) \
        == B.ENC_ERR_INVALID
    assert b"w_o is NULL" in B.lib().enc_last_error()


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        B.lib()


def test_bench_flop_count_matches_the_oracle():
    # the bench counts flops from its own per-kernel table; it must agree with
    # the oracle's count of one layer forward (times three for fwd + bwd)
    import bench
    import oracle
    from paper_2408_03505_amd.synthetic import CONFIGS
    for name, cfg in CONFIGS.items():
        assert bench.step_flops(cfg) == 3 * oracle.layer_flops(cfg), name
