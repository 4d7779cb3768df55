"""The layer chain keeps its results when it shares the GPU.

The paper runs encoder kernels beside the LLM's own work: inside its
pipeline bubbles, with the encoder's communication overlapped with LLM
computation (§3.1 design decision 3, §4.2 ScheduleKernels).  Whatever
else runs on the GPU, each kernel must compute exactly what it computes
alone.  The kernels are deterministic (fixed reduction orders, no atomics),
so the bar is bit equality.

Two settings, each against the chain run alone on an idle GPU:
  * co-run: the per-kernel chain on one stream while a loop of bf16 GEMMs
    (torch.matmul, standing in for the LLM's computation) runs on another,
    both streams allowed on every CU;
  * CU-masked co-run: the same pair on two streams restricted to
    complementary CU sets, 32 CUs for the encoder (4 in every XCD) and the
    other 224 for the load.
Both streams are made by hipExtStreamCreateWithCUMask (a full mask for the
plain co-run), which gives each its own hardware queue, and keep the default
priority.  Each test also checks that the load spans the chain.
"""

import ctypes

import pytest
import torch

from helpers import announce, cuda
from paper_2408_03505_amd import binding as B
from paper_2408_03505_amd.synthetic import CONFIGS, PARAM_ORDER, layer_inputs

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

GEMM_N = 8192


class Chain:
    """Preallocated outputs of the per-kernel layer chain (forward then
    backward, the composite's order), launched on a given stream."""

    def __init__(self, cfg, x, p, dout):
        self.cfg, self.x, self.p, self.dout = cfg, x, p, dout
        Bn, S, H, nh, d, F = (cfg[k] for k in ("batch", "seq", "hidden", "heads", "head_dim", "mlp"))
        M, A = Bn * S, nh * d
        bf = dict(dtype=torch.bfloat16, device="cuda")
        f32 = dict(dtype=torch.float32, device="cuda")
        e = torch.empty
        self.t = {
            "y1": e((M, H), **bf), "mean1": e((M,), **f32), "rstd1": e((M,), **f32), "qkv": e((M, 3 * A), **bf),
            "o": e((M, A), **bf), "lse": e((Bn, nh, S), **f32), "h": e((M, H), **bf), "y2": e((M, H), **bf),
            "mean2": e((M,), **f32), "rstd2": e((M,), **f32), "u": e((M, F), **bf), "g": e((M, F), **bf),
            "out": e((M, H), **bf), "du": e((M, F), **bf), "dy2": e((M, H), **bf), "dh": e((M, H), **bf),
            "do": e((M, A), **bf), "dqkv": e((M, 3 * A), **bf), "dy1": e((M, H), **bf), "dx": e((M, H), **bf),
        }
        self.g = {n: torch.empty(tuple(p[n].shape), **f32) for n in PARAM_ORDER}
        self.ln_ws = e((B.ln_bwd_workspace_bytes(M, H),), dtype=torch.uint8, device="cuda")
        self.attn_ws = e((B.attn_bwd_workspace_bytes(Bn, S, nh, d),), dtype=torch.uint8, device="cuda")

    def clear(self):
        for v in list(self.t.values()) + list(self.g.values()):
            v.view(torch.uint8).fill_(0xFF)  # NaN in every float format

    def run(self, s):
        c, x, p, dout, t, g = self.cfg, self.x, self.p, self.dout, self.t, self.g
        Bn, S, nh, d, eps = c["batch"], c["seq"], c["heads"], c["head_dim"], c["ln_eps"]
        B.enc_ln_fwd(x, p["ln1_g"], p["ln1_b"], eps, t["y1"], t["mean1"], t["rstd1"], stream=s)
        B.enc_qkv_fwd(t["y1"], p["w_qkv"], p["b_qkv"], t["qkv"], stream=s)
        B.enc_attn_fwd(Bn, S, nh, d, t["qkv"], t["o"], t["lse"], stream=s)
        B.enc_oproj_fwd(t["o"], p["w_o"], p["b_o"], x, t["h"], stream=s)
        B.enc_ln_fwd(t["h"], p["ln2_g"], p["ln2_b"], eps, t["y2"], t["mean2"], t["rstd2"], stream=s)
        B.enc_mlp_up_fwd(t["y2"], p["w_1"], p["b_1"], t["u"], t["g"], stream=s)
        B.enc_mlp_down_fwd(t["g"], p["w_2"], p["b_2"], t["h"], t["out"], stream=s)
        B.enc_mlp_down_bwd_data(dout, p["w_2"], t["u"], t["du"], stream=s)
        B.enc_mlp_down_bwd_weight(dout, t["g"], g["w_2"], g["b_2"], stream=s)
        B.enc_mlp_up_bwd_data(t["du"], p["w_1"], t["dy2"], stream=s)
        B.enc_mlp_up_bwd_weight(t["du"], t["y2"], g["w_1"], g["b_1"], stream=s)
        B.enc_ln_bwd(t["dy2"], t["h"], t["mean2"], t["rstd2"], p["ln2_g"], dout, t["dh"], g["ln2_g"], g["ln2_b"],
                     ws=self.ln_ws, stream=s)
        B.enc_oproj_bwd_data(t["dh"], p["w_o"], t["do"], stream=s)
        B.enc_oproj_bwd_weight(t["dh"], t["o"], g["w_o"], g["b_o"], stream=s)
        B.enc_attn_bwd(Bn, S, nh, d, t["qkv"], t["o"], t["lse"], t["do"], t["dqkv"], ws=self.attn_ws, stream=s)
        B.enc_qkv_bwd_data(t["dqkv"], p["w_qkv"], t["dy1"], stream=s)
        B.enc_qkv_bwd_weight(t["dqkv"], t["y1"], g["w_qkv"], g["b_qkv"], stream=s)
        B.enc_ln_bwd(t["dy1"], x, t["mean1"], t["rstd1"], p["ln1_g"], t["dh"], t["dx"], g["ln1_g"], g["ln1_b"],
                     ws=self.ln_ws, stream=s)

    def snapshot(self):
        snap = {k: v.clone() for k, v in self.t.items()}
        snap.update({"d" + n: v.clone() for n, v in self.g.items()})
        return snap


def _assert_bit_equal(got, ref, what):
    bad = [k for k in ref if not torch.equal(got[k].view(torch.uint8), ref[k].view(torch.uint8))]
    assert not bad, f"{what}: outputs differ from the chain run alone: {bad}"


def _load(stream, a, b, c, k):
    """Enqueue k bf16 GEMMs on stream; return events around them."""
    with torch.cuda.stream(stream):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(k):
            torch.matmul(a, b, out=c)
        e1.record()
    return e0, e1


def _timed_chain(chain, stream):
    with torch.cuda.stream(stream):
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record()
        chain.run(stream)
        s1.record()
    return s0, s1


def _setup(name):
    cfg = CONFIGS[name]
    x, params, dout = layer_inputs(cfg, seed=5)
    chain = Chain(cfg, cuda(x), {n: cuda(params[n]) for n in PARAM_ORDER}, cuda(dout))
    a = torch.randn(GEMM_N, GEMM_N, device="cuda", dtype=torch.bfloat16)
    b = torch.randn(GEMM_N, GEMM_N, device="cuda", dtype=torch.bfloat16)
    c = torch.empty(GEMM_N, GEMM_N, device="cuda", dtype=torch.bfloat16)
    return chain, a, b, c


def _gemm_ms(stream, a, b, c):
    _load(stream, a, b, c, 2)
    e0, e1 = _load(stream, a, b, c, 5)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / 5


def _hip_runtime():
    """The HIP runtime library torch already loaded into this process."""
    paths = sorted({ln.split()[-1] for ln in open("/proc/self/maps") if "libamdhip64" in ln})
    assert paths, "no HIP runtime mapped in this process"
    hip = ctypes.CDLL(paths[0])
    hip.hipExtStreamCreateWithCUMask.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint32,
                                                 ctypes.POINTER(ctypes.c_uint32)]
    hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
    return hip


class MaskedStreams:
    """Streams created with a CU mask (default priority).  Each such stream
    gets a hardware queue of its own, so two of them really run side by side;
    plain streams may share one of the process's few hardware queues and
    then run one after the other."""

    def __init__(self):
        self.hip = _hip_runtime()
        self.handles = []

    def make(self, mask):
        arr = (ctypes.c_uint32 * len(mask))(*mask)
        h = ctypes.c_void_p()
        err = self.hip.hipExtStreamCreateWithCUMask(ctypes.byref(h), len(mask), arr)
        assert err == 0, f"hipExtStreamCreateWithCUMask failed ({err})"
        self.handles.append(h)
        return torch.cuda.ExternalStream(h.value)

    def close(self):
        torch.cuda.synchronize()
        for h in self.handles:
            self.hip.hipStreamDestroy(h)


def _encoder_mask(words=8, per_word=4):
    """per_word bits of every 32-bit word, word w holding bits w, w+8, ...,
    so each XCD keeps CUs of both sets whichever way mask bits map to XCDs."""
    return [sum(1 << (w % 8 + 8 * k) for k in range(per_word)) for w in range(words)]


def _cu_words():
    ncu = torch.cuda.get_device_properties(0).multi_processor_count
    if ncu != 256:
        pytest.skip(f"the mask layout assumes 256 CUs in 8 XCDs (device has {ncu})")
    return 8


def _corun(chain, enc, load, a, b, c, ref, what, factor):
    """Chain alone on enc, then beside a GEMM loop on load sized to outlast
    it `factor` times over; both runs must equal ref bit for bit."""
    chain.clear()
    torch.cuda.synchronize()
    s0, s1 = _timed_chain(chain, enc)
    torch.cuda.synchronize()
    _assert_bit_equal(chain.snapshot(), ref, f"{what}: chain alone")
    alone_ms = s0.elapsed_time(s1)
    k = max(10, int(factor * alone_ms / _gemm_ms(load, a, b, c)) + 1)
    chain.clear()
    torch.cuda.synchronize()
    l0, l1 = _load(load, a, b, c, k)
    s0, s1 = _timed_chain(chain, enc)
    torch.cuda.synchronize()
    _assert_bit_equal(chain.snapshot(), ref, f"{what}: beside the load")
    timeline = dict(load_ms=l0.elapsed_time(l1), chain_start_ms=l0.elapsed_time(s0),
                    chain_end_ms=l0.elapsed_time(s1), chain_alone_ms=alone_ms, gemms=k)
    # the load started before the chain and ended after it: they shared the GPU
    assert timeline["chain_start_ms"] >= 0 and timeline["chain_end_ms"] <= timeline["load_ms"], timeline
    print(f"[corun] {what}: {timeline}", flush=True)


@pytest.mark.parametrize("name", ["vit_huge", "vit22b_tp8"])
def test_chain_bit_equal_beside_gemm_load(name):
    words = _cu_words()
    announce(f"co-run bit equality {name}")
    chain, a, b, c = _setup(name)
    chain.clear()
    torch.cuda.synchronize()
    chain.run(torch.cuda.current_stream())
    torch.cuda.synchronize()
    ref = chain.snapshot()
    st = MaskedStreams()
    try:
        full = [0xFFFFFFFF] * words
        enc, load = st.make(full), st.make(full)
        # enough load to outlast the chain even if sharing the GPU slows it fiftyfold
        # (its short LayerNorm kernels wait behind whole-chip GEMM workgroups)
        for rep in range(2):
            _corun(chain, enc, load, a, b, c, ref, f"co-run {name} rep {rep}", 50)
    finally:
        st.close()


@pytest.mark.parametrize("name", ["vit22b_tp8"])
def test_chain_bit_equal_on_cu_masked_streams(name):
    words = _cu_words()
    announce(f"CU-masked co-run bit equality {name}")
    chain, a, b, c = _setup(name)
    chain.clear()
    torch.cuda.synchronize()
    chain.run(torch.cuda.current_stream())
    torch.cuda.synchronize()
    ref = chain.snapshot()
    st = MaskedStreams()
    try:
        enc_mask = _encoder_mask(words)
        enc = st.make(enc_mask)
        load = st.make([(~m) & 0xFFFFFFFF for m in enc_mask])
        # on disjoint CU sets the chain is slowed only by shared caches and HBM
        _corun(chain, enc, load, a, b, c, ref, f"masked co-run {name}", 3)
    finally:
        st.close()
