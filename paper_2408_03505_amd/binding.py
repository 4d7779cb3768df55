"""ctypes binding of liboptimus_enc.so (declared in include/optimus_enc.h).

Argument marshalling only: every function checks tensor dtypes, devices,
shapes and contiguity, passes raw device pointers and the current HIP stream
to the C entry point of the same name, and raises EncError on a non-zero
status.  All computation runs in the library's HIP kernels; there is no
fallback path, and a missing library raises at first use.  torch supplies
device memory and streams (outputs are allocated with torch.empty when the
caller does not pass them).
"""

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# OPTIMUS_ENC_LIB names another build of the same C ABI (the host-only
# sanitizer build the CPU tests use); by default the in-tree library loads.
LIB_PATH = os.environ.get("OPTIMUS_ENC_LIB") or os.path.join(_HERE, "liboptimus_enc.so")

PARAM_ORDER = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
               "ln2_g", "ln2_b", "w_1", "b_1", "w_2", "b_2")
SAVED_FIELDS = ("y1", "mean1", "rstd1", "qkv", "o", "lse", "h", "y2", "mean2", "rstd2", "u", "g")
PPARAM_ORDER = ("ln_g", "ln_b", "w_qkv", "qn_g", "qn_b", "kn_g", "kn_b", "w_o", "b_o", "w_1", "b_1", "w_2", "b_2")
PSAVED_FIELDS = ("y", "mean", "rstd", "qkv", "qkvn", "qkstats", "o", "lse", "h", "u", "g")

ENC_OK, ENC_ERR_INVALID, ENC_ERR_UNSUPPORTED, ENC_ERR_ALIGN, ENC_ERR_LAUNCH, ENC_ERR_WORKSPACE = 0, -1, -2, -3, -4, -5


class EncError(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__(f"{fn} failed with status {status}: {msg}")
        self.status = status


class EncCfg(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int), ("seq", ctypes.c_int), ("hidden", ctypes.c_int),
                ("heads", ctypes.c_int), ("head_dim", ctypes.c_int), ("mlp", ctypes.c_int),
                ("ln_eps", ctypes.c_float)]


class EncParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in PARAM_ORDER]


class EncGrads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in PARAM_ORDER]


class EncSavedLayout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_size_t) for n in SAVED_FIELDS] + [("total", ctypes.c_size_t)]


class EncPParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in PPARAM_ORDER]


class EncPGrads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in PPARAM_ORDER]


class EncPSavedLayout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_size_t) for n in PSAVED_FIELDS] + [("total", ctypes.c_size_t)]


_i, _f, _p, _sz = ctypes.c_int, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t
_PCFG = ctypes.POINTER(EncCfg)

# name -> argtypes (every entry point returns int except the two string getters)
_SIGS = {
    "enc_abi_version": [],
    "enc_saved_layout": [_PCFG, ctypes.POINTER(EncSavedLayout)],
    "enc_layer_workspace_bytes": [_PCFG, ctypes.POINTER(_sz)],
    "enc_ln_bwd_workspace_bytes": [_i, _i, ctypes.POINTER(_sz)],
    "enc_attn_bwd_workspace_bytes": [_i, _i, _i, _i, ctypes.POINTER(_sz)],
    "encoder_layer_fwd": [_PCFG, ctypes.POINTER(EncParams), _p, _p, _p, _p, _sz, _p],
    "encoder_layer_bwd": [_PCFG, ctypes.POINTER(EncParams), _p, _p, _p, _p, ctypes.POINTER(EncGrads), _i, _p, _sz, _p],
    "enc_ln_fwd": [_i, _i, _p, _p, _p, _f, _p, _p, _p, _p],
    "enc_qkv_fwd": [_i, _i, _i, _p, _p, _p, _p, _p, _sz, _p],
    "enc_attn_fwd": [_i, _i, _i, _i, _p, _p, _p, _p],
    "enc_oproj_fwd": [_i, _i, _i, _p, _p, _p, _p, _p, _p, _sz, _p],
    "enc_mlp_up_fwd": [_i, _i, _i, _p, _p, _p, _p, _p, _p, _sz, _p],
    "enc_mlp_down_fwd": [_i, _i, _i, _p, _p, _p, _p, _p, _p, _sz, _p],
    "enc_mlp_down_bwd_data": [_i, _i, _i, _p, _p, _p, _p, _p, _sz, _p],
    "enc_mlp_up_bwd_data": [_i, _i, _i, _p, _p, _p, _p, _sz, _p],
    "enc_oproj_bwd_data": [_i, _i, _i, _p, _p, _p, _p, _sz, _p],
    "enc_qkv_bwd_data": [_i, _i, _i, _p, _p, _p, _p, _sz, _p],
    "enc_linear_workspace_bytes": [_i, _i, _i, ctypes.POINTER(_sz)],
    "enc_linear_plan": [_i, _i, _i, _i, ctypes.POINTER(_i), ctypes.POINTER(_i), ctypes.POINTER(_i)],
    "enc_linear_bwd_weight_workspace_bytes": [_i, _i, _i, ctypes.POINTER(_sz)],
    "enc_linear_bwd_weight": [_i, _i, _i, _p, _p, _p, _p, _i, _p, _sz, _p],
    "enc_mlp_down_bwd_weight": [_i, _i, _i, _p, _p, _p, _p, _i, _p, _sz, _p],
    "enc_mlp_up_bwd_weight": [_i, _i, _i, _p, _p, _p, _p, _i, _p, _sz, _p],
    "enc_oproj_bwd_weight": [_i, _i, _i, _p, _p, _p, _p, _i, _p, _sz, _p],
    "enc_qkv_bwd_weight": [_i, _i, _i, _p, _p, _p, _p, _i, _p, _sz, _p],
    "enc_ln_bwd": [_i, _i, _p, _p, _p, _p, _p, _p, _p, _p, _p, _i, _p, _sz, _p],
    "enc_attn_bwd": [_i, _i, _i, _i, _p, _p, _p, _p, _p, _p, _sz, _p],
    "enc_attn_bwd_noalloc": [_i, _i, _i, _i, _p, _p, _p, _p, _p, _p],
    "enc_calib_mfma": [_i, _i, _p, _p],
    "enc_schedule_kernels": [_p, _p, _i, _p, _p, _i, _p, _p],
    "enc_parallel_saved_layout": [_PCFG, ctypes.POINTER(EncPSavedLayout)],
    "enc_parallel_workspace_bytes": [_PCFG, ctypes.POINTER(_sz)],
    "encoder_parallel_fwd": [_PCFG, ctypes.POINTER(EncPParams), _p, _p, _p, _p],
    "encoder_parallel_bwd": [_PCFG, ctypes.POINTER(EncPParams), _p, _p, _p, _p, ctypes.POINTER(EncPGrads), _i, _p,
                             _sz, _p],
    "enc_qk_norm_fwd": [_i, _i, _i, _p, _p, _p, _p, _p, _f, _p, _p, _p],
    "enc_qk_norm_bwd_workspace_bytes": [_i, _i, _i, ctypes.POINTER(_sz)],
    "enc_qk_norm_bwd": [_i, _i, _i, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _i, _p, _sz, _p],
    "enc_qkv_bwd_data_add": [_i, _i, _i, _p, _p, _p, _p, _p, _sz, _p],
    "enc_patch_embed_workspace_bytes": [_i, _i, _i, _i, _i, _i, _i, ctypes.POINTER(_sz)],
    "enc_patch_embed_fwd": [_i, _i, _i, _i, _i, _i, _i, _p, _p, _p, _p, _p, _p, _p, _p, _sz, _p],
    "enc_patch_embed_bwd": [_i, _i, _i, _i, _i, _i, _i, _p, _p, _p, _p, _p, _p, _i, _p, _sz, _p],
    "enc_stack_saved_bytes": [_PCFG, _i, ctypes.POINTER(_sz)],
    "enc_stack_workspace_bytes": [_PCFG, _i, ctypes.POINTER(_sz)],
    "encoder_stack_fwd": [_PCFG, _i, _p, _p, _p, _p, _p, _p, _p],
    "encoder_stack_bwd": [_PCFG, _i, _p, _p, _p, _p, _p, _p, _p, _p, _p, _i, _p, _sz, _p],
    "enc_calib_copy": [_p, _p, _sz, _p],
}

_lib = None


def lib():
    """Load liboptimus_enc.so once; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2408_03505_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, args in _SIGS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        for name in ("enc_status_string",):
            getattr(L, name).argtypes = [ctypes.c_int]
            getattr(L, name).restype = ctypes.c_char_p
        L.enc_last_error.argtypes = []
        L.enc_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _call(name, *args):
    L = lib()
    st = getattr(L, name)(*args)
    if st != ENC_OK:
        raise EncError(name, st, L.enc_last_error().decode())
    return st


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _check(t, name, shape, dtype=torch.bfloat16):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _out(t, name, shape, like, dtype=torch.bfloat16):
    if t is None:
        return torch.empty(shape, dtype=dtype, device=like.device)
    return _check(t, name, shape, dtype)


def make_cfg(cfg):
    return EncCfg(cfg["batch"], cfg["seq"], cfg["hidden"], cfg["heads"], cfg["head_dim"], cfg["mlp"],
                  float(cfg.get("ln_eps", 1e-6)))


def param_shapes(cfg):
    H, A, F = cfg["hidden"], cfg["heads"] * cfg["head_dim"], cfg["mlp"]
    return {"ln1_g": (H,), "ln1_b": (H,), "w_qkv": (3 * A, H), "b_qkv": (3 * A,), "w_o": (H, A), "b_o": (H,),
            "ln2_g": (H,), "ln2_b": (H,), "w_1": (F, H), "b_1": (F,), "w_2": (H, F), "b_2": (H,)}


# ------------------------------------------------------------------ sizing

def saved_layout(cfg):
    L = EncSavedLayout()
    c = make_cfg(cfg)
    _call("enc_saved_layout", ctypes.byref(c), ctypes.byref(L))
    return {n: getattr(L, n) for n in SAVED_FIELDS + ("total",)}


def layer_workspace_bytes(cfg):
    n = ctypes.c_size_t()
    c = make_cfg(cfg)
    _call("enc_layer_workspace_bytes", ctypes.byref(c), ctypes.byref(n))
    return n.value


def ln_bwd_workspace_bytes(rows, cols):
    n = ctypes.c_size_t()
    _call("enc_ln_bwd_workspace_bytes", rows, cols, ctypes.byref(n))
    return n.value


def attn_bwd_workspace_bytes(batch, seq, heads, head_dim):
    n = ctypes.c_size_t()
    _call("enc_attn_bwd_workspace_bytes", batch, seq, heads, head_dim, ctypes.byref(n))
    return n.value


def saved_views(cfg, saved):
    """Typed views of the saved-for-backward buffer (uint8 tensor)."""
    lay = saved_layout(cfg)
    M = cfg["batch"] * cfg["seq"]
    H, A, F = cfg["hidden"], cfg["heads"] * cfg["head_dim"], cfg["mlp"]
    spec = {"y1": ((M, H), torch.bfloat16), "mean1": ((M,), torch.float32), "rstd1": ((M,), torch.float32),
            "qkv": ((M, 3 * A), torch.bfloat16), "o": ((M, A), torch.bfloat16),
            "lse": ((cfg["batch"], cfg["heads"], cfg["seq"]), torch.float32),
            "h": ((M, H), torch.bfloat16), "y2": ((M, H), torch.bfloat16), "mean2": ((M,), torch.float32),
            "rstd2": ((M,), torch.float32), "u": ((M, F), torch.bfloat16), "g": ((M, F), torch.bfloat16)}
    out = {}
    for n, (shape, dt) in spec.items():
        nbytes = int(torch.Size(shape).numel()) * (2 if dt == torch.bfloat16 else 4)
        out[n] = saved[lay[n]:lay[n] + nbytes].view(dt).view(shape)
    return out


# ------------------------------------------------------------------ composites

def _params_struct(cfg, params):
    shapes = param_shapes(cfg)
    return EncParams(*[_ptr(_check(params[n], n, shapes[n])) for n in PARAM_ORDER])


def encoder_layer_fwd(cfg, params, x, out=None, saved=None, ws=None, stream=None):
    """Forward of one encoder layer. Returns (out, saved) with saved a uint8
    device buffer laid out as enc_saved_layout describes."""
    M, H = cfg["batch"] * cfg["seq"], cfg["hidden"]
    _check(x, "x", (M, H))
    out = _out(out, "out", (M, H), x)
    total = saved_layout(cfg)["total"]
    saved = _out(saved, "saved", (total,), x, torch.uint8)
    c, p = make_cfg(cfg), _params_struct(cfg, params)
    if ws is None:  # the layer workspace (split-product partials in the forward)
        ws = torch.empty(layer_workspace_bytes(cfg), dtype=torch.uint8, device=x.device)
    _call("encoder_layer_fwd", ctypes.byref(c), ctypes.byref(p), _ptr(x), _ptr(out), _ptr(saved),
          _ptr(ws), ws.numel() * ws.element_size(), _stream(stream))
    return out, saved


def encoder_layer_bwd(cfg, params, x, saved, dout, grads=None, dx=None, accumulate=False, ws=None, stream=None):
    """Backward of one encoder layer. Returns (dx, grads) with fp32 grads."""
    M, H = cfg["batch"] * cfg["seq"], cfg["hidden"]
    _check(x, "x", (M, H))
    _check(dout, "dout", (M, H))
    dx = _out(dx, "dx", (M, H), x)
    shapes = param_shapes(cfg)
    if grads is None:
        if accumulate:
            raise ValueError("accumulate=True needs existing grads")
        grads = {n: torch.empty(shapes[n], dtype=torch.float32, device=x.device) for n in PARAM_ORDER}
    for n in PARAM_ORDER:
        _check(grads[n], "d" + n, shapes[n], torch.float32)
    if ws is None:
        ws = torch.empty(layer_workspace_bytes(cfg), dtype=torch.uint8, device=x.device)
    total = saved_layout(cfg)["total"]
    _check(saved, "saved", (total,), torch.uint8)
    c, p = make_cfg(cfg), _params_struct(cfg, params)
    g = EncGrads(*[_ptr(grads[n]) for n in PARAM_ORDER])
    _call("encoder_layer_bwd", ctypes.byref(c), ctypes.byref(p), _ptr(x), _ptr(saved), _ptr(dout), _ptr(dx),
          ctypes.byref(g), 1 if accumulate else 0, _ptr(ws), ws.numel(), _stream(stream))
    return dx, grads


# ------------------------------------------------------------------ forward kernels

def enc_ln_fwd(x, gamma, beta, eps, y=None, mean=None, rstd=None, stream=None):
    rows, cols = x.shape
    _check(x, "x", (rows, cols))
    _check(gamma, "gamma", (cols,))
    _check(beta, "beta", (cols,))
    y = _out(y, "y", (rows, cols), x)
    mean = _out(mean, "mean", (rows,), x, torch.float32)
    rstd = _out(rstd, "rstd", (rows,), x, torch.float32)
    _call("enc_ln_fwd", rows, cols, _ptr(x), _ptr(gamma), _ptr(beta), float(eps), _ptr(y), _ptr(mean), _ptr(rstd),
          _stream(stream))
    return y, mean, rstd


def enc_qkv_fwd(y1, w_qkv, b_qkv, qkv=None, ws=None, split=True, stream=None):
    M, H = y1.shape
    A3 = w_qkv.shape[0]
    _check(y1, "y1", (M, H))
    _check(w_qkv, "w_qkv", (A3, H))
    if b_qkv is not None:
        _check(b_qkv, "b_qkv", (A3,))
    qkv = _out(qkv, "qkv", (M, A3), y1)
    if A3 % 3:
        raise ValueError("w_qkv rows must be 3*A")
    wp, wn = _gemm_ws(M, A3, H, ws, split, y1.device)
    _call("enc_qkv_fwd", M, H, A3 // 3, _ptr(y1), _ptr(w_qkv), _ptr(b_qkv), _ptr(qkv), wp, wn, _stream(stream))
    return qkv


def enc_attn_fwd(batch, seq, heads, head_dim, qkv, o=None, lse=None, stream=None):
    A = heads * head_dim
    _check(qkv, "qkv", (batch * seq, 3 * A))
    o = _out(o, "o", (batch * seq, A), qkv)
    lse = _out(lse, "lse", (batch, heads, seq), qkv, torch.float32)
    _call("enc_attn_fwd", batch, seq, heads, head_dim, _ptr(qkv), _ptr(o), _ptr(lse), _stream(stream))
    return o, lse


def enc_oproj_fwd(o, w_o, b_o, resid, h=None, ws=None, split=True, stream=None):
    M, A = o.shape
    H = w_o.shape[0]
    _check(o, "o", (M, A))
    _check(w_o, "w_o", (H, A))
    _check(b_o, "b_o", (H,))
    _check(resid, "resid", (M, H))
    h = _out(h, "h", (M, H), o)
    wp, wn = _gemm_ws(M, H, A, ws, split, o.device)
    _call("enc_oproj_fwd", M, A, H, _ptr(o), _ptr(w_o), _ptr(b_o), _ptr(resid), _ptr(h), wp, wn, _stream(stream))
    return h


def enc_mlp_up_fwd(y2, w_1, b_1, u=None, g=None, ws=None, split=True, stream=None):
    M, H = y2.shape
    F = w_1.shape[0]
    _check(y2, "y2", (M, H))
    _check(w_1, "w_1", (F, H))
    _check(b_1, "b_1", (F,))
    u = _out(u, "u", (M, F), y2)
    g = _out(g, "g", (M, F), y2)
    wp, wn = _gemm_ws(M, F, H, ws, split, y2.device)
    _call("enc_mlp_up_fwd", M, H, F, _ptr(y2), _ptr(w_1), _ptr(b_1), _ptr(u), _ptr(g), wp, wn, _stream(stream))
    return u, g


def enc_mlp_down_fwd(g, w_2, b_2, resid, out=None, ws=None, split=True, stream=None):
    M, F = g.shape
    H = w_2.shape[0]
    _check(g, "g", (M, F))
    _check(w_2, "w_2", (H, F))
    _check(b_2, "b_2", (H,))
    _check(resid, "resid", (M, H))
    out = _out(out, "out", (M, H), g)
    wp, wn = _gemm_ws(M, H, F, ws, split, g.device)
    _call("enc_mlp_down_fwd", M, F, H, _ptr(g), _ptr(w_2), _ptr(b_2), _ptr(resid), _ptr(out), wp, wn,
          _stream(stream))
    return out


# ------------------------------------------------------------------ backward kernels

def enc_mlp_down_bwd_data(dout, w_2, u, du=None, ws=None, split=True, stream=None):
    M, H = dout.shape
    F = w_2.shape[1]
    _check(dout, "dout", (M, H))
    _check(w_2, "w_2", (H, F))
    _check(u, "u", (M, F))
    du = _out(du, "du", (M, F), dout)
    wp, wn = _gemm_ws(M, F, H, ws, split, dout.device)
    _call("enc_mlp_down_bwd_data", M, F, H, _ptr(dout), _ptr(w_2), _ptr(u), _ptr(du), wp, wn, _stream(stream))
    return du


def enc_mlp_up_bwd_data(du, w_1, dy2=None, ws=None, split=True, stream=None):
    M, F = du.shape
    H = w_1.shape[1]
    _check(du, "du", (M, F))
    _check(w_1, "w_1", (F, H))
    dy2 = _out(dy2, "dy2", (M, H), du)
    wp, wn = _gemm_ws(M, H, F, ws, split, du.device)
    _call("enc_mlp_up_bwd_data", M, H, F, _ptr(du), _ptr(w_1), _ptr(dy2), wp, wn, _stream(stream))
    return dy2


def enc_oproj_bwd_data(dh, w_o, do=None, ws=None, split=True, stream=None):
    M, H = dh.shape
    A = w_o.shape[1]
    _check(dh, "dh", (M, H))
    _check(w_o, "w_o", (H, A))
    do = _out(do, "do", (M, A), dh)
    wp, wn = _gemm_ws(M, A, H, ws, split, dh.device)
    _call("enc_oproj_bwd_data", M, A, H, _ptr(dh), _ptr(w_o), _ptr(do), wp, wn, _stream(stream))
    return do


def enc_qkv_bwd_data(dqkv, w_qkv, dy1=None, ws=None, split=True, stream=None):
    M, A3 = dqkv.shape
    H = w_qkv.shape[1]
    _check(dqkv, "dqkv", (M, A3))
    _check(w_qkv, "w_qkv", (A3, H))
    dy1 = _out(dy1, "dy1", (M, H), dqkv)
    wp, wn = _gemm_ws(M, H, A3, ws, split, dqkv.device)
    _call("enc_qkv_bwd_data", M, H, A3 // 3, _ptr(dqkv), _ptr(w_qkv), _ptr(dy1), wp, wn, _stream(stream))
    return dy1


def linear_bwd_weight_workspace_bytes(M, N, K):
    n = _sz()
    _call("enc_linear_bwd_weight_workspace_bytes", M, N, K, ctypes.byref(n))
    return n.value


def linear_workspace_bytes(M, N, K):
    n = _sz()
    _call("enc_linear_workspace_bytes", M, N, K, ctypes.byref(n))
    return n.value


LAYOUT_FWD, LAYOUT_DGRAD, LAYOUT_WGRAD = 0, 1, 2


def linear_plan(layout, M, N, K):
    """(tile_rows, tile_cols, splits) of one projection product as the entry
    points launch it with a workspace (host query, no device work)."""
    r, c, sp = _i(), _i(), _i()
    _call("enc_linear_plan", layout, M, N, K, ctypes.byref(r), ctypes.byref(c), ctypes.byref(sp))
    return r.value, c.value, sp.value


def _gemm_ws(M, N, K, ws, split, device):
    """Workspace argument of a forward or input-gradient product with output
    [M, N] and contraction K: a caller tensor, a fresh one of the queried
    size (split=True, ws=None), or none (split=False)."""
    if not split:
        return ctypes.c_void_p(0), 0
    if ws is None:
        need = linear_workspace_bytes(M, N, K)
        if need == 0:
            return ctypes.c_void_p(0), 0
        ws = torch.empty(need, dtype=torch.uint8, device=device)
    return _ptr(ws), ws.numel() * ws.element_size()


def _wgrad_ws(M, N, K, ws, split, device):
    """Workspace argument of a weight-gradient call: a caller tensor, a fresh
    one of the queried size (split=True, ws=None), or none (split=False)."""
    if not split:
        return ctypes.c_void_p(0), 0
    if ws is None:
        need = linear_bwd_weight_workspace_bytes(M, N, K)
        if need == 0:
            return ctypes.c_void_p(0), 0
        ws = torch.empty(need, dtype=torch.uint8, device=device)
    return _ptr(ws), ws.numel() * ws.element_size()


def enc_linear_bwd_weight(dY, X, dW=None, db=None, accumulate=False, with_db=True, ws=None, split=True, stream=None):
    M, N = dY.shape
    K = X.shape[1]
    _check(dY, "dY", (M, N))
    _check(X, "X", (M, K))
    if accumulate and (dW is None or (with_db and db is None)):
        raise ValueError("accumulate=True needs existing dW/db")
    dW = _out(dW, "dW", (N, K), dY, torch.float32)
    if with_db:
        db = _out(db, "db", (N,), dY, torch.float32)
    wp, wn = _wgrad_ws(M, N, K, ws, split, dY.device)
    _call("enc_linear_bwd_weight", M, N, K, _ptr(dY), _ptr(X), _ptr(dW), _ptr(db), 1 if accumulate else 0, wp, wn,
          _stream(stream))
    return dW, db


def _named_wgrad(name, M, a, b, N, K, dY, X, dW, db, accumulate, ws, split, stream):
    wp, wn = _wgrad_ws(M, N, K, ws, split, dY.device)
    _call(name, M, a, b, _ptr(dY), _ptr(X), _ptr(dW), _ptr(db), 1 if accumulate else 0, wp, wn, _stream(stream))
    return dW, db


def enc_mlp_down_bwd_weight(dout, g, dw_2, db_2, accumulate=False, ws=None, split=True, stream=None):
    M, H = dout.shape
    F = g.shape[1]
    _check(dout, "dout", (M, H)); _check(g, "g", (M, F))
    _check(dw_2, "dw_2", (H, F), torch.float32); _check(db_2, "db_2", (H,), torch.float32)
    return _named_wgrad("enc_mlp_down_bwd_weight", M, F, H, H, F, dout, g, dw_2, db_2, accumulate, ws, split, stream)


def enc_mlp_up_bwd_weight(du, y2, dw_1, db_1, accumulate=False, ws=None, split=True, stream=None):
    M, F = du.shape
    H = y2.shape[1]
    _check(du, "du", (M, F)); _check(y2, "y2", (M, H))
    _check(dw_1, "dw_1", (F, H), torch.float32); _check(db_1, "db_1", (F,), torch.float32)
    return _named_wgrad("enc_mlp_up_bwd_weight", M, H, F, F, H, du, y2, dw_1, db_1, accumulate, ws, split, stream)


def enc_oproj_bwd_weight(dh, o, dw_o, db_o, accumulate=False, ws=None, split=True, stream=None):
    M, H = dh.shape
    A = o.shape[1]
    _check(dh, "dh", (M, H)); _check(o, "o", (M, A))
    _check(dw_o, "dw_o", (H, A), torch.float32); _check(db_o, "db_o", (H,), torch.float32)
    return _named_wgrad("enc_oproj_bwd_weight", M, A, H, H, A, dh, o, dw_o, db_o, accumulate, ws, split, stream)


def enc_qkv_bwd_weight(dqkv, y1, dw_qkv, db_qkv, accumulate=False, ws=None, split=True, stream=None):
    M, A3 = dqkv.shape
    H = y1.shape[1]
    _check(dqkv, "dqkv", (M, A3)); _check(y1, "y1", (M, H))
    _check(dw_qkv, "dw_qkv", (A3, H), torch.float32); _check(db_qkv, "db_qkv", (A3,), torch.float32)
    return _named_wgrad("enc_qkv_bwd_weight", M, H, A3 // 3, A3, H, dqkv, y1, dw_qkv, db_qkv, accumulate, ws, split,
                        stream)


def enc_ln_bwd(dy, x, mean, rstd, gamma, dresid=None, dx=None, dgamma=None, dbeta=None, accumulate=False,
               ws=None, stream=None):
    rows, cols = x.shape
    _check(dy, "dy", (rows, cols))
    _check(x, "x", (rows, cols))
    _check(mean, "mean", (rows,), torch.float32)
    _check(rstd, "rstd", (rows,), torch.float32)
    _check(gamma, "gamma", (cols,))
    if dresid is not None:
        _check(dresid, "dresid", (rows, cols))
    if accumulate and (dgamma is None or dbeta is None):
        raise ValueError("accumulate=True needs existing dgamma/dbeta")
    dx = _out(dx, "dx", (rows, cols), x)
    dgamma = _out(dgamma, "dgamma", (cols,), x, torch.float32)
    dbeta = _out(dbeta, "dbeta", (cols,), x, torch.float32)
    need = ln_bwd_workspace_bytes(rows, cols)
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=x.device)
    _call("enc_ln_bwd", rows, cols, _ptr(dy), _ptr(x), _ptr(mean), _ptr(rstd), _ptr(gamma), _ptr(dresid), _ptr(dx),
          _ptr(dgamma), _ptr(dbeta), 1 if accumulate else 0, _ptr(ws), ws.numel() * ws.element_size(),
          _stream(stream))
    return dx, dgamma, dbeta


def enc_attn_bwd(batch, seq, heads, head_dim, qkv, o, lse, do, dqkv=None, ws=None, stream=None):
    A = heads * head_dim
    M = batch * seq
    _check(qkv, "qkv", (M, 3 * A))
    _check(o, "o", (M, A))
    _check(lse, "lse", (batch, heads, seq), torch.float32)
    _check(do, "do", (M, A))
    dqkv = _out(dqkv, "dqkv", (M, 3 * A), qkv)
    need = attn_bwd_workspace_bytes(batch, seq, heads, head_dim)
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=qkv.device)
    _call("enc_attn_bwd", batch, seq, heads, head_dim, _ptr(qkv), _ptr(o), _ptr(lse), _ptr(do), _ptr(dqkv),
          _ptr(ws), ws.numel() * ws.element_size(), _stream(stream))
    return dqkv


def enc_attn_bwd_noalloc(batch, seq, heads, head_dim, qkv, o, lse, do, dqkv, stream=None):
    """enc_attn_bwd with its D vector in the library's static per-GPU scratch:
    the C call allocates nothing (dqkv must be given).  Calls that overlap on
    one GPU race on the scratch."""
    A = heads * head_dim
    M = batch * seq
    _check(qkv, "qkv", (M, 3 * A))
    _check(o, "o", (M, A))
    _check(lse, "lse", (batch, heads, seq), torch.float32)
    _check(do, "do", (M, A))
    _check(dqkv, "dqkv", (M, 3 * A))
    _call("enc_attn_bwd_noalloc", batch, seq, heads, head_dim, _ptr(qkv), _ptr(o), _ptr(lse), _ptr(do), _ptr(dqkv),
          _stream(stream))
    return dqkv


# ---------------------------------------------------------------- measurement helpers

def enc_calib_mfma(blocks, iters, out=None, stream=None, device="cuda"):
    """MFMA-only reference loop: blocks * 4 * iters * 16 * 32768 flops."""
    if out is None:
        out = torch.empty(blocks * 256, dtype=torch.float32, device=device)
    _check(out, "out", (blocks * 256,), torch.float32)
    _call("enc_calib_mfma", blocks, iters, _ptr(out), _stream(stream))
    return out


def calib_mfma_flops(blocks, iters):
    return blocks * 4 * iters * 16 * 32768


def enc_calib_copy(src, dst, stream=None):
    """Reference device copy of src's bytes into dst (both contiguous, same byte size)."""
    if not (isinstance(src, torch.Tensor) and isinstance(dst, torch.Tensor)):
        raise TypeError("src and dst must be torch.Tensors")
    nbytes = src.numel() * src.element_size()
    if not (src.is_cuda and dst.is_cuda and src.is_contiguous() and dst.is_contiguous()):
        raise ValueError("src and dst must be contiguous device tensors")
    if dst.numel() * dst.element_size() != nbytes:
        raise ValueError("src and dst must have the same byte size")
    _call("enc_calib_copy", _ptr(src), _ptr(dst), nbytes, _stream(stream))
    return dst


# ---------------------------------------------------------------- kernel-to-bubble packing

def enc_schedule_kernels(kernel_us, interval_us, interval_bubble, kernel_comm=None):
    """Place kernels (chain order) into timeline intervals; host-side, no GPU.

    Returns (interval index per kernel, -1 if unplaced; start offset in us,
    -1.0 if unplaced; number placed)."""
    kus = (ctypes.c_double * len(kernel_us))(*[float(v) for v in kernel_us])
    ius = (ctypes.c_double * len(interval_us))(*[float(v) for v in interval_us])
    bub = (ctypes.c_int * len(interval_bubble))(*[1 if b else 0 for b in interval_bubble])
    if len(interval_bubble) != len(interval_us):
        raise ValueError("interval_us and interval_bubble differ in length")
    comm = None
    if kernel_comm is not None:
        if len(kernel_comm) != len(kernel_us):
            raise ValueError("kernel_us and kernel_comm differ in length")
        comm = (ctypes.c_int * len(kernel_comm))(*[1 if c else 0 for c in kernel_comm])
    where = (ctypes.c_int * max(1, len(kernel_us)))()
    off = (ctypes.c_double * max(1, len(kernel_us)))()
    L = lib()
    placed = L.enc_schedule_kernels(ctypes.cast(kus, _p), ctypes.cast(comm, _p) if comm is not None else None,
                                    len(kernel_us), ctypes.cast(ius, _p), ctypes.cast(bub, _p), len(interval_us),
                                    ctypes.cast(where, _p), ctypes.cast(off, _p))
    if placed < 0:
        raise EncError("enc_schedule_kernels", placed, L.enc_last_error().decode())
    n = len(kernel_us)
    return list(where)[:n], list(off)[:n], placed


# ---------------------------------------------------------------- ViT-22B-style parallel block

def parallel_param_shapes(cfg):
    H, A, F, d = cfg["hidden"], cfg["heads"] * cfg["head_dim"], cfg["mlp"], cfg["head_dim"]
    return {"ln_g": (H,), "ln_b": (H,), "w_qkv": (3 * A, H), "qn_g": (d,), "qn_b": (d,), "kn_g": (d,),
            "kn_b": (d,), "w_o": (H, A), "b_o": (H,), "w_1": (F, H), "b_1": (F,), "w_2": (H, F), "b_2": (H,)}


def parallel_saved_layout(cfg):
    L = EncPSavedLayout()
    c = make_cfg(cfg)
    _call("enc_parallel_saved_layout", ctypes.byref(c), ctypes.byref(L))
    return {n: getattr(L, n) for n in PSAVED_FIELDS + ("total",)}


def parallel_workspace_bytes(cfg):
    n = ctypes.c_size_t()
    c = make_cfg(cfg)
    _call("enc_parallel_workspace_bytes", ctypes.byref(c), ctypes.byref(n))
    return n.value


def parallel_saved_views(cfg, saved):
    """Typed views of the parallel block's saved buffer (uint8 tensor)."""
    lay = parallel_saved_layout(cfg)
    M, nh = cfg["batch"] * cfg["seq"], cfg["heads"]
    H, A, F = cfg["hidden"], nh * cfg["head_dim"], cfg["mlp"]
    bf, f32 = torch.bfloat16, torch.float32
    spec = {"y": ((M, H), bf), "mean": ((M,), f32), "rstd": ((M,), f32), "qkv": ((M, 3 * A), bf),
            "qkvn": ((M, 3 * A), bf), "qkstats": ((M, nh, 4), f32), "o": ((M, A), bf),
            "lse": ((cfg["batch"], nh, cfg["seq"]), f32), "h": ((M, H), bf), "u": ((M, F), bf), "g": ((M, F), bf)}
    out = {}
    for n, (shape, dt) in spec.items():
        nbytes = int(torch.Size(shape).numel()) * (2 if dt == bf else 4)
        out[n] = saved[lay[n]:lay[n] + nbytes].view(dt).view(shape)
    return out


def _pparams_struct(cfg, params):
    shapes = parallel_param_shapes(cfg)
    return EncPParams(*[_ptr(_check(params[n], n, shapes[n])) for n in PPARAM_ORDER])


def encoder_parallel_fwd(cfg, params, x, out=None, saved=None, stream=None):
    """Forward of the parallel block. Returns (out, saved)."""
    M, H = cfg["batch"] * cfg["seq"], cfg["hidden"]
    _check(x, "x", (M, H))
    out = _out(out, "out", (M, H), x)
    total = parallel_saved_layout(cfg)["total"]
    saved = _out(saved, "saved", (total,), x, torch.uint8)
    c, p = make_cfg(cfg), _pparams_struct(cfg, params)
    _call("encoder_parallel_fwd", ctypes.byref(c), ctypes.byref(p), _ptr(x), _ptr(out), _ptr(saved), _stream(stream))
    return out, saved


def encoder_parallel_bwd(cfg, params, x, saved, dout, grads=None, dx=None, accumulate=False, ws=None, stream=None):
    """Backward of the parallel block. Returns (dx, grads) with fp32 grads."""
    M, H = cfg["batch"] * cfg["seq"], cfg["hidden"]
    _check(x, "x", (M, H))
    _check(dout, "dout", (M, H))
    dx = _out(dx, "dx", (M, H), x)
    shapes = parallel_param_shapes(cfg)
    if grads is None:
        if accumulate:
            raise ValueError("accumulate=True needs existing grads")
        grads = {n: torch.empty(shapes[n], dtype=torch.float32, device=x.device) for n in PPARAM_ORDER}
    for n in PPARAM_ORDER:
        _check(grads[n], "d" + n, shapes[n], torch.float32)
    if ws is None:
        ws = torch.empty(parallel_workspace_bytes(cfg), dtype=torch.uint8, device=x.device)
    _check(saved, "saved", (parallel_saved_layout(cfg)["total"],), torch.uint8)
    c, p = make_cfg(cfg), _pparams_struct(cfg, params)
    g = EncPGrads(*[_ptr(grads[n]) for n in PPARAM_ORDER])
    _call("encoder_parallel_bwd", ctypes.byref(c), ctypes.byref(p), _ptr(x), _ptr(saved), _ptr(dout), _ptr(dx),
          ctypes.byref(g), 1 if accumulate else 0, _ptr(ws), ws.numel(), _stream(stream))
    return dx, grads


def qk_norm_bwd_workspace_bytes(M, heads, head_dim):
    n = ctypes.c_size_t()
    _call("enc_qk_norm_bwd_workspace_bytes", M, heads, head_dim, ctypes.byref(n))
    return n.value


def enc_qk_norm_fwd(heads, head_dim, qkv, qn_g, qn_b, kn_g, kn_b, eps, qkvn=None, stats=None, stream=None):
    M = qkv.shape[0]
    A = heads * head_dim
    _check(qkv, "qkv", (M, 3 * A))
    for n, t in (("qn_g", qn_g), ("qn_b", qn_b), ("kn_g", kn_g), ("kn_b", kn_b)):
        _check(t, n, (head_dim,))
    qkvn = _out(qkvn, "qkvn", (M, 3 * A), qkv)
    stats = _out(stats, "stats", (M, heads, 4), qkv, torch.float32)
    _call("enc_qk_norm_fwd", M, heads, head_dim, _ptr(qkv), _ptr(qn_g), _ptr(qn_b), _ptr(kn_g), _ptr(kn_b),
          float(eps), _ptr(qkvn), _ptr(stats), _stream(stream))
    return qkvn, stats


def enc_qk_norm_bwd(heads, head_dim, dqkvn, qkv, stats, qn_g, kn_g, dqkv=None, grads=None, accumulate=False,
                    ws=None, stream=None):
    """Returns (dqkv, grads) with grads a dict of fp32 qn_g, qn_b, kn_g, kn_b."""
    M = qkv.shape[0]
    A = heads * head_dim
    _check(dqkvn, "dqkvn", (M, 3 * A))
    _check(qkv, "qkv", (M, 3 * A))
    _check(stats, "stats", (M, heads, 4), torch.float32)
    _check(qn_g, "qn_g", (head_dim,))
    _check(kn_g, "kn_g", (head_dim,))
    dqkv = _out(dqkv, "dqkv", (M, 3 * A), qkv)
    names = ("qn_g", "qn_b", "kn_g", "kn_b")
    if grads is None:
        if accumulate:
            raise ValueError("accumulate=True needs existing grads")
        grads = {n: torch.empty(head_dim, dtype=torch.float32, device=qkv.device) for n in names}
    for n in names:
        _check(grads[n], "d" + n, (head_dim,), torch.float32)
    if ws is None:
        ws = torch.empty(qk_norm_bwd_workspace_bytes(M, heads, head_dim), dtype=torch.uint8, device=qkv.device)
    _call("enc_qk_norm_bwd", M, heads, head_dim, _ptr(dqkvn), _ptr(qkv), _ptr(stats), _ptr(qn_g), _ptr(kn_g),
          _ptr(dqkv), *[_ptr(grads[n]) for n in names], 1 if accumulate else 0, _ptr(ws), ws.numel(),
          _stream(stream))
    return dqkv, grads


def enc_qkv_bwd_data_add(dqkv, w_qkv, addend, dy=None, ws=None, split=True, stream=None):
    M, A3 = dqkv.shape
    H = w_qkv.shape[1]
    _check(dqkv, "dqkv", (M, A3))
    _check(w_qkv, "w_qkv", (A3, H))
    _check(addend, "addend", (M, H))
    dy = _out(dy, "dy", (M, H), dqkv)
    wp, wn = _gemm_ws(M, H, A3, ws, split, dqkv.device)
    _call("enc_qkv_bwd_data_add", M, H, A3 // 3, _ptr(dqkv), _ptr(w_qkv), _ptr(addend), _ptr(dy), wp, wn,
          _stream(stream))
    return dy


# ---------------------------------------------------------------- whole encoder

def patch_kp(channels, patch):
    """Columns of the patch matrix: C*p*p rounded up to a multiple of 8."""
    return (channels * patch * patch + 7) // 8 * 8


def patch_embed_workspace_bytes(batch, channels, img_h, img_w, patch, hidden, has_cls):
    n = ctypes.c_size_t()
    _call("enc_patch_embed_workspace_bytes", batch, channels, img_h, img_w, patch, hidden, int(bool(has_cls)),
          ctypes.byref(n))
    return n.value


def enc_patch_embed_fwd(images, patch, w_pe, b_pe, pos, cls=None, patches=None, x0=None, ws=None, stream=None):
    """images [B, C, H_img, W_img] bf16; w_pe [hidden, Kp] (zero beyond C*p*p).
    Returns (x0 [B*S, hidden], patches [B*N, Kp])."""
    B, C, ih, iw = images.shape
    hidden = w_pe.shape[0]
    kp = patch_kp(C, patch)
    N = (ih // patch) * (iw // patch)
    has_cls = cls is not None
    S = N + int(has_cls)
    _check(images, "images", (B, C, ih, iw))
    _check(w_pe, "w_pe", (hidden, kp))
    _check(b_pe, "b_pe", (hidden,))
    _check(pos, "pos", (S, hidden))
    if has_cls:
        _check(cls, "cls", (hidden,))
    patches = _out(patches, "patches", (B * N, kp), images)
    x0 = _out(x0, "x0", (B * S, hidden), images)
    need = patch_embed_workspace_bytes(B, C, ih, iw, patch, hidden, has_cls)
    if ws is None and need:
        ws = torch.empty(need, dtype=torch.uint8, device=images.device)
    _call("enc_patch_embed_fwd", B, C, ih, iw, patch, hidden, int(has_cls), _ptr(images), _ptr(w_pe), _ptr(b_pe),
          _ptr(cls), _ptr(pos), _ptr(patches), _ptr(x0), _ptr(ws), ws.numel() if ws is not None else 0,
          _stream(stream))
    return x0, patches


def enc_patch_embed_bwd(images_shape, patch, dx0, patches, has_cls, grads=None, accumulate=False, ws=None,
                        stream=None):
    """Returns a dict of fp32 gradients w_pe [hidden, Kp], b_pe, pos [S, hidden], cls (with has_cls)."""
    B, C, ih, iw = images_shape
    kp = patch_kp(C, patch)
    N = (ih // patch) * (iw // patch)
    S = N + int(bool(has_cls))
    hidden = dx0.shape[1]
    _check(dx0, "dx0", (B * S, hidden))
    _check(patches, "patches", (B * N, kp))
    shapes = {"w_pe": (hidden, kp), "b_pe": (hidden,), "pos": (S, hidden)}
    if has_cls:
        shapes["cls"] = (hidden,)
    if grads is None:
        if accumulate:
            raise ValueError("accumulate=True needs existing grads")
        grads = {k: torch.empty(v, dtype=torch.float32, device=dx0.device) for k, v in shapes.items()}
    for k, v in shapes.items():
        _check(grads[k], "d" + k, v, torch.float32)
    need = patch_embed_workspace_bytes(B, C, ih, iw, patch, hidden, has_cls)
    if ws is None and need:
        ws = torch.empty(need, dtype=torch.uint8, device=dx0.device)
    _call("enc_patch_embed_bwd", B, C, ih, iw, patch, hidden, int(bool(has_cls)), _ptr(dx0), _ptr(patches),
          _ptr(grads["w_pe"]), _ptr(grads["b_pe"]), _ptr(grads.get("cls")), _ptr(grads["pos"]),
          1 if accumulate else 0, _ptr(ws), ws.numel() if ws is not None else 0, _stream(stream))
    return grads


def stack_saved_bytes(cfg, layers):
    n = ctypes.c_size_t()
    c = make_cfg(cfg)
    _call("enc_stack_saved_bytes", ctypes.byref(c), layers, ctypes.byref(n))
    return n.value


def stack_workspace_bytes(cfg, layers):
    n = ctypes.c_size_t()
    c = make_cfg(cfg)
    _call("enc_stack_workspace_bytes", ctypes.byref(c), layers, ctypes.byref(n))
    return n.value


def encoder_stack_fwd(cfg, layer_params, lnf_g, lnf_b, x0, out=None, saved=None, stream=None):
    """layer_params: list of per-layer parameter dicts (PARAM_ORDER).  Returns (out, saved)."""
    L = len(layer_params)
    M, H = cfg["batch"] * cfg["seq"], cfg["hidden"]
    _check(x0, "x0", (M, H))
    _check(lnf_g, "lnf_g", (H,))
    _check(lnf_b, "lnf_b", (H,))
    out = _out(out, "out", (M, H), x0)
    saved = _out(saved, "saved", (stack_saved_bytes(cfg, L),), x0, torch.uint8)
    arr = (EncParams * L)(*[_params_struct(cfg, p) for p in layer_params])
    c = make_cfg(cfg)
    _call("encoder_stack_fwd", ctypes.byref(c), L, ctypes.cast(arr, _p), _ptr(lnf_g), _ptr(lnf_b), _ptr(x0),
          _ptr(out), _ptr(saved), _stream(stream))
    return out, saved


def encoder_stack_bwd(cfg, layer_params, lnf_g, x0, saved, dout, grads=None, lnf_grads=None, dx0=None,
                      accumulate=False, ws=None, stream=None):
    """Returns (dx0, per-layer grads list, (dlnf_g, dlnf_b))."""
    L = len(layer_params)
    M, H = cfg["batch"] * cfg["seq"], cfg["hidden"]
    _check(x0, "x0", (M, H))
    _check(dout, "dout", (M, H))
    _check(saved, "saved", (stack_saved_bytes(cfg, L),), torch.uint8)
    dx0 = _out(dx0, "dx0", (M, H), x0)
    shapes = param_shapes(cfg)
    if grads is None:
        if accumulate:
            raise ValueError("accumulate=True needs existing grads")
        grads = [{n: torch.empty(shapes[n], dtype=torch.float32, device=x0.device) for n in PARAM_ORDER}
                 for _ in range(L)]
        lnf_grads = tuple(torch.empty(H, dtype=torch.float32, device=x0.device) for _ in range(2))
    for g in grads:
        for n in PARAM_ORDER:
            _check(g[n], "d" + n, shapes[n], torch.float32)
    for t in lnf_grads:
        _check(t, "dlnf", (H,), torch.float32)
    if ws is None:
        ws = torch.empty(stack_workspace_bytes(cfg, L), dtype=torch.uint8, device=x0.device)
    arr = (EncParams * L)(*[_params_struct(cfg, p) for p in layer_params])
    garr = (EncGrads * L)(*[EncGrads(*[_ptr(g[n]) for n in PARAM_ORDER]) for g in grads])
    c = make_cfg(cfg)
    _call("encoder_stack_bwd", ctypes.byref(c), L, ctypes.cast(arr, _p), _ptr(lnf_g), _ptr(x0), _ptr(saved),
          _ptr(dout), _ptr(dx0), ctypes.cast(garr, _p), _ptr(lnf_grads[0]), _ptr(lnf_grads[1]),
          1 if accumulate else 0, _ptr(ws), ws.numel(), _stream(stream))
    return dx0, grads, lnf_grads
