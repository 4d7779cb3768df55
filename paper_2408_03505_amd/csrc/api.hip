// C-ABI entry points: argument validation, workspace/saved-buffer layout,
// and the forward/backward chains of one encoder layer on one stream.
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <string>

#include "../../include/optimus_enc.h"
#include "kernels.hpp"
#include "status.hpp"

using namespace optimus;

namespace {
thread_local std::string g_last_error;
}  // namespace

int optimus::set_error(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int optimus::clear_error() {
  g_last_error.clear();
  return ENC_OK;
}

namespace {

template <typename... Args>
int fail(int code, const char *fmt, Args... args) {
  return set_error(code, fmt, args...);
}

int ok() { return clear_error(); }

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline hipStream_t as_stream(enc_stream_t s) { return reinterpret_cast<hipStream_t>(s); }

// Null and alignment checks for a list of required pointers.
struct PtrCheck {
  int code = ENC_OK;
  const char *fn;
  explicit PtrCheck(const char *f) : fn(f) {}
  PtrCheck &req(const void *p, const char *name) {
    if (code != ENC_OK) return *this;
    if (!p) code = fail(ENC_ERR_INVALID, "%s: %s is NULL", fn, name);
    else if (!aligned16(p)) code = fail(ENC_ERR_ALIGN, "%s: %s is not 16-byte aligned", fn, name);
    return *this;
  }
  PtrCheck &opt(const void *p, const char *name) {
    if (code != ENC_OK || !p) return *this;
    if (!aligned16(p)) code = fail(ENC_ERR_ALIGN, "%s: %s is not 16-byte aligned", fn, name);
    return *this;
  }
};

int check_dims(const char *fn, std::initializer_list<int> dims) {
  for (int d : dims)
    if (d <= 0) return fail(ENC_ERR_INVALID, "%s: dimensions must be positive", fn);
  return ENC_OK;
}

int check_mult8(const char *fn, std::initializer_list<int> dims) {
  for (int d : dims)
    if (d % 8 != 0) return fail(ENC_ERR_UNSUPPORTED, "%s: feature widths must be multiples of 8 (got %d)", fn, d);
  return ENC_OK;
}

// Largest product of dimensions that still indexes safely with 32-bit ints
// inside the kernels (row index * leading dimension is computed in 64 bits,
// but tile indices and row counts are 32-bit).
constexpr long kMaxElems = 1L << 31;

// A launcher refused a shape that the argument checks accepted.  The checks
// cover every refusal condition (check_cfg), so this is unreachable; if it
// ever happens, kernels of the same call may already be enqueued, which is
// what ENC_ERR_LAUNCH reports.
int refused_after_checks(const char *fn) {
  return fail(ENC_ERR_LAUNCH, "%s: internal error: a kernel refused a shape the argument checks accepted", fn);
}

int launched(const char *fn) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(ENC_ERR_LAUNCH, "%s: kernel launch failed: %s", fn, hipGetErrorString(e));
  return ok();
}

// The attention kernels address qkv, plus one 64-token tile of overhang and a
// 256-byte row tail, with 32-bit byte offsets into a buffer resource.
bool attn_addressable(uint64_t tokens, uint64_t heads, uint64_t d) {
  return (tokens + 64) * 3 * heads * d * 2 + 256 < (1ull << 32);
}

// Every refusal condition of every kernel a layer composite launches is
// checked here, so that a composite that passes check_cfg (and its pointer
// and workspace checks) launches its whole chain: the GEMM launchers always
// have a kernel (the register-staged one covers every multiple of 8), the
// LayerNorm kernels cover widths up to 16384, and attention is limited by
// head_dim and by attn_addressable.
int check_cfg(const char *fn, const enc_cfg_t *c) {
  if (!c) return fail(ENC_ERR_INVALID, "%s: cfg is NULL", fn);
  int r = check_dims(fn, {c->batch, c->seq, c->hidden, c->heads, c->head_dim, c->mlp});
  if (r) return r;
  if (c->head_dim != 64 && c->head_dim != 80 && c->head_dim != 128)
    return fail(ENC_ERR_UNSUPPORTED, "%s: head_dim must be 64, 80 or 128 (got %d)", fn, c->head_dim);
  if ((r = check_mult8(fn, {c->hidden, c->heads * c->head_dim, c->mlp}))) return r;
  if (c->hidden > 16384) return fail(ENC_ERR_UNSUPPORTED, "%s: hidden must be <= 16384", fn);
  if (!(c->ln_eps >= 0.f)) return fail(ENC_ERR_INVALID, "%s: ln_eps must be >= 0", fn);
  const long M = static_cast<long>(c->batch) * c->seq;
  const long A = static_cast<long>(c->heads) * c->head_dim;
  if (M * c->mlp >= kMaxElems || M * 3 * A >= kMaxElems || M * c->hidden >= kMaxElems ||
      static_cast<long>(c->mlp) * c->hidden >= kMaxElems)
    return fail(ENC_ERR_UNSUPPORTED, "%s: a tensor exceeds 2^31 elements", fn);
  if (!attn_addressable(static_cast<uint64_t>(M), c->heads, c->head_dim))
    return fail(ENC_ERR_UNSUPPORTED, "%s: qkv exceeds the 4 GiB the attention kernels address", fn);
  return ENC_OK;
}

size_t round256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

void saved_layout(const enc_cfg_t *c, enc_saved_layout_t *L) {
  const size_t M = static_cast<size_t>(c->batch) * c->seq;
  const size_t H = c->hidden, A = static_cast<size_t>(c->heads) * c->head_dim, F = c->mlp;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += round256(bytes);
    return o;
  };
  L->y1 = take(M * H * 2);
  L->mean1 = take(M * 4);
  L->rstd1 = take(M * 4);
  L->qkv = take(M * 3 * A * 2);
  L->o = take(M * A * 2);
  L->lse = take(static_cast<size_t>(c->batch) * c->heads * c->seq * 4);
  L->h = take(M * H * 2);
  L->y2 = take(M * H * 2);
  L->mean2 = take(M * 4);
  L->rstd2 = take(M * 4);
  L->u = take(M * F * 2);
  L->g = take(M * F * 2);
  L->total = off;
}

// Backward workspace regions (offsets in bytes).
struct BwdWs {
  size_t du, dy2, dh, dO, dqkv, dy1, ln_part, dvec, wg, wg_bytes, total;
};

// Partial sums of the layer's split products (each GEMM uses the region in
// turn): the largest need of the four weight gradients, the four input
// gradients and the four forward projections.
size_t layer_gemm_ws(const enc_cfg_t *c) {
  const int M = c->batch * c->seq, H = c->hidden, A = c->heads * c->head_dim, F = c->mlp;
  const size_t wg = std::max(std::max(gemm_wgrad_ws_bytes(H, F, M), gemm_wgrad_ws_bytes(F, H, M)),
                             std::max(gemm_wgrad_ws_bytes(H, A, M), gemm_wgrad_ws_bytes(3 * A, H, M)));
  // input gradients: du [M, F] over H, dy2 [M, H] over F, dO [M, A] over H, dy1 [M, H] over 3A
  const size_t dg = std::max(std::max(gemm_ws_bytes(M, F, H), gemm_ws_bytes(M, H, F)),
                             std::max(gemm_ws_bytes(M, A, H), gemm_ws_bytes(M, H, 3 * A)));
  // forward: qkv [M, 3A] over H, h [M, H] over A, u [M, F] over H, out [M, H] over F
  const size_t fw = std::max(std::max(gemm_ws_bytes(M, 3 * A, H), gemm_ws_bytes(M, H, A)),
                             std::max(gemm_ws_bytes(M, F, H), gemm_ws_bytes(M, H, F)));
  return std::max(wg, std::max(dg, fw));
}

BwdWs bwd_layout(const enc_cfg_t *c) {
  const size_t M = static_cast<size_t>(c->batch) * c->seq;
  const size_t H = c->hidden, A = static_cast<size_t>(c->heads) * c->head_dim, F = c->mlp;
  BwdWs w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += round256(bytes);
    return o;
  };
  w.du = take(M * F * 2);
  w.dy2 = take(M * H * 2);
  w.dh = take(M * H * 2);
  w.dO = take(M * A * 2);
  w.dqkv = take(M * 3 * A * 2);
  w.dy1 = take(M * H * 2);
  w.ln_part = take(ln_bwd_ws_bytes(static_cast<int>(M), c->hidden));
  w.dvec = take(attn_bwd_ws_bytes(c->batch, c->seq, c->heads));
  w.wg_bytes = layer_gemm_ws(c);
  w.wg = take(w.wg_bytes);
  w.total = off;
  return w;
}

template <class T>
T *at(void *base, size_t off) {
  return reinterpret_cast<T *>(static_cast<char *>(base) + off);
}
template <class T>
const T *at(const void *base, size_t off) {
  return reinterpret_cast<const T *>(static_cast<const char *>(base) + off);
}

int check_params(const char *fn, const enc_params_t *p) {
  if (!p) return fail(ENC_ERR_INVALID, "%s: params is NULL", fn);
  PtrCheck c(fn);
  c.req(p->ln1_g, "ln1_g").req(p->ln1_b, "ln1_b").req(p->w_qkv, "w_qkv").req(p->b_qkv, "b_qkv");
  c.req(p->w_o, "w_o").req(p->b_o, "b_o").req(p->ln2_g, "ln2_g").req(p->ln2_b, "ln2_b");
  c.req(p->w_1, "w_1").req(p->b_1, "b_1").req(p->w_2, "w_2").req(p->b_2, "b_2");
  return c.code;
}

int check_grads(const char *fn, const enc_grads_t *g) {
  if (!g) return fail(ENC_ERR_INVALID, "%s: grads is NULL", fn);
  PtrCheck c(fn);
  c.req(g->ln1_g, "dln1_g").req(g->ln1_b, "dln1_b").req(g->w_qkv, "dw_qkv").req(g->b_qkv, "db_qkv");
  c.req(g->w_o, "dw_o").req(g->b_o, "db_o").req(g->ln2_g, "dln2_g").req(g->ln2_b, "dln2_b");
  c.req(g->w_1, "dw_1").req(g->b_1, "db_1").req(g->w_2, "dw_2").req(g->b_2, "db_2");
  return c.code;
}

// ---- unchecked launch helpers shared by the per-kernel entry points and the chains

bool gemm_fwd(int M, int N, int K, const bf16_t *X, const bf16_t *W, const bf16_t *bias, const bf16_t *R, bf16_t *Y,
              bf16_t *Y2, Epi epi, void *ws, size_t ws_bytes, hipStream_t s) {
  GemmArgs a{};
  a.M = M, a.N = N, a.K = K;
  a.A = X, a.lda = K, a.B = W, a.ldb = K;
  a.Y = Y, a.ldy = N, a.bias = bias, a.R = R, a.Y2 = Y2;
  return launch_gemm_fwd(a, epi, ws, ws_bytes, s);
}

// dX[M, K] = dY[M, N] * W[N, K]  (optionally times GELU'(U[M, K]))
bool gemm_dgrad(int M, int N, int K, const bf16_t *dY, const bf16_t *W, const bf16_t *U, bf16_t *dX, void *ws,
                size_t ws_bytes, hipStream_t s) {
  GemmArgs a{};
  a.M = M, a.N = K, a.K = N;
  a.A = dY, a.lda = N, a.B = W, a.ldb = K;
  a.Y = dX, a.ldy = K, a.R = U;
  return launch_gemm_dgrad(a, U ? Epi::kGeluGrad : Epi::kPlain, ws, ws_bytes, s);
}

// dX[M, K] = dY[M, N] * W[N, K] + R[M, K]
bool gemm_dgrad_add(int M, int N, int K, const bf16_t *dY, const bf16_t *W, const bf16_t *R, bf16_t *dX, void *ws,
                    size_t ws_bytes, hipStream_t s) {
  GemmArgs a{};
  a.M = M, a.N = K, a.K = N;
  a.A = dY, a.lda = N, a.B = W, a.ldb = K;
  a.Y = dX, a.ldy = K, a.R = R;
  return launch_gemm_dgrad(a, Epi::kResid, ws, ws_bytes, s);
}

// dW[N, K] (+)= dY[M, N]^T X[M, K]; db[N] (+)= sum_m dY
bool gemm_wgrad(int M, int N, int K, const bf16_t *dY, const bf16_t *X, float *dW, float *db, int acc, void *ws,
                size_t ws_bytes, hipStream_t s) {
  GemmArgs a{};
  a.M = N, a.N = K, a.K = M;
  a.A = dY, a.lda = N, a.B = X, a.ldb = K;
  a.Wf = dW, a.ldy = K, a.db = db, a.accumulate = acc;
  return launch_gemm_wgrad(a, ws, ws_bytes, s);
}

int linear_dims(const char *fn, int M, std::initializer_list<int> feats) {
  int r = check_dims(fn, {M});
  if (r) return r;
  for (int f : feats)
    if (f <= 0) return fail(ENC_ERR_INVALID, "%s: dimensions must be positive", fn);
  for (int f : feats)
    if (f % 8) return fail(ENC_ERR_UNSUPPORTED, "%s: feature widths must be multiples of 8 (got %d)", fn, f);
  for (int f : feats)
    if (static_cast<long>(M) * f >= kMaxElems) return fail(ENC_ERR_UNSUPPORTED, "%s: tensor exceeds 2^31 elements", fn);
  return ENC_OK;
}

// An optional product workspace: NULL, or 16-byte aligned and at least the
// size query's bytes for output [M, N] and contraction K.
int check_gemm_ws(const char *fn, const void *ws, size_t ws_bytes, int M, int N, int K) {
  if (!ws) return ENC_OK;
  if (!aligned16(ws)) return fail(ENC_ERR_ALIGN, "%s: ws is not 16-byte aligned", fn);
  const size_t need = gemm_ws_bytes(M, N, K);
  if (ws_bytes < need) return fail(ENC_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, need);
  return ENC_OK;
}

int attn_dims(const char *fn, int B, int S, int heads, int d) {
  int r = check_dims(fn, {B, S, heads, d});
  if (r) return r;
  if (d != 64 && d != 80 && d != 128) return fail(ENC_ERR_UNSUPPORTED, "%s: head_dim must be 64, 80 or 128", fn);
  if (static_cast<long>(B) * S * 3 * heads * d >= kMaxElems)
    return fail(ENC_ERR_UNSUPPORTED, "%s: tensor exceeds 2^31 elements", fn);
  if (!attn_addressable(static_cast<uint64_t>(B) * S, heads, d))
    return fail(ENC_ERR_UNSUPPORTED, "%s: qkv exceeds the 4 GiB the attention kernels address", fn);
  return ENC_OK;
}

int qk_dims(const char *fn, int M, int heads, int d) {
  int r = check_dims(fn, {M, heads, d});
  if (r) return r;
  if (d != 64 && d != 80 && d != 128) return fail(ENC_ERR_UNSUPPORTED, "%s: head_dim must be 64, 80 or 128", fn);
  if (static_cast<long>(M) * 3 * heads * d >= kMaxElems)
    return fail(ENC_ERR_UNSUPPORTED, "%s: tensor exceeds 2^31 elements", fn);
  return ENC_OK;
}

void psaved_layout(const enc_cfg_t *c, enc_psaved_layout_t *L) {
  const size_t M = static_cast<size_t>(c->batch) * c->seq;
  const size_t H = c->hidden, A = static_cast<size_t>(c->heads) * c->head_dim, F = c->mlp;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += round256(bytes);
    return o;
  };
  L->y = take(M * H * 2);
  L->mean = take(M * 4);
  L->rstd = take(M * 4);
  L->qkv = take(M * 3 * A * 2);
  L->qkvn = take(M * 3 * A * 2);
  L->qkstats = take(M * c->heads * 4 * 4);
  L->o = take(M * A * 2);
  L->lse = take(static_cast<size_t>(c->batch) * c->heads * c->seq * 4);
  L->h = take(M * H * 2);
  L->u = take(M * F * 2);
  L->g = take(M * F * 2);
  L->total = off;
}

struct PBwdWs {
  size_t du, dy_mlp, dO, dqkvn, dqkv, dy, ln_part, dvec, qk_part, total;
};

PBwdWs pbwd_layout(const enc_cfg_t *c) {
  const size_t M = static_cast<size_t>(c->batch) * c->seq;
  const size_t H = c->hidden, A = static_cast<size_t>(c->heads) * c->head_dim, F = c->mlp;
  PBwdWs w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += round256(bytes);
    return o;
  };
  w.du = take(M * F * 2);
  w.dy_mlp = take(M * H * 2);
  w.dO = take(M * A * 2);
  w.dqkvn = take(M * 3 * A * 2);
  w.dqkv = take(M * 3 * A * 2);
  w.dy = take(M * H * 2);
  w.ln_part = take(ln_bwd_ws_bytes(static_cast<int>(M), c->hidden));
  w.dvec = take(attn_bwd_ws_bytes(c->batch, c->seq, c->heads));
  w.qk_part = take(qk_norm_bwd_ws_bytes(static_cast<int>(M), c->heads, c->head_dim));
  w.total = off;
  return w;
}

int check_pparams(const char *fn, const enc_pparams_t *p) {
  if (!p) return fail(ENC_ERR_INVALID, "%s: params is NULL", fn);
  PtrCheck c(fn);
  c.req(p->ln_g, "ln_g").req(p->ln_b, "ln_b").req(p->w_qkv, "w_qkv").req(p->qn_g, "qn_g").req(p->qn_b, "qn_b");
  c.req(p->kn_g, "kn_g").req(p->kn_b, "kn_b").req(p->w_o, "w_o").req(p->b_o, "b_o");
  c.req(p->w_1, "w_1").req(p->b_1, "b_1").req(p->w_2, "w_2").req(p->b_2, "b_2");
  return c.code;
}

int check_pgrads(const char *fn, const enc_pgrads_t *g) {
  if (!g) return fail(ENC_ERR_INVALID, "%s: grads is NULL", fn);
  PtrCheck c(fn);
  c.req(g->ln_g, "dln_g").req(g->ln_b, "dln_b").req(g->w_qkv, "dw_qkv").req(g->qn_g, "dqn_g").req(g->qn_b, "dqn_b");
  c.req(g->kn_g, "dkn_g").req(g->kn_b, "dkn_b").req(g->w_o, "dw_o").req(g->b_o, "db_o");
  c.req(g->w_1, "dw_1").req(g->b_1, "db_1").req(g->w_2, "dw_2").req(g->b_2, "db_2");
  return c.code;
}

int patch_dims(const char *fn, int B, int C, int ih, int iw, int p, int H, int has_cls, int *N, int *S, int *Kp) {
  int r = check_dims(fn, {B, C, ih, iw, p, H});
  if (r) return r;
  if (has_cls != 0 && has_cls != 1) return fail(ENC_ERR_INVALID, "%s: has_cls must be 0 or 1", fn);
  if (ih % p || iw % p) return fail(ENC_ERR_UNSUPPORTED, "%s: image sides must be multiples of the patch", fn);
  if (H % 8) return fail(ENC_ERR_UNSUPPORTED, "%s: hidden must be a multiple of 8", fn);
  *N = (ih / p) * (iw / p);
  *S = *N + has_cls;
  *Kp = (C * p * p + 7) / 8 * 8;
  const long M = static_cast<long>(B) * *N;
  if (M * *Kp >= kMaxElems || static_cast<long>(B) * *S * H >= kMaxElems ||
      static_cast<long>(B) * C * ih * iw >= kMaxElems)
    return fail(ENC_ERR_UNSUPPORTED, "%s: tensor exceeds 2^31 elements", fn);
  return ENC_OK;
}

struct StackLayout {
  size_t x_step, layer_step, layers_off, mean, rstd, total;
};

StackLayout stack_layout(const enc_cfg_t *c, int layers) {
  const size_t M = static_cast<size_t>(c->batch) * c->seq;
  enc_saved_layout_t L;
  saved_layout(c, &L);
  StackLayout s{};
  s.x_step = round256(M * c->hidden * 2);
  s.layer_step = L.total;
  s.layers_off = s.x_step * layers;
  s.mean = s.layers_off + s.layer_step * layers;
  s.rstd = s.mean + round256(M * 4);
  s.total = s.rstd + round256(M * 4);
  return s;
}

struct StackWs {
  size_t layer, dx_a, dx_b, ln_part, total;
};

StackWs stack_ws(const enc_cfg_t *c) {
  const size_t M = static_cast<size_t>(c->batch) * c->seq;
  StackWs w{};
  w.layer = 0;
  w.dx_a = round256(bwd_layout(c).total);
  w.dx_b = w.dx_a + round256(M * c->hidden * 2);
  w.ln_part = w.dx_b + round256(M * c->hidden * 2);
  w.total = w.ln_part + round256(ln_bwd_ws_bytes(static_cast<int>(M), c->hidden));
  return w;
}

}  // namespace

extern "C" {

const char *enc_status_string(int status) {
  switch (status) {
    case ENC_OK: return "ok";
    case ENC_ERR_INVALID: return "invalid argument (null pointer or non-positive dimension)";
    case ENC_ERR_UNSUPPORTED: return "unsupported shape";
    case ENC_ERR_ALIGN: return "pointer not 16-byte aligned";
    case ENC_ERR_LAUNCH: return "kernel launch failed";
    case ENC_ERR_WORKSPACE: return "workspace too small";
    default: return "unknown status";
  }
}

const char *enc_last_error(void) { return g_last_error.c_str(); }

int enc_abi_version(void) { return 2; }

int enc_saved_layout(const enc_cfg_t *cfg, enc_saved_layout_t *layout) {
  int r = check_cfg("enc_saved_layout", cfg);
  if (r) return r;
  if (!layout) return fail(ENC_ERR_INVALID, "enc_saved_layout: layout is NULL");
  saved_layout(cfg, layout);
  return ok();
}

int enc_layer_workspace_bytes(const enc_cfg_t *cfg, size_t *bytes) {
  int r = check_cfg("enc_layer_workspace_bytes", cfg);
  if (r) return r;
  if (!bytes) return fail(ENC_ERR_INVALID, "enc_layer_workspace_bytes: bytes is NULL");
  *bytes = bwd_layout(cfg).total;
  return ok();
}

int enc_ln_bwd_workspace_bytes(int rows, int cols, size_t *bytes) {
  int r = check_dims("enc_ln_bwd_workspace_bytes", {rows, cols});
  if (r) return r;
  if (!bytes) return fail(ENC_ERR_INVALID, "enc_ln_bwd_workspace_bytes: bytes is NULL");
  *bytes = ln_bwd_ws_bytes(rows, cols);
  return ok();
}

int enc_attn_bwd_workspace_bytes(int batch, int seq, int heads, int head_dim, size_t *bytes) {
  int r = attn_dims("enc_attn_bwd_workspace_bytes", batch, seq, heads, head_dim);
  if (r) return r;
  if (!bytes) return fail(ENC_ERR_INVALID, "enc_attn_bwd_workspace_bytes: bytes is NULL");
  *bytes = attn_bwd_ws_bytes(batch, seq, heads);
  return ok();
}

// ------------------------------------------------------------ forward kernels

int enc_ln_fwd(int rows, int cols, const enc_bf16 *x, const enc_bf16 *gamma, const enc_bf16 *beta, float eps,
               enc_bf16 *y, float *mean, float *rstd, enc_stream_t stream) {
  const char *fn = "enc_ln_fwd";
  int r = check_dims(fn, {rows, cols});
  if (r) return r;
  if (cols % 8 || cols > 16384) return fail(ENC_ERR_UNSUPPORTED, "%s: cols must be a multiple of 8 and <= 16384", fn);
  if (static_cast<long>(rows) * cols >= kMaxElems) return fail(ENC_ERR_UNSUPPORTED, "%s: too many elements", fn);
  if (!(eps >= 0.f)) return fail(ENC_ERR_INVALID, "%s: eps must be >= 0", fn);
  PtrCheck c(fn);
  c.req(x, "x").req(gamma, "gamma").req(beta, "beta").req(y, "y").req(mean, "mean").req(rstd, "rstd");
  if (c.code) return c.code;
  if (!launch_ln_fwd(rows, cols, x, gamma, beta, eps, y, mean, rstd, as_stream(stream)))
    return refused_after_checks(fn);
  return launched(fn);
}

int enc_qkv_fwd(int M, int H, int A, const enc_bf16 *y1, const enc_bf16 *w_qkv, const enc_bf16 *b_qkv, enc_bf16 *qkv,
                void *ws, size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "enc_qkv_fwd";
  int r = linear_dims(fn, M, {H, A, 3 * A});
  if (r) return r;
  PtrCheck c(fn);
  c.req(y1, "y1").req(w_qkv, "w_qkv").opt(b_qkv, "b_qkv").req(qkv, "qkv");
  if (c.code) return c.code;
  if ((r = check_gemm_ws(fn, ws, ws_bytes, M, 3 * A, H))) return r;
  if (!gemm_fwd(M, 3 * A, H, y1, w_qkv, b_qkv, nullptr, qkv, nullptr, b_qkv ? Epi::kBias : Epi::kPlain, ws,
                ws_bytes, as_stream(stream)))
    return refused_after_checks(fn);
  return launched(fn);
}

int enc_attn_fwd(int batch, int seq, int heads, int head_dim, const enc_bf16 *qkv, enc_bf16 *o, float *lse,
                 enc_stream_t stream) {
  const char *fn = "enc_attn_fwd";
  int r = attn_dims(fn, batch, seq, heads, head_dim);
  if (r) return r;
  PtrCheck c(fn);
  c.req(qkv, "qkv").req(o, "o").req(lse, "lse");
  if (c.code) return c.code;
  if (!launch_attn_fwd(batch, seq, heads, head_dim, qkv, o, lse, as_stream(stream)))
    return fail(ENC_ERR_UNSUPPORTED, "%s: unsupported head_dim", fn);
  return launched(fn);
}

int enc_oproj_fwd(int M, int A, int H, const enc_bf16 *o, const enc_bf16 *w_o, const enc_bf16 *b_o,
                  const enc_bf16 *resid, enc_bf16 *h, void *ws, size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "enc_oproj_fwd";
  int r = linear_dims(fn, M, {H, A});
  if (r) return r;
  PtrCheck c(fn);
  c.req(o, "o").req(w_o, "w_o").req(b_o, "b_o").req(resid, "resid").req(h, "h");
  if (c.code) return c.code;
  if ((r = check_gemm_ws(fn, ws, ws_bytes, M, H, A))) return r;
  if (!gemm_fwd(M, H, A, o, w_o, b_o, resid, h, nullptr, Epi::kBiasResid, ws, ws_bytes, as_stream(stream)))
    return refused_after_checks(fn);
  return launched(fn);
}

int enc_mlp_up_fwd(int M, int H, int F, const enc_bf16 *y2, const enc_bf16 *w_1, const enc_bf16 *b_1, enc_bf16 *u,
                   enc_bf16 *g, void *ws, size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "enc_mlp_up_fwd";
  int r = linear_dims(fn, M, {H, F});
  if (r) return r;
  PtrCheck c(fn);
  c.req(y2, "y2").req(w_1, "w_1").req(b_1, "b_1").req(u, "u").req(g, "g");
  if (c.code) return c.code;
  if ((r = check_gemm_ws(fn, ws, ws_bytes, M, F, H))) return r;
  if (!gemm_fwd(M, F, H, y2, w_1, b_1, nullptr, u, g, Epi::kBiasGelu, ws, ws_bytes, as_stream(stream)))
    return refused_after_checks(fn);
  return launched(fn);
}

int enc_mlp_down_fwd(int M, int F, int H, const enc_bf16 *g, const enc_bf16 *w_2, const enc_bf16 *b_2,
                     const enc_bf16 *resid, enc_bf16 *out, void *ws, size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "enc_mlp_down_fwd";
  int r = linear_dims(fn, M, {H, F});
  if (r) return r;
  PtrCheck c(fn);
  c.req(g, "g").req(w_2, "w_2").req(b_2, "b_2").req(resid, "resid").req(out, "out");
  if (c.code) return c.code;
  if ((r = check_gemm_ws(fn, ws, ws_bytes, M, H, F))) return r;
  if (!gemm_fwd(M, H, F, g, w_2, b_2, resid, out, nullptr, Epi::kBiasResid, ws, ws_bytes, as_stream(stream)))
    return refused_after_checks(fn);
  return launched(fn);
}

// ------------------------------------------------------------ backward kernels

int enc_mlp_down_bwd_data(int M, int F, int H, const enc_bf16 *dout, const enc_bf16 *w_2, const enc_bf16 *u,
                          enc_bf16 *du, void *ws, size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "enc_mlp_down_bwd_data";
  int r = linear_dims(fn, M, {H, F});
  if (r) return r;
  PtrCheck c(fn);
  c.req(dout, "dout").req(w_2, "w_2").req(u, "u").req(du, "du");
  if (c.code) return c.code;
  if ((r = check_gemm_ws(fn, ws, ws_bytes, M, F, H))) return r;
  if (!gemm_dgrad(M, H, F, dout, w_2, u, du, ws, ws_bytes, as_stream(stream))) return refused_after_checks(fn);
  return launched(fn);
}

int enc_mlp_up_bwd_data(int M, int H, int F, const enc_bf16 *du, const enc_bf16 *w_1, enc_bf16 *dy2, void *ws,
                        size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "enc_mlp_up_bwd_data";
  int r = linear_dims(fn, M, {H, F});
  if (r) return r;
  PtrCheck c(fn);
  c.req(du, "du").req(w_1, "w_1").req(dy2, "dy2");
  if (c.code) return c.code;
  if ((r = check_gemm_ws(fn, ws, ws_bytes, M, H, F))) return r;
  if (!gemm_dgrad(M, F, H, du, w_1, nullptr, dy2, ws, ws_bytes, as_stream(stream))) return refused_after_checks(fn);
  return launched(fn);
}

int enc_oproj_bwd_data(int M, int A, int H, const enc_bf16 *dh, const enc_bf16 *w_o, enc_bf16 *do_, void *ws,
                       size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "enc_oproj_bwd_data";
  int r = linear_dims(fn, M, {H, A});
  if (r) return r;
  PtrCheck c(fn);
  c.req(dh, "dh").req(w_o, "w_o").req(do_, "do");
  if (c.code) return c.code;
  if ((r = check_gemm_ws(fn, ws, ws_bytes, M, A, H))) return r;
  if (!gemm_dgrad(M, H, A, dh, w_o, nullptr, do_, ws, ws_bytes, as_stream(stream))) return refused_after_checks(fn);
  return launched(fn);
}

int enc_qkv_bwd_data(int M, int H, int A, const enc_bf16 *dqkv, const enc_bf16 *w_qkv, enc_bf16 *dy1, void *ws,
                     size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "enc_qkv_bwd_data";
  int r = linear_dims(fn, M, {H, A, 3 * A});
  if (r) return r;
  PtrCheck c(fn);
  c.req(dqkv, "dqkv").req(w_qkv, "w_qkv").req(dy1, "dy1");
  if (c.code) return c.code;
  if ((r = check_gemm_ws(fn, ws, ws_bytes, M, H, 3 * A))) return r;
  if (!gemm_dgrad(M, 3 * A, H, dqkv, w_qkv, nullptr, dy1, ws, ws_bytes, as_stream(stream)))
    return refused_after_checks(fn);
  return launched(fn);
}

int enc_qkv_bwd_data_add(int M, int H, int A, const enc_bf16 *dqkv, const enc_bf16 *w_qkv, const enc_bf16 *addend,
                         enc_bf16 *dy, void *ws, size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "enc_qkv_bwd_data_add";
  int r = linear_dims(fn, M, {H, A, 3 * A});
  if (r) return r;
  PtrCheck c(fn);
  c.req(dqkv, "dqkv").req(w_qkv, "w_qkv").req(addend, "addend").req(dy, "dy");
  if (c.code) return c.code;
  if ((r = check_gemm_ws(fn, ws, ws_bytes, M, H, 3 * A))) return r;
  if (!gemm_dgrad_add(M, 3 * A, H, dqkv, w_qkv, addend, dy, ws, ws_bytes, as_stream(stream)))
    return refused_after_checks(fn);
  return launched(fn);
}

int enc_linear_workspace_bytes(int M, int N, int K, size_t *bytes) {
  const char *fn = "enc_linear_workspace_bytes";
  int r = linear_dims(fn, M, {N, K});
  if (r) return r;
  if (!bytes) return fail(ENC_ERR_INVALID, "%s: bytes is NULL", fn);
  *bytes = gemm_ws_bytes(M, N, K);
  return ok();
}

int enc_linear_bwd_weight_workspace_bytes(int M, int N, int K, size_t *bytes) {
  const char *fn = "enc_linear_bwd_weight_workspace_bytes";
  int r = linear_dims(fn, M, {N, K});
  if (r) return r;
  if (static_cast<long>(N) * K >= kMaxElems) return fail(ENC_ERR_UNSUPPORTED, "%s: dW exceeds 2^31 elements", fn);
  if (!bytes) return fail(ENC_ERR_INVALID, "%s: bytes is NULL", fn);
  *bytes = gemm_wgrad_ws_bytes(N, K, M);
  return ok();
}

int enc_linear_plan(int layout, int M, int N, int K, int *tile_rows, int *tile_cols, int *splits) {
  const char *fn = "enc_linear_plan";
  if (layout != ENC_LAYOUT_FWD && layout != ENC_LAYOUT_DGRAD && layout != ENC_LAYOUT_WGRAD)
    return fail(ENC_ERR_INVALID, "%s: unknown layout %d", fn, layout);
  int r = linear_dims(fn, M, {N, K});
  if (r) return r;
  if (layout == ENC_LAYOUT_WGRAD && static_cast<long>(N) * K >= kMaxElems)
    return fail(ENC_ERR_UNSUPPORTED, "%s: dW exceeds 2^31 elements", fn);
  if (!tile_rows || !tile_cols || !splits) return fail(ENC_ERR_INVALID, "%s: an output pointer is NULL", fn);
  // the GemmArgs geometry the launch helpers above build for each layout
  GemmArgs a{};
  bool AT = false, BT = false;
  if (layout == ENC_LAYOUT_FWD) {
    a.M = M, a.N = N, a.K = K, a.lda = K, a.ldb = K;
  } else if (layout == ENC_LAYOUT_DGRAD) {
    a.M = M, a.N = N, a.K = K, a.lda = K, a.ldb = N;
    BT = true;
  } else {
    a.M = N, a.N = K, a.K = M, a.lda = N, a.ldb = K;
    AT = BT = true;
  }
  const GemmPlan pl = gemm_plan(a.M, a.N, a.K, a.lda, a.ldb, AT, BT);
  *tile_rows = pl.tile.bm;
  *tile_cols = pl.tile.bn;
  *splits = pl.splits;
  return ok();
}

int enc_linear_bwd_weight(int M, int N, int K, const enc_bf16 *dY, const enc_bf16 *X, float *dW, float *db,
                          int accumulate, void *ws, size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "enc_linear_bwd_weight";
  int r = linear_dims(fn, M, {N, K});
  if (r) return r;
  if (static_cast<long>(N) * K >= kMaxElems) return fail(ENC_ERR_UNSUPPORTED, "%s: dW exceeds 2^31 elements", fn);
  PtrCheck c(fn);
  c.req(dY, "dY").req(X, "X").req(dW, "dW").opt(db, "db").opt(ws, "ws");
  if (c.code) return c.code;
  const size_t need = gemm_wgrad_ws_bytes(N, K, M);
  if (ws && ws_bytes < need) return fail(ENC_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, need);
  if (!gemm_wgrad(M, N, K, dY, X, dW, db, accumulate ? 1 : 0, ws, ws_bytes, as_stream(stream)))
    return refused_after_checks(fn);
  return launched(fn);
}

int enc_mlp_down_bwd_weight(int M, int F, int H, const enc_bf16 *dout, const enc_bf16 *g, float *dw_2, float *db_2,
                            int accumulate, void *ws, size_t ws_bytes, enc_stream_t stream) {
  return enc_linear_bwd_weight(M, H, F, dout, g, dw_2, db_2, accumulate, ws, ws_bytes, stream);
}

int enc_mlp_up_bwd_weight(int M, int H, int F, const enc_bf16 *du, const enc_bf16 *y2, float *dw_1, float *db_1,
                          int accumulate, void *ws, size_t ws_bytes, enc_stream_t stream) {
  return enc_linear_bwd_weight(M, F, H, du, y2, dw_1, db_1, accumulate, ws, ws_bytes, stream);
}

int enc_oproj_bwd_weight(int M, int A, int H, const enc_bf16 *dh, const enc_bf16 *o, float *dw_o, float *db_o,
                         int accumulate, void *ws, size_t ws_bytes, enc_stream_t stream) {
  return enc_linear_bwd_weight(M, H, A, dh, o, dw_o, db_o, accumulate, ws, ws_bytes, stream);
}

int enc_qkv_bwd_weight(int M, int H, int A, const enc_bf16 *dqkv, const enc_bf16 *y1, float *dw_qkv, float *db_qkv,
                       int accumulate, void *ws, size_t ws_bytes, enc_stream_t stream) {
  return enc_linear_bwd_weight(M, 3 * A, H, dqkv, y1, dw_qkv, db_qkv, accumulate, ws, ws_bytes, stream);
}

int enc_ln_bwd(int rows, int cols, const enc_bf16 *dy, const enc_bf16 *x, const float *mean, const float *rstd,
               const enc_bf16 *gamma, const enc_bf16 *dresid, enc_bf16 *dx, float *dgamma, float *dbeta,
               int accumulate, void *ws, size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "enc_ln_bwd";
  int r = check_dims(fn, {rows, cols});
  if (r) return r;
  if (cols % 8 || cols > 16384) return fail(ENC_ERR_UNSUPPORTED, "%s: cols must be a multiple of 8 and <= 16384", fn);
  if (static_cast<long>(rows) * cols >= kMaxElems) return fail(ENC_ERR_UNSUPPORTED, "%s: too many elements", fn);
  PtrCheck c(fn);
  c.req(dy, "dy").req(x, "x").req(mean, "mean").req(rstd, "rstd").req(gamma, "gamma").opt(dresid, "dresid");
  c.req(dx, "dx").req(dgamma, "dgamma").req(dbeta, "dbeta").req(ws, "ws");
  if (c.code) return c.code;
  if (ws_bytes < ln_bwd_ws_bytes(rows, cols))
    return fail(ENC_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, ln_bwd_ws_bytes(rows, cols));
  if (!launch_ln_bwd(rows, cols, dy, x, mean, rstd, gamma, dresid, dx, dgamma, dbeta, accumulate ? 1 : 0,
                     static_cast<float *>(ws), as_stream(stream)))
    return refused_after_checks(fn);
  return launched(fn);
}

int enc_attn_bwd(int batch, int seq, int heads, int head_dim, const enc_bf16 *qkv, const enc_bf16 *o, const float *lse,
                 const enc_bf16 *do_, enc_bf16 *dqkv, void *ws, size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "enc_attn_bwd";
  int r = attn_dims(fn, batch, seq, heads, head_dim);
  if (r) return r;
  PtrCheck c(fn);
  c.req(qkv, "qkv").req(o, "o").req(lse, "lse").req(do_, "do").req(dqkv, "dqkv").req(ws, "ws");
  if (c.code) return c.code;
  const size_t need = attn_bwd_ws_bytes(batch, seq, heads);
  if (ws_bytes < need) return fail(ENC_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, need);
  if (!launch_attn_bwd(batch, seq, heads, head_dim, qkv, o, lse, do_, dqkv, static_cast<float *>(ws),
                       as_stream(stream)))
    return fail(ENC_ERR_UNSUPPORTED, "%s: unsupported head_dim", fn);
  return launched(fn);
}

int enc_attn_bwd_noalloc(int batch, int seq, int heads, int head_dim, const enc_bf16 *qkv, const enc_bf16 *o,
                         const float *lse, const enc_bf16 *do_, enc_bf16 *dqkv, enc_stream_t stream) {
  const char *fn = "enc_attn_bwd_noalloc";
  int r = attn_dims(fn, batch, seq, heads, head_dim);
  if (r) return r;
  PtrCheck c(fn);
  c.req(qkv, "qkv").req(o, "o").req(lse, "lse").req(do_, "do").req(dqkv, "dqkv");
  if (c.code) return c.code;
  const size_t need = attn_bwd_ws_bytes(batch, seq, heads), have = kAttnScratchFloats * sizeof(float);
  if (need > have)
    return fail(ENC_ERR_UNSUPPORTED, "%s: batch*heads*seq = %zu exceeds the static scratch's %zu rows (%zu bytes)", fn,
                need / sizeof(float), kAttnScratchFloats, have);
  float *dvec = nullptr;
  const hipError_t e = attn_bwd_scratch(&dvec);
  if (e != hipSuccess)
    return fail(ENC_ERR_LAUNCH, "%s: looking up the static scratch failed: %s", fn, hipGetErrorString(e));
  if (!launch_attn_bwd(batch, seq, heads, head_dim, qkv, o, lse, do_, dqkv, dvec, as_stream(stream)))
    return refused_after_checks(fn);
  return launched(fn);
}

// ------------------------------------------------------------ composites

int encoder_layer_fwd(const enc_cfg_t *cfg, const enc_params_t *params, const enc_bf16 *x, enc_bf16 *out, void *saved,
                      void *ws, size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "encoder_layer_fwd";
  int r = check_cfg(fn, cfg);
  if (r) return r;
  if ((r = check_params(fn, params))) return r;
  PtrCheck c(fn);
  c.req(x, "x").req(out, "out").req(saved, "saved").opt(ws, "ws");
  if (c.code) return c.code;
  // the workspace only holds split-product partials here (ws = NULL: no split)
  const size_t gneed = layer_gemm_ws(cfg);
  if (ws && ws_bytes < gneed) return fail(ENC_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, gneed);
  void *gp = ws && gneed ? ws : nullptr;
  enc_saved_layout_t L;
  saved_layout(cfg, &L);
  const int M = cfg->batch * cfg->seq, H = cfg->hidden, F = cfg->mlp, A = cfg->heads * cfg->head_dim;
  const hipStream_t s = as_stream(stream);
  const enc_params_t &p = *params;
  bf16_t *y1 = at<bf16_t>(saved, L.y1), *qkv = at<bf16_t>(saved, L.qkv), *o = at<bf16_t>(saved, L.o);
  bf16_t *h = at<bf16_t>(saved, L.h), *y2 = at<bf16_t>(saved, L.y2), *u = at<bf16_t>(saved, L.u);
  bf16_t *g = at<bf16_t>(saved, L.g);
  float *mean1 = at<float>(saved, L.mean1), *rstd1 = at<float>(saved, L.rstd1), *lse = at<float>(saved, L.lse);
  float *mean2 = at<float>(saved, L.mean2), *rstd2 = at<float>(saved, L.rstd2);

  bool okk = launch_ln_fwd(M, H, x, p.ln1_g, p.ln1_b, cfg->ln_eps, y1, mean1, rstd1, s);
  okk = okk && gemm_fwd(M, 3 * A, H, y1, p.w_qkv, p.b_qkv, nullptr, qkv, nullptr, Epi::kBias, gp, gneed, s);
  okk = okk && launch_attn_fwd(cfg->batch, cfg->seq, cfg->heads, cfg->head_dim, qkv, o, lse, s);
  okk = okk && gemm_fwd(M, H, A, o, p.w_o, p.b_o, x, h, nullptr, Epi::kBiasResid, gp, gneed, s);
  okk = okk && launch_ln_fwd(M, H, h, p.ln2_g, p.ln2_b, cfg->ln_eps, y2, mean2, rstd2, s);
  okk = okk && gemm_fwd(M, F, H, y2, p.w_1, p.b_1, nullptr, u, g, Epi::kBiasGelu, gp, gneed, s);
  okk = okk && gemm_fwd(M, H, F, g, p.w_2, p.b_2, h, out, nullptr, Epi::kBiasResid, gp, gneed, s);
  if (!okk) return refused_after_checks(fn);
  return launched(fn);
}

int encoder_layer_bwd(const enc_cfg_t *cfg, const enc_params_t *params, const enc_bf16 *x, const void *saved,
                      const enc_bf16 *dout, enc_bf16 *dx, const enc_grads_t *grads, int accumulate, void *ws,
                      size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "encoder_layer_bwd";
  int r = check_cfg(fn, cfg);
  if (r) return r;
  if ((r = check_params(fn, params))) return r;
  if ((r = check_grads(fn, grads))) return r;
  PtrCheck c(fn);
  c.req(x, "x").req(saved, "saved").req(dout, "dout").req(dx, "dx").req(ws, "ws");
  if (c.code) return c.code;
  const BwdWs W = bwd_layout(cfg);
  if (ws_bytes < W.total) return fail(ENC_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, W.total);
  enc_saved_layout_t L;
  saved_layout(cfg, &L);
  const int M = cfg->batch * cfg->seq, H = cfg->hidden, F = cfg->mlp, A = cfg->heads * cfg->head_dim;
  const int acc = accumulate ? 1 : 0;
  const hipStream_t s = as_stream(stream);
  const enc_params_t &p = *params;
  const enc_grads_t &gr = *grads;
  const bf16_t *y1 = at<bf16_t>(saved, L.y1), *qkv = at<bf16_t>(saved, L.qkv), *o = at<bf16_t>(saved, L.o);
  const bf16_t *h = at<bf16_t>(saved, L.h), *y2 = at<bf16_t>(saved, L.y2), *u = at<bf16_t>(saved, L.u);
  const bf16_t *g = at<bf16_t>(saved, L.g);
  const float *mean1 = at<float>(saved, L.mean1), *rstd1 = at<float>(saved, L.rstd1), *lse = at<float>(saved, L.lse);
  const float *mean2 = at<float>(saved, L.mean2), *rstd2 = at<float>(saved, L.rstd2);
  bf16_t *du = at<bf16_t>(ws, W.du), *dy2 = at<bf16_t>(ws, W.dy2), *dh = at<bf16_t>(ws, W.dh);
  bf16_t *dO = at<bf16_t>(ws, W.dO), *dqkv = at<bf16_t>(ws, W.dqkv), *dy1 = at<bf16_t>(ws, W.dy1);
  float *part = at<float>(ws, W.ln_part), *dvec = at<float>(ws, W.dvec);
  void *wg = W.wg_bytes ? at<char>(ws, W.wg) : nullptr;  // split weight-gradient partials

  bool okk = gemm_dgrad(M, H, F, dout, p.w_2, u, du, wg, W.wg_bytes, s);      // du = dout W2 * GELU'(u)
  okk = okk && gemm_wgrad(M, H, F, dout, g, gr.w_2, gr.b_2, acc, wg, W.wg_bytes, s);          // dW2, db2
  okk = okk && gemm_dgrad(M, F, H, du, p.w_1, nullptr, dy2, wg, W.wg_bytes, s);  // dy2 = du W1
  okk = okk && gemm_wgrad(M, F, H, du, y2, gr.w_1, gr.b_1, acc, wg, W.wg_bytes, s);           // dW1, db1
  okk = okk && launch_ln_bwd(M, H, dy2, h, mean2, rstd2, p.ln2_g, dout, dh, gr.ln2_g, gr.ln2_b, acc, part, s);
  okk = okk && gemm_dgrad(M, H, A, dh, p.w_o, nullptr, dO, wg, W.wg_bytes, s);   // dO = dh Wo
  okk = okk && gemm_wgrad(M, H, A, dh, o, gr.w_o, gr.b_o, acc, wg, W.wg_bytes, s);            // dWo, dbo
  okk = okk && launch_attn_bwd(cfg->batch, cfg->seq, cfg->heads, cfg->head_dim, qkv, o, lse, dO, dqkv, dvec, s);
  okk = okk && gemm_dgrad(M, 3 * A, H, dqkv, p.w_qkv, nullptr, dy1, wg, W.wg_bytes, s);  // dy1 = dqkv Wqkv
  okk = okk && gemm_wgrad(M, 3 * A, H, dqkv, y1, gr.w_qkv, gr.b_qkv, acc, wg, W.wg_bytes, s);  // dWqkv, dbqkv
  okk = okk && launch_ln_bwd(M, H, dy1, x, mean1, rstd1, p.ln1_g, dh, dx, gr.ln1_g, gr.ln1_b, acc, part, s);
  if (!okk) return refused_after_checks(fn);
  return launched(fn);
}

// ------------------------------------------------------------ ViT-22B-style parallel block

int enc_qk_norm_fwd(int M, int heads, int head_dim, const enc_bf16 *qkv, const enc_bf16 *qn_g, const enc_bf16 *qn_b,
                    const enc_bf16 *kn_g, const enc_bf16 *kn_b, float eps, enc_bf16 *qkvn, float *stats,
                    enc_stream_t stream) {
  const char *fn = "enc_qk_norm_fwd";
  int r = qk_dims(fn, M, heads, head_dim);
  if (r) return r;
  if (!(eps >= 0.f)) return fail(ENC_ERR_INVALID, "%s: eps must be >= 0", fn);
  PtrCheck c(fn);
  c.req(qkv, "qkv").req(qn_g, "qn_g").req(qn_b, "qn_b").req(kn_g, "kn_g").req(kn_b, "kn_b");
  c.req(qkvn, "qkvn").req(stats, "stats");
  if (c.code) return c.code;
  launch_qk_norm_fwd(M, heads, head_dim, qkv, qn_g, qn_b, kn_g, kn_b, eps, qkvn, stats, as_stream(stream));
  return launched(fn);
}

int enc_qk_norm_bwd_workspace_bytes(int M, int heads, int head_dim, size_t *bytes) {
  const char *fn = "enc_qk_norm_bwd_workspace_bytes";
  int r = qk_dims(fn, M, heads, head_dim);
  if (r) return r;
  if (!bytes) return fail(ENC_ERR_INVALID, "%s: bytes is NULL", fn);
  *bytes = qk_norm_bwd_ws_bytes(M, heads, head_dim);
  return ok();
}

int enc_qk_norm_bwd(int M, int heads, int head_dim, const enc_bf16 *dqkvn, const enc_bf16 *qkv, const float *stats,
                    const enc_bf16 *qn_g, const enc_bf16 *kn_g, enc_bf16 *dqkv, float *dqn_g, float *dqn_b,
                    float *dkn_g, float *dkn_b, int accumulate, void *ws, size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "enc_qk_norm_bwd";
  int r = qk_dims(fn, M, heads, head_dim);
  if (r) return r;
  PtrCheck c(fn);
  c.req(dqkvn, "dqkvn").req(qkv, "qkv").req(stats, "stats").req(qn_g, "qn_g").req(kn_g, "kn_g");
  c.req(dqkv, "dqkv").req(dqn_g, "dqn_g").req(dqn_b, "dqn_b").req(dkn_g, "dkn_g").req(dkn_b, "dkn_b").req(ws, "ws");
  if (c.code) return c.code;
  const size_t need = qk_norm_bwd_ws_bytes(M, heads, head_dim);
  if (ws_bytes < need) return fail(ENC_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, need);
  launch_qk_norm_bwd(M, heads, head_dim, dqkvn, qkv, stats, qn_g, kn_g, dqkv, dqn_g, dqn_b, dkn_g, dkn_b,
                     accumulate ? 1 : 0, static_cast<float *>(ws), as_stream(stream));
  return launched(fn);
}

int enc_parallel_saved_layout(const enc_cfg_t *cfg, enc_psaved_layout_t *layout) {
  const char *fn = "enc_parallel_saved_layout";
  int r = check_cfg(fn, cfg);
  if (r) return r;
  if (!layout) return fail(ENC_ERR_INVALID, "%s: layout is NULL", fn);
  psaved_layout(cfg, layout);
  return ok();
}

int enc_parallel_workspace_bytes(const enc_cfg_t *cfg, size_t *bytes) {
  const char *fn = "enc_parallel_workspace_bytes";
  int r = check_cfg(fn, cfg);
  if (r) return r;
  if (!bytes) return fail(ENC_ERR_INVALID, "%s: bytes is NULL", fn);
  *bytes = pbwd_layout(cfg).total;
  return ok();
}

int encoder_parallel_fwd(const enc_cfg_t *cfg, const enc_pparams_t *params, const enc_bf16 *x, enc_bf16 *out,
                         void *saved, enc_stream_t stream) {
  const char *fn = "encoder_parallel_fwd";
  int r = check_cfg(fn, cfg);
  if (r) return r;
  if ((r = check_pparams(fn, params))) return r;
  PtrCheck c(fn);
  c.req(x, "x").req(out, "out").req(saved, "saved");
  if (c.code) return c.code;
  enc_psaved_layout_t L;
  psaved_layout(cfg, &L);
  const int M = cfg->batch * cfg->seq, H = cfg->hidden, F = cfg->mlp, A = cfg->heads * cfg->head_dim;
  const hipStream_t s = as_stream(stream);
  const enc_pparams_t &p = *params;
  bf16_t *y = at<bf16_t>(saved, L.y), *qkv = at<bf16_t>(saved, L.qkv), *qkvn = at<bf16_t>(saved, L.qkvn);
  bf16_t *o = at<bf16_t>(saved, L.o), *h = at<bf16_t>(saved, L.h), *u = at<bf16_t>(saved, L.u);
  bf16_t *g = at<bf16_t>(saved, L.g);
  float *mean = at<float>(saved, L.mean), *rstd = at<float>(saved, L.rstd), *lse = at<float>(saved, L.lse);
  float *qks = at<float>(saved, L.qkstats);

  bool okk = launch_ln_fwd(M, H, x, p.ln_g, p.ln_b, cfg->ln_eps, y, mean, rstd, s);
  okk = okk && gemm_fwd(M, 3 * A, H, y, p.w_qkv, nullptr, nullptr, qkv, nullptr, Epi::kPlain, nullptr, 0, s);
  okk = okk && launch_qk_norm_fwd(M, cfg->heads, cfg->head_dim, qkv, p.qn_g, p.qn_b, p.kn_g, p.kn_b, cfg->ln_eps,
                                  qkvn, qks, s);
  okk = okk && launch_attn_fwd(cfg->batch, cfg->seq, cfg->heads, cfg->head_dim, qkvn, o, lse, s);
  okk = okk && gemm_fwd(M, H, A, o, p.w_o, p.b_o, x, h, nullptr, Epi::kBiasResid, nullptr, 0, s);  // + attention
  okk = okk && gemm_fwd(M, F, H, y, p.w_1, p.b_1, nullptr, u, g, Epi::kBiasGelu, nullptr, 0, s);  // MLP reads y
  okk = okk && gemm_fwd(M, H, F, g, p.w_2, p.b_2, h, out, nullptr, Epi::kBiasResid, nullptr, 0, s);  // + MLP
  if (!okk) return refused_after_checks(fn);
  return launched(fn);
}

int encoder_parallel_bwd(const enc_cfg_t *cfg, const enc_pparams_t *params, const enc_bf16 *x, const void *saved,
                         const enc_bf16 *dout, enc_bf16 *dx, const enc_pgrads_t *grads, int accumulate, void *ws,
                         size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "encoder_parallel_bwd";
  int r = check_cfg(fn, cfg);
  if (r) return r;
  if ((r = check_pparams(fn, params))) return r;
  if ((r = check_pgrads(fn, grads))) return r;
  PtrCheck c(fn);
  c.req(x, "x").req(saved, "saved").req(dout, "dout").req(dx, "dx").req(ws, "ws");
  if (c.code) return c.code;
  const PBwdWs W = pbwd_layout(cfg);
  if (ws_bytes < W.total) return fail(ENC_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, W.total);
  enc_psaved_layout_t L;
  psaved_layout(cfg, &L);
  const int M = cfg->batch * cfg->seq, H = cfg->hidden, F = cfg->mlp, A = cfg->heads * cfg->head_dim;
  const int acc = accumulate ? 1 : 0;
  const hipStream_t s = as_stream(stream);
  const enc_pparams_t &p = *params;
  const enc_pgrads_t &gr = *grads;
  const bf16_t *y = at<bf16_t>(saved, L.y), *qkv = at<bf16_t>(saved, L.qkv), *qkvn = at<bf16_t>(saved, L.qkvn);
  const bf16_t *o = at<bf16_t>(saved, L.o), *u = at<bf16_t>(saved, L.u), *g = at<bf16_t>(saved, L.g);
  const float *mean = at<float>(saved, L.mean), *rstd = at<float>(saved, L.rstd), *lse = at<float>(saved, L.lse);
  const float *qks = at<float>(saved, L.qkstats);
  bf16_t *du = at<bf16_t>(ws, W.du), *dy_mlp = at<bf16_t>(ws, W.dy_mlp), *dO = at<bf16_t>(ws, W.dO);
  bf16_t *dqkvn = at<bf16_t>(ws, W.dqkvn), *dqkv = at<bf16_t>(ws, W.dqkv), *dy = at<bf16_t>(ws, W.dy);
  float *ln_part = at<float>(ws, W.ln_part), *dvec = at<float>(ws, W.dvec), *qk_part = at<float>(ws, W.qk_part);

  bool okk = gemm_dgrad(M, H, F, dout, p.w_2, u, du, nullptr, 0, s);      // du = dout W2 * GELU'(u)
  okk = okk && gemm_wgrad(M, H, F, dout, g, gr.w_2, gr.b_2, acc, nullptr, 0, s);      // dW2, db2
  okk = okk && gemm_dgrad(M, F, H, du, p.w_1, nullptr, dy_mlp, nullptr, 0, s);  // MLP branch's dy
  okk = okk && gemm_wgrad(M, F, H, du, y, gr.w_1, gr.b_1, acc, nullptr, 0, s);        // dW1, db1
  okk = okk && gemm_dgrad(M, H, A, dout, p.w_o, nullptr, dO, nullptr, 0, s);  // dO = dout Wo
  okk = okk && gemm_wgrad(M, H, A, dout, o, gr.w_o, gr.b_o, acc, nullptr, 0, s);      // dWo, dbo
  okk = okk && launch_attn_bwd(cfg->batch, cfg->seq, cfg->heads, cfg->head_dim, qkvn, o, lse, dO, dqkvn, dvec, s);
  okk = okk && launch_qk_norm_bwd(M, cfg->heads, cfg->head_dim, dqkvn, qkv, qks, p.qn_g, p.kn_g, dqkv, gr.qn_g,
                                  gr.qn_b, gr.kn_g, gr.kn_b, acc, qk_part, s);
  okk = okk && gemm_wgrad(M, 3 * A, H, dqkv, y, gr.w_qkv, nullptr, acc, nullptr, 0, s);  // dWqkv (no bias)
  okk = okk && gemm_dgrad_add(M, 3 * A, H, dqkv, p.w_qkv, dy_mlp, dy, nullptr, 0, s);  // + dy_mlp
  okk = okk && launch_ln_bwd(M, H, dy, x, mean, rstd, p.ln_g, dout, dx, gr.ln_g, gr.ln_b, acc, ln_part, s);
  if (!okk) return refused_after_checks(fn);
  return launched(fn);
}

// ------------------------------------------------------------ patch embedding and layer stack

int enc_patch_embed_workspace_bytes(int batch, int channels, int img_h, int img_w, int patch, int hidden, int has_cls,
                                    size_t *bytes) {
  const char *fn = "enc_patch_embed_workspace_bytes";
  int N, S, Kp;
  int r = patch_dims(fn, batch, channels, img_h, img_w, patch, hidden, has_cls, &N, &S, &Kp);
  if (r) return r;
  if (!bytes) return fail(ENC_ERR_INVALID, "%s: bytes is NULL", fn);
  *bytes = has_cls ? static_cast<size_t>(batch) * N * hidden * 2 : 0;
  return ok();
}

int enc_patch_embed_fwd(int batch, int channels, int img_h, int img_w, int patch, int hidden, int has_cls,
                        const enc_bf16 *images, const enc_bf16 *w_pe, const enc_bf16 *b_pe, const enc_bf16 *cls,
                        const enc_bf16 *pos, enc_bf16 *patches, enc_bf16 *x0, void *ws, size_t ws_bytes,
                        enc_stream_t stream) {
  const char *fn = "enc_patch_embed_fwd";
  int N, S, Kp;
  int r = patch_dims(fn, batch, channels, img_h, img_w, patch, hidden, has_cls, &N, &S, &Kp);
  if (r) return r;
  PtrCheck c(fn);
  c.req(images, "images").req(w_pe, "w_pe").req(b_pe, "b_pe").req(pos, "pos").req(patches, "patches").req(x0, "x0");
  if (has_cls) c.req(cls, "cls").req(ws, "ws");
  if (c.code) return c.code;
  const size_t need = has_cls ? static_cast<size_t>(batch) * N * hidden * 2 : 0;
  if (ws_bytes < need) return fail(ENC_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, need);
  const hipStream_t s = as_stream(stream);
  bf16_t *tok = has_cls ? static_cast<bf16_t *>(ws) : x0;  // without a class token the tokens are x0's rows
  bool okk = launch_patchify(batch, channels, img_h, img_w, patch, Kp, images, patches, s);
  okk = okk && gemm_fwd(batch * N, hidden, Kp, patches, w_pe, b_pe, nullptr, tok, nullptr, Epi::kBias, nullptr, 0,
                        s);
  okk = okk && launch_patch_assemble(batch, N, S, hidden, has_cls, tok, cls, pos, x0, s);
  if (!okk) return refused_after_checks(fn);
  return launched(fn);
}

int enc_patch_embed_bwd(int batch, int channels, int img_h, int img_w, int patch, int hidden, int has_cls,
                        const enc_bf16 *dx0, const enc_bf16 *patches, float *dw_pe, float *db_pe, float *dcls,
                        float *dpos, int accumulate, void *ws, size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "enc_patch_embed_bwd";
  int N, S, Kp;
  int r = patch_dims(fn, batch, channels, img_h, img_w, patch, hidden, has_cls, &N, &S, &Kp);
  if (r) return r;
  PtrCheck c(fn);
  c.req(dx0, "dx0").req(patches, "patches").req(dw_pe, "dw_pe").req(db_pe, "db_pe").req(dpos, "dpos");
  if (has_cls) c.req(dcls, "dcls").req(ws, "ws");
  if (c.code) return c.code;
  const size_t need = has_cls ? static_cast<size_t>(batch) * N * hidden * 2 : 0;
  if (ws_bytes < need) return fail(ENC_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, need);
  const hipStream_t s = as_stream(stream);
  const int acc = accumulate ? 1 : 0;
  bool okk = launch_patch_pos_grad(batch, S, hidden, dx0, dpos, has_cls ? dcls : nullptr, acc, s);
  const bf16_t *dtok = dx0;
  if (has_cls) {
    okk = okk && launch_patch_token_rows(batch, N, S, hidden, dx0, static_cast<bf16_t *>(ws), s);
    dtok = static_cast<const bf16_t *>(ws);
  }
  okk = okk && gemm_wgrad(batch * N, hidden, Kp, dtok, patches, dw_pe, db_pe, acc, nullptr, 0, s);
  if (!okk) return refused_after_checks(fn);
  return launched(fn);
}

int enc_stack_saved_bytes(const enc_cfg_t *cfg, int layers, size_t *bytes) {
  const char *fn = "enc_stack_saved_bytes";
  int r = check_cfg(fn, cfg);
  if (r) return r;
  if (layers <= 0) return fail(ENC_ERR_INVALID, "%s: layers must be positive", fn);
  if (!bytes) return fail(ENC_ERR_INVALID, "%s: bytes is NULL", fn);
  *bytes = stack_layout(cfg, layers).total;
  return ok();
}

int enc_stack_workspace_bytes(const enc_cfg_t *cfg, int layers, size_t *bytes) {
  const char *fn = "enc_stack_workspace_bytes";
  int r = check_cfg(fn, cfg);
  if (r) return r;
  if (layers <= 0) return fail(ENC_ERR_INVALID, "%s: layers must be positive", fn);
  if (!bytes) return fail(ENC_ERR_INVALID, "%s: bytes is NULL", fn);
  *bytes = stack_ws(cfg).total;
  return ok();
}

int encoder_stack_fwd(const enc_cfg_t *cfg, int layers, const enc_params_t *params, const enc_bf16 *lnf_g,
                      const enc_bf16 *lnf_b, const enc_bf16 *x0, enc_bf16 *out, void *saved, enc_stream_t stream) {
  const char *fn = "encoder_stack_fwd";
  int r = check_cfg(fn, cfg);
  if (r) return r;
  if (layers <= 0) return fail(ENC_ERR_INVALID, "%s: layers must be positive", fn);
  if (!params) return fail(ENC_ERR_INVALID, "%s: params is NULL", fn);
  for (int l = 0; l < layers; ++l)
    if ((r = check_params(fn, &params[l]))) return r;
  PtrCheck c(fn);
  c.req(lnf_g, "lnf_g").req(lnf_b, "lnf_b").req(x0, "x0").req(out, "out").req(saved, "saved");
  if (c.code) return c.code;
  const StackLayout L = stack_layout(cfg, layers);
  const int M = cfg->batch * cfg->seq;
  const enc_bf16 *x = x0;
  for (int l = 0; l < layers; ++l) {
    enc_bf16 *y = at<enc_bf16>(saved, L.x_step * l);  // layer l's output = layer l+1's input
    if ((r = encoder_layer_fwd(cfg, &params[l], x, y, at<char>(saved, L.layers_off + L.layer_step * l), nullptr, 0,
                               stream)))
      return r;
    x = y;
  }
  if (!launch_ln_fwd(M, cfg->hidden, x, lnf_g, lnf_b, cfg->ln_eps, out, at<float>(saved, L.mean),
                     at<float>(saved, L.rstd), as_stream(stream)))
    return refused_after_checks(fn);
  return launched(fn);
}

int encoder_stack_bwd(const enc_cfg_t *cfg, int layers, const enc_params_t *params, const enc_bf16 *lnf_g,
                      const enc_bf16 *x0, const void *saved, const enc_bf16 *dout, enc_bf16 *dx0,
                      const enc_grads_t *grads, float *dlnf_g, float *dlnf_b, int accumulate, void *ws,
                      size_t ws_bytes, enc_stream_t stream) {
  const char *fn = "encoder_stack_bwd";
  int r = check_cfg(fn, cfg);
  if (r) return r;
  if (layers <= 0) return fail(ENC_ERR_INVALID, "%s: layers must be positive", fn);
  if (!params || !grads) return fail(ENC_ERR_INVALID, "%s: params or grads is NULL", fn);
  for (int l = 0; l < layers; ++l) {
    if ((r = check_params(fn, &params[l]))) return r;
    if ((r = check_grads(fn, &grads[l]))) return r;
  }
  PtrCheck c(fn);
  c.req(lnf_g, "lnf_g").req(x0, "x0").req(saved, "saved").req(dout, "dout").req(dx0, "dx0");
  c.req(dlnf_g, "dlnf_g").req(dlnf_b, "dlnf_b").req(ws, "ws");
  if (c.code) return c.code;
  const StackWs W = stack_ws(cfg);
  if (ws_bytes < W.total) return fail(ENC_ERR_WORKSPACE, "%s: workspace %zu bytes < %zu needed", fn, ws_bytes, W.total);
  const StackLayout L = stack_layout(cfg, layers);
  const int M = cfg->batch * cfg->seq;
  const hipStream_t s = as_stream(stream);
  enc_bf16 *bufs[2] = {at<enc_bf16>(ws, W.dx_a), at<enc_bf16>(ws, W.dx_b)};
  const enc_bf16 *xL = at<enc_bf16>(saved, L.x_step * (layers - 1));
  if (!launch_ln_bwd(M, cfg->hidden, dout, xL, at<float>(saved, L.mean), at<float>(saved, L.rstd), lnf_g, nullptr,
                     bufs[0], dlnf_g, dlnf_b, accumulate ? 1 : 0, at<float>(ws, W.ln_part), s))
    return refused_after_checks(fn);
  if ((r = launched(fn))) return r;
  int cur = 0;
  for (int l = layers - 1; l >= 0; --l) {
    const enc_bf16 *xl = l == 0 ? x0 : at<enc_bf16>(saved, L.x_step * (l - 1));
    enc_bf16 *dxl = l == 0 ? dx0 : bufs[cur ^ 1];
    if ((r = encoder_layer_bwd(cfg, &params[l], xl, at<char>(saved, L.layers_off + L.layer_step * l), bufs[cur], dxl,
                               &grads[l], accumulate, ws, W.dx_a, stream)))
      return r;
    cur ^= 1;
  }
  return ok();
}

// ------------------------------------------------------------ measurement helpers

int enc_calib_mfma(int blocks, int iters, float *out, enc_stream_t stream) {
  const char *fn = "enc_calib_mfma";
  int r = check_dims(fn, {blocks, iters});
  if (r) return r;
  if (blocks > (1 << 20)) return fail(ENC_ERR_UNSUPPORTED, "%s: at most 2^20 blocks", fn);
  PtrCheck c(fn);
  c.req(out, "out");
  if (c.code) return c.code;
  launch_calib_mfma(blocks, iters, out, as_stream(stream));
  return launched(fn);
}

int enc_calib_copy(const void *src, void *dst, size_t bytes, enc_stream_t stream) {
  const char *fn = "enc_calib_copy";
  if (bytes == 0 || bytes % 16) return fail(ENC_ERR_INVALID, "%s: bytes must be a positive multiple of 16", fn);
  PtrCheck c(fn);
  c.req(src, "src").req(dst, "dst");
  if (c.code) return c.code;
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
  if (s0 < d0 + bytes && d0 < s0 + bytes) return fail(ENC_ERR_INVALID, "%s: src and dst overlap", fn);
  launch_calib_copy(src, dst, bytes, as_stream(stream));
  return launched(fn);
}

}  // extern "C"
