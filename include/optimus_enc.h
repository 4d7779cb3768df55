/*
 * optimus_enc.h - C ABI of the fine-grained ViT encoder-layer kernels.
 *
 * Optimus (arXiv 2408.03505) trains multimodal LLMs by running vision-encoder
 * work inside the LLM pipeline's idle periods.  Many of those bubbles last
 * well under a millisecond (about 300 us for tensor-parallel bubbles, §2.3,
 * challenge 3), shorter than one encoder layer's forward or backward, so the
 * paper splits the encoder layer into separately launched kernels and places
 * each one on its own (abstract; §3.1, design decision 3; §4.2, the
 * ScheduleKernels step, which packs kernels into a bubble while their summed
 * time fits and keeps the encoder's internal order).  Forward and backward are
 * scheduled separately, and the backward may be skipped for a frozen encoder
 * (§6, frozen parameters).
 *
 * This library provides that chain for one pre-LN ViT layer on one
 * micro-batch: a composite forward and backward plus one entry point per
 * kernel, each of which only enqueues work on a caller-given HIP stream.
 * Parameters and activations are bfloat16; parameter gradients are fp32
 * (bf16 parameters with fp32 gradients, §4.5 memory analysis).
 *
 * Conventions shared by every entry point
 *  - enc_bf16 is bfloat16 storage (round-to-nearest-even from fp32).
 *  - Every tensor is dense and row-major.  Token rows M = batch*seq are
 *    ordered sequence-major (row r = b*seq + s).  Weights are [out, in].
 *    qkv columns are packed [3][heads][head_dim]; attention outputs are
 *    packed [heads][head_dim].
 *  - Every pointer is a DEVICE pointer owned by the caller.  The library never
 *    allocates, frees or synchronises, and keeps no global mutable state
 *    besides a thread-local last-error string.  Inputs are never written.
 *    Outputs must not alias inputs, except that with accumulate=1 the fp32
 *    gradient buffers are read and written.
 *  - Every tensor pointer must be 16-byte aligned.  hidden, heads*head_dim and
 *    mlp must be multiples of 8; head_dim must be 64, 80 or 128.
 *  - Each call validates its arguments, enqueues its kernels on `stream`
 *    (a hipStream_t; NULL is the null stream) and returns.  Device faults
 *    surface at the caller's next synchronisation.  Calls contain no host
 *    synchronisation and no allocation, so they can be captured into HIP
 *    graphs.
 *  - Return value: ENC_OK (0) or a negative enc_status; enc_last_error()
 *    then describes the failure.  On error nothing has been enqueued, except
 *    for ENC_ERR_LAUNCH, which reports a failed launch after earlier kernels
 *    of the same call may already have been enqueued.
 */
#ifndef OPTIMUS_ENC_H
#define OPTIMUS_ENC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t enc_bf16;
typedef void *enc_stream_t; /* hipStream_t */

enum enc_status {
  ENC_OK = 0,
  ENC_ERR_INVALID = -1,     /* null pointer or non-positive dimension */
  ENC_ERR_UNSUPPORTED = -2, /* shape outside what the kernels support */
  ENC_ERR_ALIGN = -3,       /* a pointer is not 16-byte aligned */
  ENC_ERR_LAUNCH = -4,      /* a HIP kernel launch failed */
  ENC_ERR_WORKSPACE = -5    /* workspace smaller than the size query returned */
};

/* Shape of one encoder layer on one micro-batch.  heads*head_dim may differ
 * from hidden: one tensor-parallel rank keeps the full LayerNorm width but
 * only heads/TP heads and mlp/TP of the MLP.  Widths follow the ViT table
 * of Appendix A (width, MLP dimension, heads, head dimension). */
typedef struct {
  int batch;    /* sequences in the micro-batch */
  int seq;      /* tokens per sequence (patches + class token) */
  int hidden;   /* model width H */
  int heads;    /* attention heads on this GPU */
  int head_dim; /* 64, 80 or 128 */
  int mlp;      /* MLP width F on this GPU */
  float ln_eps; /* LayerNorm epsilon, added to the variance */
} enc_cfg_t;

/* The twelve bf16 parameters (A = heads*head_dim). */
typedef struct {
  const enc_bf16 *ln1_g, *ln1_b; /* [H] */
  const enc_bf16 *w_qkv;         /* [3A, H] */
  const enc_bf16 *b_qkv;         /* [3A] */
  const enc_bf16 *w_o;           /* [H, A] */
  const enc_bf16 *b_o;           /* [H] */
  const enc_bf16 *ln2_g, *ln2_b; /* [H] */
  const enc_bf16 *w_1;           /* [F, H] */
  const enc_bf16 *b_1;           /* [F] */
  const enc_bf16 *w_2;           /* [H, F] */
  const enc_bf16 *b_2;           /* [H] */
} enc_params_t;

/* fp32 parameter gradients, same shapes as enc_params_t. */
typedef struct {
  float *ln1_g, *ln1_b, *w_qkv, *b_qkv, *w_o, *b_o;
  float *ln2_g, *ln2_b, *w_1, *b_1, *w_2, *b_2;
} enc_grads_t;

/* Byte offsets of the saved-for-backward tensors inside one caller buffer
 * (every offset is a multiple of 256).  bf16: y1, h, y2 [M,H]; qkv [M,3A];
 * o [M,A]; u, g [M,F].  fp32: mean1, rstd1, mean2, rstd2 [M];
 * lse [batch, heads, seq]. */
typedef struct {
  size_t y1, mean1, rstd1, qkv, o, lse, h, y2, mean2, rstd2, u, g;
  size_t total; /* bytes the saved buffer must hold */
} enc_saved_layout_t;

/* ------------------------------------------------------------ status */

/* Static text for a status code. */
const char *enc_status_string(int status);
/* Description of the last failure on the calling thread ("" if none). */
const char *enc_last_error(void);
/* ABI version of this header (bumped on incompatible change; 2: workspace
 * arguments of the projection entry points). */
int enc_abi_version(void);

/* ------------------------------------------------------------ sizing */

/* [Caller-owned buffers of one scheduling unit: the layer's saved tensors
 * and workspaces (§4.2; memory accounting §4.5)]
 * Validates cfg and fills the saved-buffer layout. */
int enc_saved_layout(const enc_cfg_t *cfg, enc_saved_layout_t *layout);
/* Workspace bytes that encoder_layer_fwd / encoder_layer_bwd need. */
int enc_layer_workspace_bytes(const enc_cfg_t *cfg, size_t *bytes);
/* Workspace of the per-kernel entry points that take one. */
int enc_ln_bwd_workspace_bytes(int rows, int cols, size_t *bytes);
int enc_attn_bwd_workspace_bytes(int batch, int seq, int heads, int head_dim, size_t *bytes);

/* ------------------------------------------------------------ composites */

/* [One micro-batch of one encoder layer, as one scheduling unit (§4.2);
 * the chain of the kernels below (§3.1 decision 3)]
 * Both composites check every argument, and every shape limit of every
 * kernel they launch, before the first launch: a status other than ENC_OK
 * and ENC_ERR_LAUNCH means nothing was enqueued.
 * Forward of one pre-LN encoder layer on one micro-batch: the kernels of
 * the forward chain in order (LN1, QKV projection, attention, output
 * projection + residual, LN2, MLP up + GELU, MLP down + residual) on one
 * stream.  x, out: [M, H].  saved: enc_saved_layout().total bytes, filled
 * with the intermediates the backward needs.  ws: NULL (no product is
 * split) or a workspace of enc_layer_workspace_bytes() bytes (ws_bytes
 * states its size; the forward uses it for split-product partials). */
int encoder_layer_fwd(const enc_cfg_t *cfg, const enc_params_t *params,
                      const enc_bf16 *x, enc_bf16 *out, void *saved,
                      void *ws, size_t ws_bytes, enc_stream_t stream);

/* Backward of encoder_layer_fwd given dout = dL/dout [M, H]: writes
 * dx [M, H] and the twelve parameter gradients (overwritten when
 * accumulate=0, added to when accumulate=1).  saved is the buffer the
 * forward filled for the same x and params. */
int encoder_layer_bwd(const enc_cfg_t *cfg, const enc_params_t *params,
                      const enc_bf16 *x, const void *saved,
                      const enc_bf16 *dout, enc_bf16 *dx,
                      const enc_grads_t *grads, int accumulate,
                      void *ws, size_t ws_bytes, enc_stream_t stream);

/* ------------------------------------------------------------ product workspaces
 *
 * Every projection entry point (forward, input gradient, weight gradient)
 * takes an optional workspace `ws` of `ws_bytes` bytes.  With ws = NULL the
 * product runs unsplit.  With a workspace of at least the size query's bytes,
 * a product whose output tiles would leave most of the GPU idle splits its
 * contraction over several workgroups per tile: fp32 partials go to ws and a
 * second kernel adds them in a fixed order and applies the epilogue, so
 * results stay deterministic for a given shape and workspace choice.  The
 * queries return 0 for shapes that never split; a given workspace smaller
 * than the query is ENC_ERR_WORKSPACE.  Forward and input-gradient products
 * with output [M, N] and contraction K:
 *   enc_qkv_fwd        (M, 3A, H)   enc_oproj_fwd       (M, H, A)
 *   enc_mlp_up_fwd     (M, F, H)    enc_mlp_down_fwd    (M, H, F)
 *   enc_mlp_down_bwd_data (M, F, H) enc_mlp_up_bwd_data (M, H, F)
 *   enc_oproj_bwd_data (M, A, H)    enc_qkv_bwd_data[_add] (M, H, 3A) */
int enc_linear_workspace_bytes(int M, int N, int K, size_t *bytes);

/* ------------------------------------------------------------ forward kernels
 *
 * One entry point per kernel of the layer's decomposition.  The paper
 * splits the encoder layer into kernels so that each one can be placed in a
 * bubble on its own (§3.1, design decision 3; §4.2, ScheduleKernels), but
 * it does not write the layer out: it names the encoders (Appendix A, ViT
 * table: width, MLP dimension, heads, head dimension).  The layer these
 * kernels compute is the pre-LN ViT block of those encoders,
 *   h = x + Attn(LN1(x)) w_o^T + b_o,  out = h + GELU(LN2(h) w_1^T + b_1) w_2^T + b_2,
 * whose parameter count, 4H^2 + 2HF per layer, reproduces the table's model
 * sizes.  Each declaration below names its step of that block. */

/* [Block steps LN1 and LN2 (Appendix A encoders; §3.1 decision 3)]
 * LayerNorm over each of `rows` rows of `cols` values: per row the mean and
 * biased variance, rstd = 1/sqrt(var + eps), y = (x - mean)*rstd*gamma + beta.
 * x, y: [rows, cols] bf16; gamma, beta: [cols] bf16; mean, rstd: [rows] fp32
 * (kept for the backward).  cols must be a multiple of 8 and <= 16384. */
int enc_ln_fwd(int rows, int cols, const enc_bf16 *x, const enc_bf16 *gamma,
               const enc_bf16 *beta, float eps, enc_bf16 *y, float *mean,
               float *rstd, enc_stream_t stream);

/* [Block step: fused Q, K, V projection (Appendix A heads x head dim; §3.1 decision 3)]
 * QKV projection: qkv[M, 3A] = y1[M, H] * w_qkv[3A, H]^T + b_qkv[3A].
 * b_qkv may be NULL (no bias, as in the ViT-22B-style block below). */
int enc_qkv_fwd(int M, int H, int A, const enc_bf16 *y1, const enc_bf16 *w_qkv,
                const enc_bf16 *b_qkv, enc_bf16 *qkv, void *ws, size_t ws_bytes,
                enc_stream_t stream);

/* [Block step: multi-head self-attention (Appendix A heads x head dim; §3.1 decision 3)]
 * Bidirectional softmax attention of every (sequence, head): for queries i
 * and keys j of one sequence, P = softmax_j(q_i . k_j / sqrt(head_dim)),
 * o_i = sum_j P_ij v_j.  qkv: [batch*seq, 3*heads*head_dim] as written by
 * enc_qkv_fwd; o: [batch*seq, heads*head_dim]; lse: [batch, heads, seq] fp32,
 * the natural-log normaliser log sum_j exp(q_i . k_j / sqrt(head_dim)). */
int enc_attn_fwd(int batch, int seq, int heads, int head_dim,
                 const enc_bf16 *qkv, enc_bf16 *o, float *lse,
                 enc_stream_t stream);

/* [Block step: attention output projection + residual (§3.1 decision 3)]
 * Output projection with residual: h[M, H] = resid[M, H] + o[M, A] *
 * w_o[H, A]^T + b_o[H]. */
int enc_oproj_fwd(int M, int A, int H, const enc_bf16 *o, const enc_bf16 *w_o,
                  const enc_bf16 *b_o, const enc_bf16 *resid, enc_bf16 *h,
                  void *ws, size_t ws_bytes, enc_stream_t stream);

/* [Block step: MLP up-projection to the MLP dimension of Appendix A, GELU (§3.1 decision 3)]
 * MLP up-projection with GELU: u[M, F] = y2[M, H] * w_1[F, H]^T + b_1[F];
 * g = GELU(u) = u * Phi(u) (exact erf form).  Both u and g are written
 * (u is kept for the backward). */
int enc_mlp_up_fwd(int M, int H, int F, const enc_bf16 *y2, const enc_bf16 *w_1,
                   const enc_bf16 *b_1, enc_bf16 *u, enc_bf16 *g, void *ws,
                   size_t ws_bytes, enc_stream_t stream);

/* [Block step: MLP down-projection + residual (§3.1 decision 3)]
 * MLP down-projection with residual: out[M, H] = resid[M, H] + g[M, F] *
 * w_2[H, F]^T + b_2[H]. */
int enc_mlp_down_fwd(int M, int F, int H, const enc_bf16 *g, const enc_bf16 *w_2,
                     const enc_bf16 *b_2, const enc_bf16 *resid, enc_bf16 *out,
                     void *ws, size_t ws_bytes, enc_stream_t stream);

/* ------------------------------------------------------------ backward kernels
 *
 * The backward of the same block, one kernel per step, scheduled apart from
 * the forward (§4.2; the backward may be skipped for a frozen encoder, §6).
 * Parameter gradients are fp32 (bf16 parameters with fp32 gradients, §4.5
 * memory analysis). */

/* [Backward of the MLP down-projection and GELU (§3.1 decision 3; §4.2)]
 * MLP down input gradient through GELU: du[M, F] = (dout[M, H] * w_2[H, F])
 * * GELU'(u), GELU'(u) = Phi(u) + u*phi(u); u is the saved pre-activation. */
int enc_mlp_down_bwd_data(int M, int F, int H, const enc_bf16 *dout,
                          const enc_bf16 *w_2, const enc_bf16 *u, enc_bf16 *du,
                          void *ws, size_t ws_bytes, enc_stream_t stream);

/* [Backward of the MLP up-projection, input side (§3.1 decision 3; §4.2)]
 * MLP up input gradient: dy2[M, H] = du[M, F] * w_1[F, H]. */
int enc_mlp_up_bwd_data(int M, int H, int F, const enc_bf16 *du,
                        const enc_bf16 *w_1, enc_bf16 *dy2, void *ws,
                        size_t ws_bytes, enc_stream_t stream);

/* [Backward of the output projection, input side (§3.1 decision 3; §4.2)]
 * Output projection input gradient: do_[M, A] = dh[M, H] * w_o[H, A]. */
int enc_oproj_bwd_data(int M, int A, int H, const enc_bf16 *dh,
                       const enc_bf16 *w_o, enc_bf16 *do_, void *ws,
                       size_t ws_bytes, enc_stream_t stream);

/* [Backward of the QKV projection, input side (§3.1 decision 3; §4.2)]
 * QKV projection input gradient: dy1[M, H] = dqkv[M, 3A] * w_qkv[3A, H]. */
int enc_qkv_bwd_data(int M, int H, int A, const enc_bf16 *dqkv,
                     const enc_bf16 *w_qkv, enc_bf16 *dy1, void *ws,
                     size_t ws_bytes, enc_stream_t stream);

/* [Backward of the four projections, parameter side; fp32 gradients (§4.5)]
 * Parameter gradients of a linear layer Y = X W^T + b, summed over the M
 * token rows: dW[N, K] = dY[M, N]^T * X[M, K]; db[N] = sum_m dY[m, :]
 * (db may be NULL).  fp32 outputs are overwritten (accumulate=0) or added
 * to (accumulate=1).  The sums are deterministic (no atomics).
 * ws: NULL, or at least enc_linear_bwd_weight_workspace_bytes(M, N, K)
 * bytes (else ENC_ERR_WORKSPACE).  When the output's tiles would leave most
 * of the GPU idle (a small dW with many tokens), a workspace lets the token
 * sum be split over several workgroups per tile; their fp32 partials are
 * added in a fixed order, so results stay deterministic for a given shape
 * and workspace choice.  The size query returns 0 for shapes that never
 * split.  With ws = NULL nothing is split. */
int enc_linear_bwd_weight_workspace_bytes(int M, int N, int K, size_t *bytes);
int enc_linear_bwd_weight(int M, int N, int K, const enc_bf16 *dY,
                          const enc_bf16 *X, float *dW, float *db,
                          int accumulate, void *ws, size_t ws_bytes,
                          enc_stream_t stream);
/* The four uses of enc_linear_bwd_weight in the layer, by name (ws as above,
 * sized for the same M, N, K):
 *  MLP down: dw_2[H, F] = dout^T g,   db_2[H]      (N = H, K = F)
 *  MLP up:   dw_1[F, H] = du^T y2,    db_1[F]      (N = F, K = H)
 *  out proj: dw_o[H, A] = dh^T o,     db_o[H]      (N = H, K = A)
 *  QKV:      dw_qkv[3A, H] = dqkv^T y1, db_qkv[3A]  (N = 3A, K = H) */
int enc_mlp_down_bwd_weight(int M, int F, int H, const enc_bf16 *dout,
                            const enc_bf16 *g, float *dw_2, float *db_2,
                            int accumulate, void *ws, size_t ws_bytes,
                            enc_stream_t stream);
int enc_mlp_up_bwd_weight(int M, int H, int F, const enc_bf16 *du,
                          const enc_bf16 *y2, float *dw_1, float *db_1,
                          int accumulate, void *ws, size_t ws_bytes,
                          enc_stream_t stream);
int enc_oproj_bwd_weight(int M, int A, int H, const enc_bf16 *dh,
                         const enc_bf16 *o, float *dw_o, float *db_o,
                         int accumulate, void *ws, size_t ws_bytes,
                         enc_stream_t stream);
int enc_qkv_bwd_weight(int M, int H, int A, const enc_bf16 *dqkv,
                       const enc_bf16 *y1, float *dw_qkv, float *db_qkv,
                       int accumulate, void *ws, size_t ws_bytes,
                       enc_stream_t stream);

/* [Backward of LN2 and LN1 with the residual branch (§3.1 decision 3; §4.2)]
 * LayerNorm backward (exact gradient of enc_ln_fwd) with the residual
 * branch added: with xhat = (x - mean)*rstd and ghat = dy*gamma, per row
 * dx = dresid + rstd*(ghat - mean(ghat) - xhat*mean(ghat*xhat)); and over
 * all rows dgamma = sum dy*xhat, dbeta = sum dy (fp32, overwritten or
 * accumulated).  dresid may be NULL (treated as zero).  The column sums use
 * a fixed-order two-pass reduction through ws
 * (enc_ln_bwd_workspace_bytes). */
int enc_ln_bwd(int rows, int cols, const enc_bf16 *dy, const enc_bf16 *x,
               const float *mean, const float *rstd, const enc_bf16 *gamma,
               const enc_bf16 *dresid, enc_bf16 *dx, float *dgamma,
               float *dbeta, int accumulate, void *ws, size_t ws_bytes,
               enc_stream_t stream);

/* [Backward of the self-attention step (§3.1 decision 3; §4.2)]
 * Attention backward (exact gradient of enc_attn_fwd): with P recomputed
 * from lse, D_i = sum_e do_ie*o_ie, dV = P^T dO, dP = dO V^T,
 * dS = P*(dP - D), dQ = dS K/sqrt(d), dK = dS^T Q/sqrt(d), written to
 * dqkv [batch*seq, 3*heads*head_dim] in the qkv packing.  ws holds D
 * (enc_attn_bwd_workspace_bytes); no atomics, deterministic. */
int enc_attn_bwd(int batch, int seq, int heads, int head_dim,
                 const enc_bf16 *qkv, const enc_bf16 *o, const float *lse,
                 const enc_bf16 *do_, enc_bf16 *dqkv, void *ws,
                 size_t ws_bytes, enc_stream_t stream);

/* [For callers that cannot allocate: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.]
 * enc_attn_bwd without a workspace argument: same kernels, same results, with
 * the D vector kept in a static device array of the library (4 MiB per GPU,
 * held until the process ends), so the call allocates nothing and needs no
 * caller memory beyond its inputs and outputs.  Limit: batch*heads*seq <=
 * 1048576 (2^20 queries in all), else ENC_ERR_UNSUPPORTED.  The first call
 * on a device looks the array up for that device (hipGetSymbolAddress); a
 * failure there is ENC_ERR_LAUNCH.  Every call on one GPU shares that GPU's
 * array: calls that overlap on one GPU (different streams, or different
 * threads without ordering) race on it and their results are undefined;
 * calls ordered on one stream are safe.  Nothing in the array needs to start
 * at zero (each call writes D before reading it). */
int enc_attn_bwd_noalloc(int batch, int seq, int heads, int head_dim,
                         const enc_bf16 *qkv, const enc_bf16 *o, const float *lse,
                         const enc_bf16 *do_, enc_bf16 *dqkv, enc_stream_t stream);

/* ------------------------------------------------------------ ViT-22B-style block
 *
 * The paper's largest encoder is ViT-22B (Appendix A).  The cited ViT-22B
 * architecture differs from the sequential pre-LN block above: attention and
 * MLP run in parallel on one LayerNorm of the input, queries and keys are
 * layer-normalised per head before the dot product, and the QKV projection
 * has no bias:
 *   y    = LN(x)                          (ln_g, ln_b over H)
 *   qkv  = y * w_qkv^T                    (no bias)
 *   qkvn = QKnorm(qkv)                    (LN over head_dim of every query and
 *                                          key vector: qn_g, qn_b, kn_g, kn_b
 *                                          of length head_dim, shared by heads;
 *                                          values unchanged)
 *   o    = Attn(qkvn)                     (as enc_attn_fwd)
 *   h    = x + o * w_o^T + b_o            (residual + attention branch)
 *   out  = h + GELU(y * w_1^T + b_1) * w_2^T + b_2   (+ MLP branch, fed by y)
 * Every LayerNorm uses cfg->ln_eps.  Shapes as in enc_params_t, plus the four
 * QK-norm vectors of length head_dim. */
typedef struct {
  const enc_bf16 *ln_g, *ln_b;               /* [H] */
  const enc_bf16 *w_qkv;                     /* [3A, H] */
  const enc_bf16 *qn_g, *qn_b, *kn_g, *kn_b; /* [head_dim] */
  const enc_bf16 *w_o, *b_o;                 /* [H, A], [H] */
  const enc_bf16 *w_1, *b_1;                 /* [F, H], [F] */
  const enc_bf16 *w_2, *b_2;                 /* [H, F], [H] */
} enc_pparams_t;

/* fp32 parameter gradients, same shapes as enc_pparams_t. */
typedef struct {
  float *ln_g, *ln_b, *w_qkv, *qn_g, *qn_b, *kn_g, *kn_b, *w_o, *b_o, *w_1, *b_1, *w_2, *b_2;
} enc_pgrads_t;

/* Byte offsets (multiples of 256) of the block's saved tensors in one caller
 * buffer.  bf16: y, h [M,H]; qkv, qkvn [M,3A]; o [M,A]; u, g [M,F].  fp32:
 * mean, rstd [M]; qkstats [M, heads, 4] = (query mean, query rstd, key mean,
 * key rstd) per token and head; lse [batch, heads, seq]. */
typedef struct {
  size_t y, mean, rstd, qkv, qkvn, qkstats, o, lse, h, u, g;
  size_t total;
} enc_psaved_layout_t;

/* [ViT-22B block (Appendix A): buffers]
 * Fills layout with the offsets above for cfg (256-byte aligned, disjoint);
 * ENC_ERR_INVALID / ENC_ERR_UNSUPPORTED for a bad cfg. */
int enc_parallel_saved_layout(const enc_cfg_t *cfg, enc_psaved_layout_t *layout);
/* Workspace bytes encoder_parallel_bwd needs. */
int enc_parallel_workspace_bytes(const enc_cfg_t *cfg, size_t *bytes);

/* [ViT-22B block (Appendix A): forward as one scheduling unit (§4.2)]
 * Forward of the block: LN, QKV projection, QK norm, attention, output
 * projection + residual, MLP up + GELU (from y), MLP down + residual, on one
 * stream.  x, out: [M, H]; saved: enc_parallel_saved_layout().total bytes. */
int encoder_parallel_fwd(const enc_cfg_t *cfg, const enc_pparams_t *params,
                         const enc_bf16 *x, enc_bf16 *out, void *saved,
                         enc_stream_t stream);

/* [ViT-22B block (Appendix A): backward as one scheduling unit (§4.2)]
 * (The block's two composites run every product unsplit.)
 * Exact gradient of encoder_parallel_fwd.  dy of the shared LayerNorm is the
 * sum of both branches' input gradients (the QKV input gradient adds the
 * MLP branch's in its epilogue); dx = dout + LN backward(dy).  accumulate as
 * for encoder_layer_bwd; deterministic. */
int encoder_parallel_bwd(const enc_cfg_t *cfg, const enc_pparams_t *params,
                         const enc_bf16 *x, const void *saved,
                         const enc_bf16 *dout, enc_bf16 *dx,
                         const enc_pgrads_t *grads, int accumulate, void *ws,
                         size_t ws_bytes, enc_stream_t stream);

/* [ViT-22B block step (Appendix A): query/key normalisation]
 * QK normalisation: qkvn = qkv with every (token, head) query vector replaced
 * by LN(q) * qn_g + qn_b and every key vector by LN(k) * kn_g + kn_b (LN over
 * head_dim, biased variance, eps inside the square root); values copied.
 * qkv, qkvn: [M, 3*heads*head_dim]; stats: [M, heads, 4] fp32 (query mean,
 * query rstd, key mean, key rstd).  head_dim in {64, 80, 128}. */
int enc_qk_norm_fwd(int M, int heads, int head_dim, const enc_bf16 *qkv,
                    const enc_bf16 *qn_g, const enc_bf16 *qn_b,
                    const enc_bf16 *kn_g, const enc_bf16 *kn_b, float eps,
                    enc_bf16 *qkvn, float *stats, enc_stream_t stream);

/* [ViT-22B block step (Appendix A): backward of the query/key normalisation]
 * Workspace bytes enc_qk_norm_bwd needs (per-block partial sums of the four
 * affine gradients, reduced in a fixed order). */
int enc_qk_norm_bwd_workspace_bytes(int M, int heads, int head_dim, size_t *bytes);

/* Gradient of enc_qk_norm_fwd: dqkv from dqkvn (LayerNorm backward for
 * queries and keys, values copied) and the fp32 gradients of the four
 * affine vectors, summed over tokens and heads in a fixed order (overwritten,
 * or added with accumulate=1).  ws: enc_qk_norm_bwd_workspace_bytes. */
int enc_qk_norm_bwd(int M, int heads, int head_dim, const enc_bf16 *dqkvn,
                    const enc_bf16 *qkv, const float *stats,
                    const enc_bf16 *qn_g, const enc_bf16 *kn_g, enc_bf16 *dqkv,
                    float *dqn_g, float *dqn_b, float *dkn_g, float *dkn_b,
                    int accumulate, void *ws, size_t ws_bytes,
                    enc_stream_t stream);

/* [ViT-22B block step (Appendix A): the shared LayerNorm's input gradient]
 * QKV input gradient plus an addend (the other branch's input gradient of
 * the shared LayerNorm output): dy[M, H] = dqkv[M, 3A] * w_qkv[3A, H] +
 * addend[M, H], accumulated in fp32 before one rounding to bf16. */
int enc_qkv_bwd_data_add(int M, int H, int A, const enc_bf16 *dqkv,
                         const enc_bf16 *w_qkv, const enc_bf16 *addend,
                         enc_bf16 *dy, void *ws, size_t ws_bytes,
                         enc_stream_t stream);

/* ------------------------------------------------------------ whole encoder
 *
 * The encoders of the paper are ViTs (Appendix A): a patch embedding, a
 * stack of encoder layers and a final LayerNorm.  An image of side img cut
 * into p x p patches gives N = (img_h/p)(img_w/p) tokens, plus one class
 * token when has_cls (224/16 -> 196 + 1 = 197; 224/14 -> 256).
 *
 * Patch embedding: the stride-p convolution as a matrix product,
 *   patches[b*N + n, c*p*p + i*p + j] = images[b, c, py*p + i, px*p + j]
 *   (n = py*(img_w/p) + px; images [B, C, img_h, img_w] bf16),
 *   tok = patches * w_pe^T + b_pe,
 *   x0[b*S + s] = (has_cls and s == 0 ? cls : tok[b*N + s - has_cls]) + pos[s],
 * with S = N + has_cls.  Kp = C*p*p rounded up to a multiple of 8: patches
 * is [B*N, Kp] and w_pe is [hidden, Kp] whose columns C*p*p .. Kp-1 must be
 * zero (they are written zero in patches).  cls [hidden] (only with
 * has_cls), pos [S, hidden], b_pe [hidden].  ws: with has_cls,
 * enc_patch_embed_workspace_bytes (the tokens before the class token is
 * placed); without, none (the tokens are x0's rows). */
int enc_patch_embed_workspace_bytes(int batch, int channels, int img_h, int img_w, int patch, int hidden,
                                    int has_cls, size_t *bytes);
int enc_patch_embed_fwd(int batch, int channels, int img_h, int img_w, int patch, int hidden, int has_cls,
                        const enc_bf16 *images, const enc_bf16 *w_pe, const enc_bf16 *b_pe, const enc_bf16 *cls,
                        const enc_bf16 *pos, enc_bf16 *patches, enc_bf16 *x0, void *ws, size_t ws_bytes,
                        enc_stream_t stream);
/* [Whole ViT encoder (Appendix A): backward of the patch embedding]
 * Parameter gradients of the patch embedding from dx0 [B*S, hidden] and the
 * forward's patches: dw_pe [hidden, Kp], db_pe [hidden], dpos [S, hidden]
 * (sum over the batch in order), dcls [hidden] (only with has_cls) -- all
 * fp32, overwritten or (accumulate=1) added.  The images get no gradient.
 * ws: as for the forward. */
int enc_patch_embed_bwd(int batch, int channels, int img_h, int img_w, int patch, int hidden, int has_cls,
                        const enc_bf16 *dx0, const enc_bf16 *patches, float *dw_pe, float *db_pe, float *dcls,
                        float *dpos, int accumulate, void *ws, size_t ws_bytes, enc_stream_t stream);

/* [Whole ViT encoder (Appendix A): the layer stack and final LayerNorm]
 * A stack of `layers` sequential encoder layers (params[layers], each as for
 * encoder_layer_fwd) followed by a final LayerNorm (lnf_g, lnf_b):
 * out = LN(layer_{L-1}(... layer_0(x0))).  saved (enc_stack_saved_bytes)
 * holds every layer's output (the next layer's input), every layer's saved
 * tensors and the final LayerNorm's statistics. */
int enc_stack_saved_bytes(const enc_cfg_t *cfg, int layers, size_t *bytes);
int enc_stack_workspace_bytes(const enc_cfg_t *cfg, int layers, size_t *bytes);
int encoder_stack_fwd(const enc_cfg_t *cfg, int layers, const enc_params_t *params,
                      const enc_bf16 *lnf_g, const enc_bf16 *lnf_b, const enc_bf16 *x0,
                      enc_bf16 *out, void *saved, enc_stream_t stream);
/* [Whole ViT encoder (Appendix A): backward of the stack]
 * Backward of encoder_stack_fwd: dx0 and the gradients of every layer
 * (grads[layers]) and of the final LayerNorm; accumulate as for
 * encoder_layer_bwd.  ws: enc_stack_workspace_bytes. */
int encoder_stack_bwd(const enc_cfg_t *cfg, int layers, const enc_params_t *params,
                      const enc_bf16 *lnf_g, const enc_bf16 *x0, const void *saved,
                      const enc_bf16 *dout, enc_bf16 *dx0, const enc_grads_t *grads,
                      float *dlnf_g, float *dlnf_b, int accumulate, void *ws,
                      size_t ws_bytes, enc_stream_t stream);

/* ---- Kernel-to-bubble packing (host code, no GPU)
 *
 * The bubble scheduler's ScheduleKernels step (§4.2, fine-grained bubble
 * exploitation): one micro-batch's encoder kernels are placed, in chain
 * order (each kernel after the one whose output it reads), into the LLM timeline.
 * Computation kernels go into bubbles, several per bubble as long as their
 * summed time fits; communication kernels are not put into bubbles but
 * overlapped with LLM computation (§3.1, design decision 3).  Kernels are
 * never split or reordered: each goes into the earliest interval of its
 * kind, at or after its predecessor's interval, whose remaining time holds
 * it -- the componentwise-earliest of all feasible order-keeping placements.
 *
 * kernel_us[n_kernels]      durations in chain order (finite, >= 0)
 * kernel_comm[n_kernels]    1 for a communication kernel; NULL: none is
 * interval_us[n_intervals]  interval lengths in time order (finite, >= 0)
 * interval_bubble[n_int.]   1 for a bubble, 0 for a period of LLM computation
 * out_interval[n_kernels]   interval of each kernel; -1 when it does not fit
 *                           (every later kernel is then -1 too)
 * out_offset_us[n_kernels]  start within its interval (-1 if unplaced); may
 *                           be NULL
 * All arrays are host memory owned by the caller.  Returns the number of
 * kernels placed (n_kernels when all fit) or a negative enc_status; outputs
 * are written only after the arguments validate. */
int enc_schedule_kernels(const double *kernel_us, const int *kernel_comm, int n_kernels,
                         const double *interval_us, const int *interval_bubble, int n_intervals,
                         int *out_interval, double *out_offset_us);

/* ---- Measurement helpers (not steps of the layer)
 *
 * Two reference kernels that bound what the layer's kernels can reach on the
 * GPU at hand: an MFMA-only loop (the sustained bf16 matrix-core rate under
 * the clock the chip holds while every matrix core is busy) and a device
 * copy (the sustained HBM rate).  The caller times them with events on
 * `stream`; both follow the conventions above. */

/* blocks x 256 threads; every wave issues iters x 16 independent
 * v_mfma_f32_32x32x16_bf16 on register operands whose mantissa bits change
 * every iteration, i.e. blocks * 4 * iters * 16 * 32768 flops.  One float
 * per thread is written to out[blocks * 256] so that nothing is elided.
 * blocks, iters > 0. */
int enc_calib_mfma(int blocks, int iters, float *out, enc_stream_t stream);

/* dst[0, bytes) = src[0, bytes) with 16-byte loads and stores.  bytes is a
 * positive multiple of 16; src and dst are 16-byte aligned and do not
 * overlap. */
int enc_calib_copy(const void *src, void *dst, size_t bytes, enc_stream_t stream);

/* Launch plan of one projection product, for tools that model its memory
 * traffic or dispatches: the output tile (*tile_rows x *tile_cols of the
 * output as stored) and the number of contraction splits (*splits, 1 when
 * not split) that the entry points use when given a workspace of the size
 * their query returns (with ws = NULL nothing is split).  layout:
 *   ENC_LAYOUT_FWD    the forward projections: output [M, N] = X[M, K] W^T
 *   ENC_LAYOUT_DGRAD  the input gradients: output [M, N] = dY[M, K] W[K, N]
 *   ENC_LAYOUT_WGRAD  the weight gradients: dW[N, K] over M tokens (M, N, K
 *                     as enc_linear_bwd_weight)
 * Sizes follow the entry points' rules (ENC_ERR_INVALID / ENC_ERR_UNSUPPORTED
 * as they would return); ENC_ERR_INVALID for another layout or a NULL
 * output.  Host only: touches no device. */
enum { ENC_LAYOUT_FWD = 0, ENC_LAYOUT_DGRAD = 1, ENC_LAYOUT_WGRAD = 2 };
int enc_linear_plan(int layout, int M, int N, int K, int *tile_rows, int *tile_cols, int *splits);

#ifdef __cplusplus
}
#endif

#endif /* OPTIMUS_ENC_H */
