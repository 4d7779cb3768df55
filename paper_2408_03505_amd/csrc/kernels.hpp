// Host-side launchers of the device kernels (internal to the library).
// Shapes and pointers are validated by the C-ABI layer before these run;
// each launcher only configures the grid and enqueues on the given stream.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "geometry.hpp"

namespace optimus {

typedef uint16_t bf16_t;

// ---- LayerNorm
bool launch_ln_fwd(int rows, int cols, const bf16_t *x, const bf16_t *gamma, const bf16_t *beta, float eps,
                   bf16_t *y, float *mean, float *rstd, hipStream_t s);
bool launch_ln_bwd(int rows, int cols, const bf16_t *dy, const bf16_t *x, const float *mean, const float *rstd,
                   const bf16_t *gamma, const bf16_t *dresid, bf16_t *dx, float *dgamma, float *dbeta,
                   int accumulate, float *part, hipStream_t s);

// ---- GEMM family: C[m, n] = sum_k A(m, k) B(n, k)
enum class Epi : int {
  kBias = 0,       // Y = acc + bias[n]                       (bf16 out)
  kBiasResid = 1,  // Y = acc + bias[n] + R[m, n]             (bf16 out)
  kBiasGelu = 2,   // U = acc + bias[n]; G = GELU(U)          (two bf16 outs)
  kGeluGrad = 3,   // Y = acc * GELU'(U[m, n])                (bf16 out)
  kPlain = 4,      // Y = acc                                 (bf16 out)
  kF32 = 5,        // Wf (+)= acc; optional fused db         (fp32 out)
  kResid = 6,      // Y = acc + R[m, n]                       (bf16 out)
};

struct GemmArgs {
  int M, N, K;
  const bf16_t *A;  // A(m, k)
  int lda;
  const bf16_t *B;  // B(n, k)
  int ldb;
  bf16_t *Y;  // bf16 output [M, ldy]
  int ldy;
  const bf16_t *bias;  // [N]
  const bf16_t *R;     // residual / saved pre-activation [M, ldy]
  bf16_t *Y2;          // second bf16 output (GELU)
  float *Wf;           // fp32 output [M, ldy]
  float *db;           // fused row sums of A over k (fp32, [M]) for the weight gradient
  int accumulate;
  // Split contraction: when splits > 1, workgroup split s of a tile covers
  // k in [s * k_chunk, min(K, (s + 1) * k_chunk)) (k_chunk a multiple of the
  // k-step) and writes its fp32 partial to Wf + s * split_stride (and, for a
  // weight gradient, db + s * M), overwriting.
  int splits;
  int k_chunk;
  size_t split_stride;
};

// Forward projections: A = X [M, K] row-major, B = W [N, K] row-major.
// Input gradient: A = dY [M, K] row-major, B(n, k) = W[k, n] (W stored [K, N]).
// With a workspace of at least gemm_ws_bytes(M, N, K) bytes, a product whose
// output tiles leave most CUs idle splits its contraction (gemm_split_plan);
// ws = nullptr never splits.
bool launch_gemm_fwd(const GemmArgs &a, Epi epi, void *ws, size_t ws_bytes, hipStream_t s);
bool launch_gemm_dgrad(const GemmArgs &a, Epi epi, void *ws, size_t ws_bytes, hipStream_t s);
// Weight gradient: A(m, k) = dY[k, m], B(n, k) = X[k, n] (contraction over tokens).
// With a workspace of at least gemm_wgrad_ws_bytes(M, N, K) bytes, a problem
// whose output tiles leave most CUs idle splits the token contraction over
// several workgroups per tile and adds the fp32 partials in a fixed order;
// ws = nullptr never splits.
bool launch_gemm_wgrad(const GemmArgs &a, void *ws, size_t ws_bytes, hipStream_t s);

// ---- QK normalisation (LayerNorm of every query and key vector over head_dim)
bool launch_qk_norm_fwd(int M, int heads, int d, const bf16_t *qkv, const bf16_t *qg, const bf16_t *qb,
                        const bf16_t *kg, const bf16_t *kb, float eps, bf16_t *qkvn, float *stats, hipStream_t s);
bool launch_qk_norm_bwd(int M, int heads, int d, const bf16_t *dqkvn, const bf16_t *qkv, const float *stats,
                        const bf16_t *qg, const bf16_t *kg, bf16_t *dqkv, float *dqg, float *dqb, float *dkg,
                        float *dkb, int accumulate, float *part, hipStream_t s);

// ---- Attention
bool launch_attn_fwd(int B, int S, int heads, int d, const bf16_t *qkv, bf16_t *o, float *lse, hipStream_t s);
bool launch_attn_bwd(int B, int S, int heads, int d, const bf16_t *qkv, const bf16_t *o, const float *lse,
                     const bf16_t *dO, bf16_t *dqkv, float *dvec, hipStream_t s);
// Static per-device scratch for the allocation-free backward: room for the
// D vector of B*heads*S <= kAttnScratchFloats queries (4 MiB).  Returns the
// current device's address of the array (looked up once per device).
constexpr size_t kAttnScratchFloats = static_cast<size_t>(1) << 20;
hipError_t attn_bwd_scratch(float **ptr);

// ---- Patch embedding (images -> patch rows; tokens + class token + positions)
bool launch_patchify(int B, int C, int img_h, int img_w, int p, int Kp, const bf16_t *images, bf16_t *patches,
                     hipStream_t s);
bool launch_patch_assemble(int B, int N, int S, int H, int has_cls, const bf16_t *tok, const bf16_t *cls,
                           const bf16_t *pos, bf16_t *x0, hipStream_t s);
bool launch_patch_pos_grad(int B, int S, int H, const bf16_t *dx0, float *dpos, float *dcls, int accumulate,
                           hipStream_t s);
bool launch_patch_token_rows(int B, int N, int S, int H, const bf16_t *dx0, bf16_t *dtok, hipStream_t s);

// ---- Measurement reference kernels
bool launch_calib_mfma(int blocks, int iters, float *out, hipStream_t s);
bool launch_calib_copy(const void *src, void *dst, size_t bytes, hipStream_t s);

}  // namespace optimus
