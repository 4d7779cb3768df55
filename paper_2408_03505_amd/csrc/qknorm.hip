// QK normalisation of the ViT-22B-style block: LayerNorm of every query and
// key vector over head_dim, per token and head, with affine parameters of
// length head_dim shared by all heads; values pass through unchanged.
//
// One 16-lane group per (token, head) pair: lane j holds elements
// [8j, 8j + 8) of the pair's query and key vectors (lanes with 8j >= d hold
// nothing), loaded and stored as 16-byte chunks; sums are group reductions
// over four xor-shuffles.  The backward writes dq, dk (LayerNorm backward)
// and dv (copied), and reduces the affine gradients in a fixed order: every
// lane sums its elements over the pairs its group visits, the 16 groups of a
// block are added in LDS, and a second kernel adds the blocks' partials
// (one block per gradient element, fixed-order tree).
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace optimus {

namespace {

constexpr int kGroups = kQkGroups;  // 16-lane groups per 256-thread block

__device__ __forceinline__ float group16_sum(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ void unpack8(const u32x4_t w, float (&x)[8]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[2 * e] = lo_bf(w[e]);
    x[2 * e + 1] = hi_bf(w[e]);
  }
}

__device__ __forceinline__ u32x4_t pack8f(const float (&x)[8]) {
  u32x4_t w;
#pragma unroll
  for (int e = 0; e < 4; ++e) w[e] = pack2(x[2 * e], x[2 * e + 1]);
  return w;
}

// Normalise one d-vector held as 8 elements per lane; returns mean and rstd.
template <int D>
__device__ __forceinline__ void norm8(float (&x)[8], bool act, float eps, const bf16_t *g, const bf16_t *b, int j,
                                      float &mean, float &rstd) {
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) s += act ? x[e] : 0.f;
  mean = group16_sum(s) / D;
  float v = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    x[e] -= mean;
    v += act ? x[e] * x[e] : 0.f;
  }
  rstd = 1.0f / sqrtf(group16_sum(v) / D + eps);
  if (act) {
    float gw[8], bw[8];
    unpack8(ldg16(g + j * 8), gw);
    unpack8(ldg16(b + j * 8), bw);
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = x[e] * rstd * gw[e] + bw[e];
  }
}

template <int D>
__global__ __launch_bounds__(256) void qk_norm_fwd_kernel(int pairs, int heads, const bf16_t *__restrict__ qkv,
                                                          const bf16_t *__restrict__ qg, const bf16_t *__restrict__ qb,
                                                          const bf16_t *__restrict__ kg, const bf16_t *__restrict__ kb,
                                                          float eps, bf16_t *__restrict__ qkvn,
                                                          float *__restrict__ stats) {
  const int p = (blockIdx.x * 256 + threadIdx.x) >> 4;
  const int j = threadIdx.x & 15;
  if (p >= pairs) return;  // whole 16-lane groups leave together
  const int row = p / heads, h = p % heads;
  const size_t A = static_cast<size_t>(heads) * D;
  const bool act = j < D / 8;
  const size_t base = static_cast<size_t>(row) * 3 * A + static_cast<size_t>(h) * D + j * 8;
  const u32x4_t z{0u, 0u, 0u, 0u};
  float q[8], k[8], qm, qr, km, kr;
  unpack8(act ? ldg16(qkv + base) : z, q);
  unpack8(act ? ldg16(qkv + base + A) : z, k);
  norm8<D>(q, act, eps, qg, qb, j, qm, qr);
  norm8<D>(k, act, eps, kg, kb, j, km, kr);
  if (act) {
    stg16(qkvn + base, pack8f(q));
    stg16(qkvn + base + A, pack8f(k));
    stg16(qkvn + base + 2 * A, ldg16(qkv + base + 2 * A));
  }
  if (j == 0) *reinterpret_cast<f32x4_t *>(stats + static_cast<size_t>(p) * 4) = f32x4_t{qm, qr, km, kr};
}

// LayerNorm backward of one d-vector; accumulates the lane's dgamma/dbeta.
template <int D>
__device__ __forceinline__ void norm8_bwd(const bf16_t *x_src, const bf16_t *dy_src, bf16_t *dx_dst, bool act,
                                          float mean, float rstd, const bf16_t *g, int j, float (&dg)[8],
                                          float (&db)[8]) {
  const u32x4_t z{0u, 0u, 0u, 0u};
  float x[8], dy[8], gw[8];
  unpack8(act ? ldg16(x_src) : z, x);
  unpack8(act ? ldg16(dy_src) : z, dy);
  unpack8(act ? ldg16(g + j * 8) : z, gw);
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    x[e] = (x[e] - mean) * rstd;  // xhat
    const float gh = dy[e] * gw[e];
    s1 += gh;
    s2 += gh * x[e];
    dg[e] += dy[e] * x[e];
    db[e] += dy[e];
  }
  s1 = group16_sum(s1) / D;
  s2 = group16_sum(s2) / D;
  if (act) {
    float dx[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) dx[e] = rstd * (dy[e] * gw[e] - s1 - x[e] * s2);
    stg16(dx_dst, pack8f(dx));
  }
}

template <int D>
__global__ __launch_bounds__(256) void qk_norm_bwd_kernel(int pairs, int heads, const bf16_t *__restrict__ dqkvn,
                                                          const bf16_t *__restrict__ qkv,
                                                          const float *__restrict__ stats,
                                                          const bf16_t *__restrict__ qg, const bf16_t *__restrict__ kg,
                                                          bf16_t *__restrict__ dqkv, float *__restrict__ part) {
  __shared__ float red[kGroups][4][128];
  const int gi = threadIdx.x >> 4, j = threadIdx.x & 15;
  const bool act = j < D / 8;
  const size_t A = static_cast<size_t>(heads) * D;
  float acc[4][8];
#pragma unroll
  for (int k = 0; k < 4; ++k)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[k][e] = 0.f;
  for (int p = blockIdx.x * kGroups + gi; p < pairs; p += gridDim.x * kGroups) {
    const int row = p / heads, h = p % heads;
    const size_t base = static_cast<size_t>(row) * 3 * A + static_cast<size_t>(h) * D + j * 8;
    const f32x4_t st = *reinterpret_cast<const f32x4_t *>(stats + static_cast<size_t>(p) * 4);
    norm8_bwd<D>(qkv + base, dqkvn + base, dqkv + base, act, st[0], st[1], qg, j, acc[0], acc[1]);
    norm8_bwd<D>(qkv + base + A, dqkvn + base + A, dqkv + base + A, act, st[2], st[3], kg, j, acc[2], acc[3]);
    if (act) stg16(dqkv + base + 2 * A, ldg16(dqkvn + base + 2 * A));
  }
  if (act) {
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int e = 0; e < 8; ++e) red[gi][k][j * 8 + e] = acc[k][e];
  }
  __syncthreads();
  for (int t = threadIdx.x; t < 4 * D; t += 256) {
    const int k = t / D, e = t % D;
    float s = 0.f;
#pragma unroll
    for (int g = 0; g < kGroups; ++g) s += red[g][k][e];
    part[(static_cast<size_t>(blockIdx.x) * 4 + k) * D + e] = s;
  }
}

// One block per affine-gradient element: strided partial sums over the
// blocks' partials, then a fixed-order tree in LDS (deterministic).
__global__ __launch_bounds__(256) void qk_norm_reduce_kernel(int blocks, int D, const float *__restrict__ part,
                                                             float *__restrict__ dqg, float *__restrict__ dqb,
                                                             float *__restrict__ dkg, float *__restrict__ dkb,
                                                             int accumulate) {
  __shared__ float red[256];
  const int k = blockIdx.x / D, e = blockIdx.x % D;
  float s = 0.f;
  for (int b = threadIdx.x; b < blocks; b += 256) s += part[(static_cast<size_t>(b) * 4 + k) * D + e];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    float *out = k == 0 ? dqg : k == 1 ? dqb : k == 2 ? dkg : dkb;
    out[e] = accumulate ? out[e] + red[0] : red[0];
  }
}

template <int D>
void fwd_d(int M, int heads, const bf16_t *qkv, const bf16_t *qg, const bf16_t *qb, const bf16_t *kg,
           const bf16_t *kb, float eps, bf16_t *qkvn, float *stats, hipStream_t s) {
  const int pairs = M * heads;
  hipLaunchKernelGGL(qk_norm_fwd_kernel<D>, dim3((pairs + kGroups - 1) / kGroups), dim3(256), 0, s, pairs, heads,
                     qkv, qg, qb, kg, kb, eps, qkvn, stats);
}

template <int D>
void bwd_d(int M, int heads, const bf16_t *dqkvn, const bf16_t *qkv, const float *stats, const bf16_t *qg,
           const bf16_t *kg, bf16_t *dqkv, float *dqg, float *dqb, float *dkg, float *dkb, int accumulate,
           float *part, hipStream_t s) {
  const int nb = qk_norm_bwd_blocks(M, heads);
  hipLaunchKernelGGL(qk_norm_bwd_kernel<D>, dim3(nb), dim3(256), 0, s, M * heads, heads, dqkvn, qkv, stats, qg, kg,
                     dqkv, part);
  hipLaunchKernelGGL(qk_norm_reduce_kernel, dim3(4 * D), dim3(256), 0, s, nb, D, part, dqg, dqb, dkg, dkb,
                     accumulate);
}

}  // namespace

bool launch_qk_norm_fwd(int M, int heads, int d, const bf16_t *qkv, const bf16_t *qg, const bf16_t *qb,
                        const bf16_t *kg, const bf16_t *kb, float eps, bf16_t *qkvn, float *stats, hipStream_t s) {
  switch (d) {
    case 64: fwd_d<64>(M, heads, qkv, qg, qb, kg, kb, eps, qkvn, stats, s); return true;
    case 80: fwd_d<80>(M, heads, qkv, qg, qb, kg, kb, eps, qkvn, stats, s); return true;
    case 128: fwd_d<128>(M, heads, qkv, qg, qb, kg, kb, eps, qkvn, stats, s); return true;
    default: return false;
  }
}

bool launch_qk_norm_bwd(int M, int heads, int d, const bf16_t *dqkvn, const bf16_t *qkv, const float *stats,
                        const bf16_t *qg, const bf16_t *kg, bf16_t *dqkv, float *dqg, float *dqb, float *dkg,
                        float *dkb, int accumulate, float *part, hipStream_t s) {
  switch (d) {
    case 64: bwd_d<64>(M, heads, dqkvn, qkv, stats, qg, kg, dqkv, dqg, dqb, dkg, dkb, accumulate, part, s); return true;
    case 80: bwd_d<80>(M, heads, dqkvn, qkv, stats, qg, kg, dqkv, dqg, dqb, dkg, dkb, accumulate, part, s); return true;
    case 128:
      bwd_d<128>(M, heads, dqkvn, qkv, stats, qg, kg, dqkv, dqg, dqb, dkg, dkb, accumulate, part, s);
      return true;
    default: return false;
  }
}

}  // namespace optimus
