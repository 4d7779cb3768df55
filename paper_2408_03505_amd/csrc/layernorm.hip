// LayerNorm forward and backward for gfx950 (HBM-bound).
//
// Rows are processed by TPR threads each (one wave for rows up to 4096 wide,
// a whole 256-thread block beyond), every thread holding CPT 16-byte chunks
// of the row in registers: one read and one write of every element, two
// reductions per row (a wave butterfly, plus an LDS exchange across the four
// waves when TPR = 256).
//
// The backward is three kernels: dx (row-parallel, like the forward), the
// column partial sums of dy * xhat and dy over row chunks (column-tiled with
// 16-byte loads), and a fixed-order sum of those partials, so dgamma and
// dbeta are deterministic.
#include "common.hpp"
#include "kernels.hpp"

namespace optimus {

namespace {

constexpr int kThreads = 256;

// Sum over the TPR threads that share a row (TPR = 64 or 256).
template <int TPR, int NV>
__device__ __forceinline__ void row_sum(float (&v)[NV], float (*red)[4][NV]) {
#pragma unroll
  for (int k = 0; k < NV; ++k) v[k] = wave_sum(v[k]);
  if constexpr (TPR == 256) {
    const int wid = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0)
#pragma unroll
      for (int k = 0; k < NV; ++k) (*red)[wid][k] = v[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < NV; ++k) v[k] = (((*red)[0][k] + (*red)[1][k]) + (*red)[2][k]) + (*red)[3][k];
    __syncthreads();
  }
}

__device__ __forceinline__ void unpack8(const u32x4_t w, float (&f)[8]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    f[2 * e] = lo_bf(w[e]);
    f[2 * e + 1] = hi_bf(w[e]);
  }
}

template <int TPR, int CPT>
__global__ __launch_bounds__(kThreads) void ln_fwd_kernel(int rows, int cols, const bf16_t *__restrict__ x,
                                                          const bf16_t *__restrict__ gamma,
                                                          const bf16_t *__restrict__ beta, float eps,
                                                          bf16_t *__restrict__ y, float *__restrict__ mean,
                                                          float *__restrict__ rstd) {
  __shared__ float red[2][4][1];
  constexpr int RPB = kThreads / TPR;  // rows per block
  const int t = threadIdx.x % TPR;
  const int row = blockIdx.x * RPB + threadIdx.x / TPR;
  // TPR == 256 blocks are one row: the whole block takes the same branch.
  if (row >= rows) return;
  const int nch = cols >> 3;
  const size_t off = static_cast<size_t>(row) * cols;
  float v[CPT][8];
  float s[1] = {0.f};
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int idx = t + TPR * c;
    if (idx < nch) {
      unpack8(ldg16(x + off + idx * 8), v[c]);
#pragma unroll
      for (int e = 0; e < 8; ++e) s[0] += v[c][e];
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[c][e] = 0.f;
    }
  }
  row_sum<TPR, 1>(s, &red[0]);
  const float inv_n = 1.0f / static_cast<float>(cols);
  const float mu = s[0] * inv_n;
  float q[1] = {0.f};
#pragma unroll
  for (int c = 0; c < CPT; ++c)
    if (t + TPR * c < nch)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = v[c][e] - mu;
        q[0] += d * d;
      }
  row_sum<TPR, 1>(q, &red[1]);
  const float r = 1.0f / sqrtf(q[0] * inv_n + eps);
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int idx = t + TPR * c;
    if (idx < nch) {
      float g[8], b[8];
      unpack8(ldg16(gamma + idx * 8), g);
      unpack8(ldg16(beta + idx * 8), b);
      u32x4_t o;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        o[e] = pack2((v[c][2 * e] - mu) * r * g[2 * e] + b[2 * e], (v[c][2 * e + 1] - mu) * r * g[2 * e + 1] + b[2 * e + 1]);
      stg16(y + off + idx * 8, o);
    }
  }
  if (t == 0) {
    mean[row] = mu;
    rstd[row] = r;
  }
}

// dx = dresid + rstd * (ghat - mean(ghat) - xhat * mean(ghat * xhat)), ghat = dy * gamma
template <int TPR, int CPT>
__global__ __launch_bounds__(kThreads) void ln_bwd_dx_kernel(int rows, int cols, const bf16_t *__restrict__ dy,
                                                             const bf16_t *__restrict__ x,
                                                             const float *__restrict__ mean,
                                                             const float *__restrict__ rstd,
                                                             const bf16_t *__restrict__ gamma,
                                                             const bf16_t *__restrict__ dresid,
                                                             bf16_t *__restrict__ dx) {
  __shared__ float red[4][2];
  constexpr int RPB = kThreads / TPR;
  const int t = threadIdx.x % TPR;
  const int row = blockIdx.x * RPB + threadIdx.x / TPR;
  if (row >= rows) return;
  const int nch = cols >> 3;
  const size_t off = static_cast<size_t>(row) * cols;
  const float mu = mean[row], r = rstd[row];
  float xh[CPT][8], gh[CPT][8];
  float s[2] = {0.f, 0.f};
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int idx = t + TPR * c;
    if (idx < nch) {
      float d[8], xv[8], g[8];
      unpack8(ldg16(dy + off + idx * 8), d);
      unpack8(ldg16(x + off + idx * 8), xv);
      unpack8(ldg16(gamma + idx * 8), g);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        xh[c][e] = (xv[e] - mu) * r;
        gh[c][e] = d[e] * g[e];
        s[0] += gh[c][e];
        s[1] += gh[c][e] * xh[c][e];
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) xh[c][e] = gh[c][e] = 0.f;
    }
  }
  row_sum<TPR, 2>(s, &red);
  const float inv_n = 1.0f / static_cast<float>(cols);
  const float c1 = s[0] * inv_n, c2 = s[1] * inv_n;
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int idx = t + TPR * c;
    if (idx < nch) {
      float res[8];
      if (dresid)
        unpack8(ldg16(dresid + off + idx * 8), res);
      else
#pragma unroll
        for (int e = 0; e < 8; ++e) res[e] = 0.f;
      u32x4_t o;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        o[e] = pack2(res[2 * e] + r * (gh[c][2 * e] - c1 - xh[c][2 * e] * c2),
                     res[2 * e + 1] + r * (gh[c][2 * e + 1] - c1 - xh[c][2 * e + 1] * c2));
      stg16(dx + off + idx * 8, o);
    }
  }
}

// Column partial sums over one chunk of rows: part[0][chunk][col] = sum dy * xhat,
// part[1][chunk][col] = sum dy.  Block = 64 columns (8 chunks of 8) x 32 row
// groups; the 32 group sums are added in a fixed order through LDS.
constexpr int kParamCols = 64, kParamGroups = 32;

__global__ __launch_bounds__(kThreads) void ln_bwd_param_kernel(int rows, int cols, int rows_per_chunk,
                                                                const bf16_t *__restrict__ dy,
                                                                const bf16_t *__restrict__ x,
                                                                const float *__restrict__ mean,
                                                                const float *__restrict__ rstd,
                                                                float *__restrict__ part) {
  __shared__ float red[2][kParamGroups][kParamCols + 1];
  const int chunk = threadIdx.x & 7, grp = threadIdx.x >> 3;
  const int c0 = blockIdx.x * kParamCols + chunk * 8;
  const int r_begin = blockIdx.y * rows_per_chunk;
  const int r_end = min(rows, r_begin + rows_per_chunk);
  float sg[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f}, sb[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (c0 < cols) {
#pragma unroll 2
    for (int r = r_begin + grp; r < r_end; r += kParamGroups) {
      const size_t off = static_cast<size_t>(r) * cols + c0;
      float d[8], xv[8];
      unpack8(ldg16(dy + off), d);
      unpack8(ldg16(x + off), xv);
      const float mu = mean[r], rs = rstd[r];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        sg[e] += d[e] * ((xv[e] - mu) * rs);
        sb[e] += d[e];
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    red[0][grp][chunk * 8 + e] = sg[e];
    red[1][grp][chunk * 8 + e] = sb[e];
  }
  __syncthreads();
  if (threadIdx.x < 2 * kParamCols) {
    const int which = threadIdx.x / kParamCols, cl = threadIdx.x % kParamCols;
    const int col = blockIdx.x * kParamCols + cl;
    float tsum = 0.f;
#pragma unroll 8
    for (int g = 0; g < kParamGroups; ++g) tsum += red[which][g][cl];
    if (col < cols) part[(static_cast<size_t>(which) * gridDim.y + blockIdx.y) * cols + col] = tsum;
  }
}

// dgamma/dbeta (+)= fixed-order sum of the row-chunk partials.
__global__ __launch_bounds__(kThreads) void ln_bwd_reduce_kernel(int nchunks, int cols, const float *__restrict__ part,
                                                                 float *__restrict__ dgamma,
                                                                 float *__restrict__ dbeta, int accumulate) {
  const int col = blockIdx.x * kThreads + threadIdx.x;
  if (col >= cols) return;
  float g = 0.f, b = 0.f;
  for (int c = 0; c < nchunks; ++c) {
    g += part[static_cast<size_t>(c) * cols + col];
    b += part[(static_cast<size_t>(nchunks) + c) * cols + col];
  }
  if (accumulate) {
    g += dgamma[col];
    b += dbeta[col];
  }
  dgamma[col] = g;
  dbeta[col] = b;
}

// Row chunks of the parameter-gradient pass: about four blocks per CU.
int param_chunks(int rows, int cols) {
  const int col_blocks = (cols + kParamCols - 1) / kParamCols;
  int chunks = (1024 + col_blocks - 1) / col_blocks;
  const int max_chunks = (rows + kParamGroups - 1) / kParamGroups;  // keep >= 32 rows per chunk
  if (chunks > max_chunks) chunks = max_chunks;
  return chunks < 1 ? 1 : chunks;
}

}  // namespace

size_t ln_bwd_ws_bytes(int rows, int cols) {
  return static_cast<size_t>(param_chunks(rows, cols)) * static_cast<size_t>(cols) * 2 * sizeof(float);
}

#define OPT_LN_DISPATCH(KERNEL, ...)                                                                           \
  do {                                                                                                          \
    const int nch = cols >> 3;                                                                                  \
    if (nch > 512) {                                                                                            \
      const int cpt = (nch + 255) / 256;                                                                        \
      const dim3 grid(rows);                                                                                    \
      if (cpt <= 2) hipLaunchKernelGGL((KERNEL<256, 2>), grid, dim3(kThreads), 0, s, __VA_ARGS__);             \
      else if (cpt <= 3) hipLaunchKernelGGL((KERNEL<256, 3>), grid, dim3(kThreads), 0, s, __VA_ARGS__);        \
      else if (cpt <= 4) hipLaunchKernelGGL((KERNEL<256, 4>), grid, dim3(kThreads), 0, s, __VA_ARGS__);        \
      else if (cpt <= 6) hipLaunchKernelGGL((KERNEL<256, 6>), grid, dim3(kThreads), 0, s, __VA_ARGS__);        \
      else if (cpt <= 8) hipLaunchKernelGGL((KERNEL<256, 8>), grid, dim3(kThreads), 0, s, __VA_ARGS__);        \
      else return false;                                                                                        \
    } else {                                                                                                    \
      const int cpt = (nch + 63) / 64;                                                                          \
      const dim3 grid((rows + 3) / 4);                                                                          \
      if (cpt <= 1) hipLaunchKernelGGL((KERNEL<64, 1>), grid, dim3(kThreads), 0, s, __VA_ARGS__);              \
      else if (cpt <= 2) hipLaunchKernelGGL((KERNEL<64, 2>), grid, dim3(kThreads), 0, s, __VA_ARGS__);         \
      else if (cpt <= 3) hipLaunchKernelGGL((KERNEL<64, 3>), grid, dim3(kThreads), 0, s, __VA_ARGS__);         \
      else if (cpt <= 4) hipLaunchKernelGGL((KERNEL<64, 4>), grid, dim3(kThreads), 0, s, __VA_ARGS__);         \
      else if (cpt <= 6) hipLaunchKernelGGL((KERNEL<64, 6>), grid, dim3(kThreads), 0, s, __VA_ARGS__);         \
      else if (cpt <= 8) hipLaunchKernelGGL((KERNEL<64, 8>), grid, dim3(kThreads), 0, s, __VA_ARGS__);         \
      else return false;                                                                                        \
    }                                                                                                           \
  } while (0)

bool launch_ln_fwd(int rows, int cols, const bf16_t *x, const bf16_t *gamma, const bf16_t *beta, float eps,
                   bf16_t *y, float *mean, float *rstd, hipStream_t s) {
  OPT_LN_DISPATCH(ln_fwd_kernel, rows, cols, x, gamma, beta, eps, y, mean, rstd);
  return true;
}

bool launch_ln_bwd(int rows, int cols, const bf16_t *dy, const bf16_t *x, const float *mean, const float *rstd,
                   const bf16_t *gamma, const bf16_t *dresid, bf16_t *dx, float *dgamma, float *dbeta,
                   int accumulate, float *part, hipStream_t s) {
  OPT_LN_DISPATCH(ln_bwd_dx_kernel, rows, cols, dy, x, mean, rstd, gamma, dresid, dx);
  const int chunks = param_chunks(rows, cols);
  const int rpc = (rows + chunks - 1) / chunks;
  hipLaunchKernelGGL(ln_bwd_param_kernel, dim3((cols + kParamCols - 1) / kParamCols, chunks), dim3(kThreads), 0, s,
                     rows, cols, rpc, dy, x, mean, rstd, part);
  hipLaunchKernelGGL(ln_bwd_reduce_kernel, dim3((cols + kThreads - 1) / kThreads), dim3(kThreads), 0, s, chunks, cols,
                     part, dgamma, dbeta, accumulate);
  return true;
}

#undef OPT_LN_DISPATCH

}  // namespace optimus
