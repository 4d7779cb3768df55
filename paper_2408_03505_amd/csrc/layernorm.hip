// LayerNorm forward and backward for gfx950 (HBM-bound).
//
// Rows are processed by TPR threads each (one wave for rows up to 4096 wide,
// a whole 256-thread block beyond), every thread holding CPT 16-byte chunks
// of the row in registers: one read and one write of every element, two
// reductions per row (a wave butterfly, plus an LDS exchange across the four
// waves when TPR = 256).
//
// The backward is two kernels: one pass over the rows that writes dx and
// per-block column sums of dy * xhat and dy, and a fixed-order sum of those
// partials, so dgamma and dbeta are deterministic.
#include "common.hpp"
#include "kernels.hpp"

namespace optimus {

namespace {

constexpr int kThreads = kLnThreads;

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

// Backward, one pass over the rows.  Each block owns a contiguous range of
// rows and walks it RG rows at a time (one row per TPR-thread group), with the
// next row's loads in flight while the current row is reduced:
//   dx = dresid + rstd * (ghat - mean(ghat) - xhat * mean(ghat * xhat)),
//   ghat = dy * gamma.
// Every thread keeps the column sums of dy * xhat and dy for its own columns
// over the block's rows; the RG groups' sums are added in a fixed order
// through LDS and the block writes one row of partials per gradient, which a
// second kernel sums in a fixed order (deterministic dgamma / dbeta).
// Blocks (partial rows) of the backward pass: one per CU.  Measured at
// 2048 x 6144: 512, 1024 and 2048 blocks are slower (the partials grow with
// the block count), and so is loading two rows ahead instead of one.
constexpr int kBwdBlocks = kLnBwdBlocks;

template <int TPR, int CPT, bool RES>
__global__ __launch_bounds__(kThreads) void ln_bwd_kernel(int rows, int cols, int rows_per_block,
                                                    const bf16_t *__restrict__ dy, const bf16_t *__restrict__ x,
                                                    const float *__restrict__ mean, const float *__restrict__ rstd,
                                                    const bf16_t *__restrict__ gamma,
                                                    const bf16_t *__restrict__ dresid, bf16_t *__restrict__ dx,
                                                    float *__restrict__ part) {
  constexpr int RG = kThreads / TPR;  // row groups: rows in flight per block
  __shared__ float red[kThreads / 64][2];
  extern __shared__ __attribute__((aligned(16))) float comb[];  // [2][cols]
  const int t = threadIdx.x % TPR, g = threadIdx.x / TPR;
  const int wid = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nch = cols >> 3;
  const int r_begin = blockIdx.x * rows_per_block;
  const int r_end = min(rows, r_begin + rows_per_block);
  // every group runs the same number of iterations (the block-wide barriers
  // of TPR = 256 are reached by all threads); rows past r_end are masked
  const int iters = (r_end - r_begin + RG - 1) / RG;

  // This thread's chunks: idx[c] is clamped into the row so that every load
  // is unconditional (the compiler can then count loads in flight exactly and
  // wait for the current row only); chunks past the row end are masked at use.
  int idx[CPT];
  unsigned in_row = 0;
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int i = t + TPR * c;
    idx[c] = min(i, nch - 1);
    if (i < nch) in_row |= 1u << c;
  }

  float gm[CPT][8], sg[CPT][8], sb[CPT][8];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    unpack8(ldg16(gamma + idx[c] * 8), gm[c]);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (!((in_row >> c) & 1u)) gm[c][e] = 0.f;
      sg[c][e] = sb[c][e] = 0.f;
    }
  }

  // Row r's data and statistics (a row past r_end reads row r_end - 1, and
  // its statistics are zeroed at use).  The statistics come with the row:
  // loads retire in issue order, so loading them later would also wait for
  // the row loaded ahead.
  auto load = [&](int r, u32x4_t(&d)[CPT], u32x4_t(&xv)[CPT], u32x4_t(&res)[CPT], float &mu, float &rs) {
    const int rr = min(r, r_end - 1);
    const size_t off = static_cast<size_t>(rr) * cols;
    mu = mean[rr];
    rs = rstd[rr];
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      d[c] = ldg16(dy + off + idx[c] * 8);
      xv[c] = ldg16(x + off + idx[c] * 8);
      if constexpr (RES) res[c] = ldg16(dresid + off + idx[c] * 8);
    }
  };
  // sum over the TPR threads of this group (wave butterfly, then LDS across
  // the group's four waves when TPR = 256)
  auto group_sum = [&](float (&v)[2]) {
#pragma unroll
    for (int k = 0; k < 2; ++k) v[k] = wave_sum(v[k]);
    if constexpr (TPR == 256) {
      if (lane == 0) {
        red[wid][0] = v[0];
        red[wid][1] = v[1];
      }
      lds_barrier();  // the next row's loads stay in flight
      const int w0 = g * 4;
#pragma unroll
      for (int k = 0; k < 2; ++k) v[k] = ((red[w0][k] + red[w0 + 1][k]) + red[w0 + 2][k]) + red[w0 + 3][k];
      lds_barrier();
    }
  };

  const float inv_n = 1.0f / static_cast<float>(cols);
  // One row: column sums, the row reduction, dx.  Rows past r_end are masked.
  auto row = [&](int r, const u32x4_t(&cd)[CPT], const u32x4_t(&cx)[CPT], const u32x4_t(&cr)[CPT], float mu,
                 float rs) {
    const bool live = r < r_end;
    const unsigned mask = live ? in_row : 0u;
    if (!live) mu = rs = 0.f;
    float s[2] = {0.f, 0.f};
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      float d[8], xv[8];
      unpack8(cd[c], d);
      unpack8(cx[c], xv);
      const bool in = (mask >> c) & 1u;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // masked chunks contribute dy = 0: they add nothing
        const float dv = in ? d[e] : 0.f;
        const float xh = (xv[e] - mu) * rs, gh = dv * gm[c][e];
        s[0] += gh;
        s[1] += gh * xh;
        sg[c][e] += dv * xh;
        sb[c][e] += dv;
      }
    }
    group_sum(s);
    const float c1 = s[0] * inv_n, c2 = s[1] * inv_n;
    const size_t off = static_cast<size_t>(r) * cols;
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      if ((mask >> c) & 1u) {
        // xhat and ghat again from the row still in registers
        float d[8], xv[8], res[8], o8[8];
        unpack8(cd[c], d);
        unpack8(cx[c], xv);
        if constexpr (RES) {
          unpack8(cr[c], res);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) res[e] = 0.f;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float xh = (xv[e] - mu) * rs, gh = d[e] * gm[c][e];
          o8[e] = res[e] + rs * (gh - c1 - xh * c2);
        }
        u32x4_t o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = pack2(o8[2 * e], o8[2 * e + 1]);
        stg16(dx + off + idx[c] * 8, o);
      }
    }
  };

  if constexpr (CPT <= 4) {
    // Two register buffers in turn: each row's loads are issued one row ahead
    // (no register copies between iterations, which would wait for them).
    // Pairs of iterations; an odd last one runs on a masked row.
    u32x4_t d0[CPT], x0[CPT], q0[CPT], d1[CPT], x1[CPT], q1[CPT];
    float mu0, rs0, mu1, rs1;
    load(r_begin + g, d0, x0, q0, mu0, rs0);
    for (int it = 0; it < iters; it += 2) {
      const int r = r_begin + g + it * RG;
      load(r + RG, d1, x1, q1, mu1, rs1);
      row(r, d0, x0, q0, mu0, rs0);
      load(r + 2 * RG, d0, x0, q0, mu0, rs0);
      row(r + RG, d1, x1, q1, mu1, rs1);
    }
  } else {
    // wide rows: no room for a second row in registers
    u32x4_t d0[CPT], x0[CPT], q0[CPT];
    float mu0, rs0;
    for (int it = 0; it < iters; ++it) {
      const int r = r_begin + g + it * RG;
      load(r, d0, x0, q0, mu0, rs0);
      row(r, d0, x0, q0, mu0, rs0);
    }
  }

  // groups 1..RG-1 hand their column sums to group 0, one at a time
#pragma unroll 1
  for (int h = 1; h < RG; ++h) {
    __syncthreads();
    if (g == h) {
#pragma unroll
      for (int c = 0; c < CPT; ++c) {
        if ((in_row >> c) & 1u)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            comb[idx[c] * 8 + e] = sg[c][e];
            comb[cols + idx[c] * 8 + e] = sb[c][e];
          }
      }
    }
    __syncthreads();
    if (g == 0) {
#pragma unroll
      for (int c = 0; c < CPT; ++c) {
        if ((in_row >> c) & 1u)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            sg[c][e] += comb[idx[c] * 8 + e];
            sb[c][e] += comb[cols + idx[c] * 8 + e];
          }
      }
    }
  }
  if (g == 0) {
    float *pg = part + static_cast<size_t>(blockIdx.x) * cols;
    float *pb = part + (static_cast<size_t>(gridDim.x) + blockIdx.x) * cols;
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      if ((in_row >> c) & 1u) {
        const int i8 = idx[c] * 8;
        *reinterpret_cast<f32x4_t *>(pg + i8) = f32x4_t{sg[c][0], sg[c][1], sg[c][2], sg[c][3]};
        *reinterpret_cast<f32x4_t *>(pg + i8 + 4) = f32x4_t{sg[c][4], sg[c][5], sg[c][6], sg[c][7]};
        *reinterpret_cast<f32x4_t *>(pb + i8) = f32x4_t{sb[c][0], sb[c][1], sb[c][2], sb[c][3]};
        *reinterpret_cast<f32x4_t *>(pb + i8 + 4) = f32x4_t{sb[c][4], sb[c][5], sb[c][6], sb[c][7]};
      }
    }
  }
}

// dgamma (blockIdx.y 0) or dbeta (1) (+)= the fixed-order sum of the nblk
// partial rows.  Block = 64 columns (8 chunks of 8) x 32 groups of partial
// rows; the 32 group sums are added in a fixed order through LDS.
constexpr int kRedCols = 64, kRedGroups = 32;

__global__ __launch_bounds__(kThreads) void ln_bwd_reduce_kernel(int nblk, int cols, const float *__restrict__ part,
                                                                 float *__restrict__ dgamma,
                                                                 float *__restrict__ dbeta, int accumulate) {
  __shared__ float red[kRedGroups][kRedCols + 1];
  const int chunk = threadIdx.x & 7, grp = threadIdx.x >> 3;
  const int c0 = blockIdx.x * kRedCols + chunk * 8;
  const float *src = part + static_cast<size_t>(blockIdx.y) * nblk * cols;
  float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (c0 < cols) {
#pragma unroll 4
    for (int b = grp; b < nblk; b += kRedGroups) {
      const float *q = src + static_cast<size_t>(b) * cols + c0;
      const f32x4_t a = *reinterpret_cast<const f32x4_t *>(q);
      const f32x4_t c = *reinterpret_cast<const f32x4_t *>(q + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[e] += a[e];
        v[4 + e] += c[e];
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[grp][chunk * 8 + e] = v[e];
  __syncthreads();
  if (threadIdx.x < kRedCols) {
    const int col = blockIdx.x * kRedCols + threadIdx.x;
    float tsum = 0.f;
#pragma unroll 8
    for (int q = 0; q < kRedGroups; ++q) tsum += red[q][threadIdx.x];
    if (col < cols) {
      float *out = blockIdx.y == 0 ? dgamma : dbeta;
      out[col] = accumulate ? out[col] + tsum : tsum;
    }
  }
}

}  // namespace

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
  const int nch = cols >> 3;
  const int tpr = ln_bwd_tpr(cols);
  const int rpb = ln_bwd_rows_per_block(rows, cols);
  const int nblk = (rows + rpb - 1) / rpb;
  const dim3 grid(nblk);
  // LDS for the hand-over of column sums between the row groups of a block
  const size_t comb = tpr < kThreads ? static_cast<size_t>(cols) * 2 * sizeof(float) : 0;
#define OPT_LN_BWD(T, C)                                                                                       \
  do {                                                                                                          \
    if (dresid)                                                                                                 \
      hipLaunchKernelGGL((ln_bwd_kernel<T, C, true>), grid, dim3(kThreads), comb, s, rows, cols, rpb, dy, x,      \
                         mean, rstd, gamma, dresid, dx, part);                                                  \
    else                                                                                                        \
      hipLaunchKernelGGL((ln_bwd_kernel<T, C, false>), grid, dim3(kThreads), comb, s, rows, cols, rpb, dy, x,     \
                         mean, rstd, gamma, dresid, dx, part);                                                  \
  } while (0)
  if (tpr == 256) {
    const int cpt = (nch + 255) / 256;
    if (cpt <= 2) OPT_LN_BWD(256, 2);
    else if (cpt <= 3) OPT_LN_BWD(256, 3);
    else if (cpt <= 4) OPT_LN_BWD(256, 4);
    else if (cpt <= 6) OPT_LN_BWD(256, 6);
    else if (cpt <= 8) OPT_LN_BWD(256, 8);
    else return false;
  } else {
    const int cpt = (nch + 63) / 64;
    if (cpt <= 1) OPT_LN_BWD(64, 1);
    else if (cpt <= 2) OPT_LN_BWD(64, 2);
    else if (cpt <= 3) OPT_LN_BWD(64, 3);
    else OPT_LN_BWD(64, 4);
  }
#undef OPT_LN_BWD
  hipLaunchKernelGGL(ln_bwd_reduce_kernel, dim3((cols + kRedCols - 1) / kRedCols, 2), dim3(kThreads), 0, s, nblk, cols,
                     part, dgamma, dbeta, accumulate);
  return true;
}

#undef OPT_LN_DISPATCH

}  // namespace optimus
