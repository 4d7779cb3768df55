// LayerNorm forward and backward for gfx950.
//
// Forward: one wave per row, the row held in registers (16-byte loads, two
// passes over registers for mean and variance), no LDS and no barriers.
// Backward: one block per group of rows, each thread owning fixed 8-column
// chunks so that its dgamma/dbeta partial sums stay in registers across the
// rows; the per-block partials are summed in a fixed order by a second
// kernel, so the column sums are deterministic.
#include "common.hpp"
#include "kernels.hpp"

namespace optimus {

namespace {

template <int NCH>
__global__ __launch_bounds__(256) void ln_fwd_kernel(int rows, int cols, const bf16_t *__restrict__ x,
                                                     const bf16_t *__restrict__ gamma,
                                                     const bf16_t *__restrict__ beta, float eps,
                                                     bf16_t *__restrict__ y, float *__restrict__ mean,
                                                     float *__restrict__ rstd) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;  // whole wave leaves; the kernel has no barriers
  const int nch = cols >> 3;
  const bf16_t *xr = x + static_cast<size_t>(row) * cols;
  float v[NCH][8];
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int idx = lane + kWave * c;
    if (idx < nch) {
      u32x4_t w = ldg16(xr + idx * 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[c][2 * e] = lo_bf(w[e]);
        v[c][2 * e + 1] = hi_bf(w[e]);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) s += v[c][e];
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[c][e] = 0.f;
    }
  }
  const float inv_n = 1.0f / static_cast<float>(cols);
  const float mu = wave_sum(s) * inv_n;
  float q = 0.f;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    if (lane + kWave * c < nch) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = v[c][e] - mu;
        q += d * d;
      }
    }
  }
  const float var = wave_sum(q) * inv_n;
  const float r = 1.0f / sqrtf(var + eps);
  bf16_t *yr = y + static_cast<size_t>(row) * cols;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int idx = lane + kWave * c;
    if (idx < nch) {
      const u32x4_t gw = ldg16(gamma + idx * 8);
      const u32x4_t bw = ldg16(beta + idx * 8);
      u32x4_t o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float y0 = (v[c][2 * e] - mu) * r * lo_bf(gw[e]) + lo_bf(bw[e]);
        const float y1 = (v[c][2 * e + 1] - mu) * r * hi_bf(gw[e]) + hi_bf(bw[e]);
        o[e] = pack2(y0, y1);
      }
      stg16(yr + idx * 8, o);
    }
  }
  if (lane == 0) {
    mean[row] = mu;
    rstd[row] = r;
  }
}

constexpr int kLnBwdThreads = 256;

template <int CPT>
__global__ __launch_bounds__(kLnBwdThreads) void ln_bwd_kernel(
    int rows, int cols, const bf16_t *__restrict__ dy, const bf16_t *__restrict__ x,
    const float *__restrict__ mean, const float *__restrict__ rstd, const bf16_t *__restrict__ gamma,
    const bf16_t *__restrict__ dresid, bf16_t *__restrict__ dx, float *__restrict__ part) {
  __shared__ float red[2][kLnBwdThreads / kWave][2];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wid = tid >> 6;
  const int nch = cols >> 3;
  const float inv_n = 1.0f / static_cast<float>(cols);

  float g[CPT][8], pg[CPT][8], pb[CPT][8];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int idx = tid + kLnBwdThreads * c;
#pragma unroll
    for (int e = 0; e < 8; ++e) pg[c][e] = pb[c][e] = g[c][e] = 0.f;
    if (idx < nch) {
      const u32x4_t gw = ldg16(gamma + idx * 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        g[c][2 * e] = lo_bf(gw[e]);
        g[c][2 * e + 1] = hi_bf(gw[e]);
      }
    }
  }

  int parity = 0;
  for (int row = blockIdx.x; row < rows; row += gridDim.x, parity ^= 1) {
    const size_t off = static_cast<size_t>(row) * cols;
    const float mu = mean[row], r = rstd[row];
    float xh[CPT][8], gh[CPT][8];
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int idx = tid + kLnBwdThreads * c;
      if (idx < nch) {
        const u32x4_t dw = ldg16(dy + off + idx * 8);
        const u32x4_t xw = ldg16(x + off + idx * 8);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float d = (e & 1) ? hi_bf(dw[e >> 1]) : lo_bf(dw[e >> 1]);
          const float xv = (e & 1) ? hi_bf(xw[e >> 1]) : lo_bf(xw[e >> 1]);
          xh[c][e] = (xv - mu) * r;
          gh[c][e] = d * g[c][e];
          s1 += gh[c][e];
          s2 += gh[c][e] * xh[c][e];
          pg[c][e] += d * xh[c][e];
          pb[c][e] += d;
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) xh[c][e] = gh[c][e] = 0.f;
      }
    }
    s1 = wave_sum(s1);
    s2 = wave_sum(s2);
    if (lane == 0) {
      red[parity][wid][0] = s1;
      red[parity][wid][1] = s2;
    }
    __syncthreads();
    float t1 = 0.f, t2 = 0.f;
#pragma unroll
    for (int w = 0; w < kLnBwdThreads / kWave; ++w) {
      t1 += red[parity][w][0];
      t2 += red[parity][w][1];
    }
    const float c1 = t1 * inv_n, c2 = t2 * inv_n;
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int idx = tid + kLnBwdThreads * c;
      if (idx < nch) {
        float res[8];
        if (dresid) {
          const u32x4_t rw = ldg16(dresid + off + idx * 8);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            res[2 * e] = lo_bf(rw[e]);
            res[2 * e + 1] = hi_bf(rw[e]);
          }
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) res[e] = 0.f;
        }
        u32x4_t o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float a = res[2 * e] + r * (gh[c][2 * e] - c1 - xh[c][2 * e] * c2);
          const float b = res[2 * e + 1] + r * (gh[c][2 * e + 1] - c1 - xh[c][2 * e + 1] * c2);
          o[e] = pack2(a, b);
        }
        stg16(dx + off + idx * 8, o);
      }
    }
  }
  // Per-block partial column sums: part[0][blk][col] = dgamma, part[1][blk][col] = dbeta.
  float *pgam = part + static_cast<size_t>(blockIdx.x) * cols;
  float *pbet = part + (static_cast<size_t>(gridDim.x) + blockIdx.x) * cols;
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int idx = tid + kLnBwdThreads * c;
    if (idx < nch) {
#pragma unroll
      for (int e = 0; e < 8; e += 4) {
        *reinterpret_cast<f32x4_t *>(pgam + idx * 8 + e) = f32x4_t{pg[c][e], pg[c][e + 1], pg[c][e + 2], pg[c][e + 3]};
        *reinterpret_cast<f32x4_t *>(pbet + idx * 8 + e) = f32x4_t{pb[c][e], pb[c][e + 1], pb[c][e + 2], pb[c][e + 3]};
      }
    }
  }
}

// Fixed-order sum of the per-block partials: block = 64 columns x 4 row
// groups; each group sums every 4th partial row, then the four group sums
// are added in order.
__global__ __launch_bounds__(256) void ln_bwd_reduce_kernel(int nblk, int cols, const float *__restrict__ part,
                                                            float *__restrict__ dgamma,
                                                            float *__restrict__ dbeta, int accumulate) {
  __shared__ float red[2][4][64];
  const int tid = threadIdx.x;
  const int cl = tid & 63, grp = tid >> 6;
  const int col = blockIdx.x * 64 + cl;
  float sg = 0.f, sb = 0.f;
  if (col < cols) {
    for (int b = grp; b < nblk; b += 4) {
      sg += part[static_cast<size_t>(b) * cols + col];
      sb += part[(static_cast<size_t>(nblk) + b) * cols + col];
    }
  }
  red[0][grp][cl] = sg;
  red[1][grp][cl] = sb;
  __syncthreads();
  if (grp == 0 && col < cols) {
    float tg = ((red[0][0][cl] + red[0][1][cl]) + red[0][2][cl]) + red[0][3][cl];
    float tb = ((red[1][0][cl] + red[1][1][cl]) + red[1][2][cl]) + red[1][3][cl];
    if (accumulate) {
      tg += dgamma[col];
      tb += dbeta[col];
    }
    dgamma[col] = tg;
    dbeta[col] = tb;
  }
}

template <int NCH>
void launch_ln_fwd_n(int rows, int cols, const bf16_t *x, const bf16_t *gamma, const bf16_t *beta, float eps,
                     bf16_t *y, float *mean, float *rstd, hipStream_t s) {
  hipLaunchKernelGGL(ln_fwd_kernel<NCH>, dim3((rows + 3) / 4), dim3(256), 0, s, rows, cols, x, gamma, beta, eps, y,
                     mean, rstd);
}

template <int CPT>
void launch_ln_bwd_n(int nblk, int rows, int cols, const bf16_t *dy, const bf16_t *x, const float *mean,
                     const float *rstd, const bf16_t *gamma, const bf16_t *dresid, bf16_t *dx, float *part,
                     hipStream_t s) {
  hipLaunchKernelGGL(ln_bwd_kernel<CPT>, dim3(nblk), dim3(kLnBwdThreads), 0, s, rows, cols, dy, x, mean, rstd,
                     gamma, dresid, dx, part);
}

}  // namespace

int ln_bwd_blocks(int rows) { return rows < 256 ? rows : 256; }

size_t ln_bwd_ws_bytes(int rows, int cols) {
  return static_cast<size_t>(ln_bwd_blocks(rows)) * static_cast<size_t>(cols) * 2 * sizeof(float);
}

bool launch_ln_fwd(int rows, int cols, const bf16_t *x, const bf16_t *gamma, const bf16_t *beta, float eps,
                   bf16_t *y, float *mean, float *rstd, hipStream_t s) {
  const int need = ((cols >> 3) + kWave - 1) / kWave;  // 16-byte chunks per lane
#define OPT_LN_FWD(N) \
  if (need <= N) {    \
    launch_ln_fwd_n<N>(rows, cols, x, gamma, beta, eps, y, mean, rstd, s); \
    return true;      \
  }
  OPT_LN_FWD(1) OPT_LN_FWD(2) OPT_LN_FWD(3) OPT_LN_FWD(4) OPT_LN_FWD(6) OPT_LN_FWD(8)
  OPT_LN_FWD(12) OPT_LN_FWD(16) OPT_LN_FWD(24) OPT_LN_FWD(32)
#undef OPT_LN_FWD
  return false;
}

bool launch_ln_bwd(int rows, int cols, const bf16_t *dy, const bf16_t *x, const float *mean, const float *rstd,
                   const bf16_t *gamma, const bf16_t *dresid, bf16_t *dx, float *dgamma, float *dbeta,
                   int accumulate, float *part, hipStream_t s) {
  const int nblk = ln_bwd_blocks(rows);
  const int need = ((cols >> 3) + kLnBwdThreads - 1) / kLnBwdThreads;
  bool ok = false;
#define OPT_LN_BWD(N)                                                                       \
  if (!ok && need <= N) {                                                                  \
    launch_ln_bwd_n<N>(nblk, rows, cols, dy, x, mean, rstd, gamma, dresid, dx, part, s);   \
    ok = true;                                                                             \
  }
  OPT_LN_BWD(1) OPT_LN_BWD(2) OPT_LN_BWD(3) OPT_LN_BWD(4) OPT_LN_BWD(6) OPT_LN_BWD(8)
#undef OPT_LN_BWD
  if (!ok) return false;
  hipLaunchKernelGGL(ln_bwd_reduce_kernel, dim3((cols + 63) / 64), dim3(256), 0, s, nblk, cols, part, dgamma, dbeta,
                     accumulate);
  return true;
}

}  // namespace optimus
