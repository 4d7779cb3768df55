// bf16 MFMA GEMM family for the four projections of the encoder layer, in
// their forward, input-gradient and weight-gradient forms.
//
//   C[m, n] = sum_k A(m, k) * B(n, k),  fp32 accumulation on
//   v_mfma_f32_32x32x16_bf16.
//
// Operands whose contraction index is contiguous in memory (activations in
// the forward, weights [out, in] in the forward) are copied to LDS with
// 16-byte loads.  Operands whose contraction index is strided (the weight in
// the input gradient, both operands of the weight gradient) are read as 8x8
// bf16 blocks, transposed in registers with v_perm_b32 and written to LDS so
// that every LDS tile is [row][k] with k contiguous; all MFMA operand reads
// are then 16-byte ds_read_b128 from rows padded by 16 bytes (conflict-free
// for 8 consecutive lanes).  Tiles are double-buffered in LDS with one
// barrier per k-step; the next tile's global loads are issued before the
// current tile's MFMAs.
//
// The MFMA is issued as D = Btile * Atile^T so that each lane of the 32x32
// result owns one output row m and four consecutive output columns n: the
// bf16 epilogue stores 8 bytes and the fp32 epilogue 16 bytes per access.
// Epilogues fuse bias, residual, GELU (writing both pre- and post-activation),
// GELU' (for the MLP input gradient) and, for weight gradients, the bias
// gradient as row sums of the transposed A operand (deterministic).
//
// Workgroup order is XCD-aware: MI355X dispatches workgroup i to XCD i % 8,
// so each XCD is given its own block of the tile grid, walked M-fastest in
// groups of row tiles, which keeps the operand panels it shares in its L2.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"
#include "lds_dma.hpp"

namespace optimus {

namespace {

// 1 + erf(x) for the GELU epilogues, from Abramowitz & Stegun, Handbook of
// Mathematical Functions (1964), formula 7.1.26: for x >= 0,
// erfc(x) = (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) e^(-x^2) with
// t = 1 / (1 + p x), absolute error <= 1.5e-7.  Then 1 + erf(x) is 2 - erfc(x)
// for x >= 0 and erfc(-x) for x < 0, so the negative side does not cancel in
// fp32.  On the hardware reciprocal and exponential this is a fraction of the
// library erff's instructions; the epilogue evaluates it for every output
// element, and results are rounded to bf16.  Also returns e^(-x^2), which
// GELU' needs as well.
__device__ __forceinline__ float one_plus_erf(float x, float &ex2) {
  const float ax = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(1.0f + 0.3275911f * ax);
  const float poly =
      t * (0.254829592f + t * (-0.284496736f + t * (1.421413741f + t * (-1.453152027f + t * 1.061405429f))));
  ex2 = __builtin_amdgcn_exp2f(-(ax * ax) * 1.4426950408889634f);
  const float erfc_ax = poly * ex2;
  return x >= 0.0f ? 2.0f - erfc_ax : erfc_ax;
}

// GELU(u) = u Phi(u) and GELU'(u) = Phi(u) + u phi(u), with
// Phi(u) = (1 + erf(u / sqrt 2)) / 2 and phi(u) = e^(-u^2 / 2) / sqrt(2 pi).
__device__ __forceinline__ float gelu_f(float u) {
  float ex2;
  return 0.5f * u * one_plus_erf(u * 0.70710678118654752f, ex2);
}

__device__ __forceinline__ float gelu_grad_f(float u) {
  float ex2;  // e^(-u^2 / 2)
  const float Phi = 0.5f * one_plus_erf(u * 0.70710678118654752f, ex2);
  return Phi + u * ex2 * 0.39894228040143268f;
}

// Logical tile for this workgroup.  MI355X dispatches workgroup i to XCD
// i % 8.  When the tile grid splits evenly, the XCDs form two halves along
// M, the four XCDs of a half split its column tiles, and each XCD walks its
// block of tiles in groups of 4 row tiles that sweep the block's columns.
// Otherwise each XCD takes one contiguous range of logical tiles, grouped by
// 8 row tiles.  (Measured on the twelve ViT-22B layer GEMMs: 0.7% less time
// in total than the contiguous order, from 5% on the MLP-up weight gradient
// to -2% on the QKV weight gradient.)
__device__ __forceinline__ void tile_of(int pid, int nb, int tiles_m, int tiles_n, int &tm, int &tn) {
  const int xcd = pid & 7, local = pid >> 3;
  if (tiles_m % 2 == 0 && tiles_n % 4 == 0) {
    constexpr int GM = 4;
    const int rows_p = tiles_m / 2, cols_x = tiles_n / 4;
    const int gs = GM * cols_x;
    const int g = local / gs, first_m = g * GM;
    const int gm = min(rows_p - first_m, GM);
    const int in_g = local - g * gs;
    tm = (xcd >> 2) * rows_p + first_m + in_g % gm;
    tn = (xcd & 3) * cols_x + in_g / gm;
    return;
  }
  const int per = nb >> 3, rem = nb & 7;
  const int logical = (xcd < rem) ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
  constexpr int GROUP_M = 8;
  const int group_size = GROUP_M * tiles_n;
  const int g = logical / group_size;
  const int first_m = g * GROUP_M;
  const int gm = min(tiles_m - first_m, GROUP_M);
  const int in_g = logical - g * group_size;
  tm = first_m + in_g % gm;
  tn = in_g / gm;
}

__device__ __forceinline__ void tile_of(int tiles_m, int tiles_n, int &tm, int &tn) {
  tile_of(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
}

// Split of the contraction handled by this workgroup.  With p.splits > 1 the
// grid holds splits x tiles work items, listed split-major and M-fastest
// within a split; each XCD (workgroup i runs on XCD i % 8) takes one
// contiguous range of that list, so the items on one XCD mostly share a
// split and with it the operand panels of its k-range (the tiles of one
// tile column share the weight-gradient rows' panel, those of one tile row
// the other operand's).  Returns the split; kbeg/klen give its contraction
// range.
__device__ __forceinline__ int split_of(const GemmArgs &p, int tiles_m, int tiles_n, int &tm, int &tn, int &kbeg,
                                       int &klen) {
  if (p.splits > 1) {
    const int nt = tiles_m * tiles_n;
    const int pid = blockIdx.x, nb = gridDim.x;
    const int xcd = pid & 7, local = pid >> 3, per = nb >> 3, rem = nb & 7;
    const int item = (xcd < rem) ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
    const int split = item / nt, t = item - split * nt;
    tm = t % tiles_m;
    tn = t / tiles_m;
    kbeg = split * p.k_chunk;
    klen = min(p.K - kbeg, p.k_chunk);
    return split;
  }
  tile_of(tiles_m, tiles_n, tm, tn);
  kbeg = 0;
  klen = p.K;
  return 0;
}

// Output pointers of split `split`: its own partial slice, overwritten.
__device__ __forceinline__ GemmArgs split_outputs(const GemmArgs &p, int split) {
  GemmArgs q = p;
  if (p.splits > 1) {
    q.Wf = p.Wf + static_cast<size_t>(split) * p.split_stride;
    if (q.db) q.db = p.db + static_cast<size_t>(split) * p.M;
    q.accumulate = 0;
  }
  return q;
}

// Epilogue of one wave tile: lane owns row m and columns nb..nb+3 of each
// 32x32 fragment (the MFMA is issued as D = Btile * Atile^T).
template <Epi EPI, int FM, int FN, int WTM, int WTN>
__device__ __forceinline__ void store_tile(const GemmArgs &p, const f32x16_t (&acc)[FM][FN], int m0, int n0, int wm,
                                           int wn, int lane) {
  const int lrow = lane & 31;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int m = m0 + wm * WTM + i * 32 + lrow;
    if (m >= p.M) continue;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int nb = n0 + wn * WTN + j * 32 + q * 8 + (lane >> 5) * 4;
        if (nb >= p.N) continue;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[i][j][q * 4 + e];
        const size_t off = static_cast<size_t>(m) * p.ldy + nb;
        if constexpr (EPI == Epi::kF32) {
          f32x4_t w{v[0], v[1], v[2], v[3]};
          if (p.accumulate) w += *reinterpret_cast<const f32x4_t *>(p.Wf + off);
          *reinterpret_cast<f32x4_t *>(p.Wf + off) = w;
        } else {
          if constexpr (EPI == Epi::kBias || EPI == Epi::kBiasResid || EPI == Epi::kBiasGelu) {
            const u32x2_t bw = *reinterpret_cast<const u32x2_t *>(p.bias + nb);
            v[0] += lo_bf(bw[0]);
            v[1] += hi_bf(bw[0]);
            v[2] += lo_bf(bw[1]);
            v[3] += hi_bf(bw[1]);
          }
          if constexpr (EPI == Epi::kBiasResid || EPI == Epi::kResid) {
            const u32x2_t rw = *reinterpret_cast<const u32x2_t *>(p.R + off);
            v[0] += lo_bf(rw[0]);
            v[1] += hi_bf(rw[0]);
            v[2] += lo_bf(rw[1]);
            v[3] += hi_bf(rw[1]);
          }
          if constexpr (EPI == Epi::kGeluGrad) {
            const u32x2_t uw = *reinterpret_cast<const u32x2_t *>(p.R + off);
            v[0] *= gelu_grad_f(lo_bf(uw[0]));
            v[1] *= gelu_grad_f(hi_bf(uw[0]));
            v[2] *= gelu_grad_f(lo_bf(uw[1]));
            v[3] *= gelu_grad_f(hi_bf(uw[1]));
          }
          *reinterpret_cast<u32x2_t *>(p.Y + off) = u32x2_t{pack2(v[0], v[1]), pack2(v[2], v[3])};
          if constexpr (EPI == Epi::kBiasGelu) {
            *reinterpret_cast<u32x2_t *>(p.Y2 + off) =
                u32x2_t{pack2(gelu_f(v[0]), gelu_f(v[1])), pack2(gelu_f(v[2]), gelu_f(v[3]))};
          }
        }
      }
    }
  }

}

// Epilogue through LDS (direct-to-LDS kernels; the k-loop's buffers are free
// by then).  The tile is written out in chunks of 64 rows: the waves owning a
// chunk store their fp32 results (bias added) into LDS, row-major with a
// 16-byte row pad (conflict-free for the 64-bank LDS), then every thread
// streams whole rows out with 16-byte accesses, applying the residual, GELU,
// GELU' or the fp32 accumulation on the way.  Output rows are written in full
// 128-byte lines instead of 8-byte pieces scattered over 32 rows, with
// non-temporal stores: every CU writes its tile at about the same time, and
// streaming the burst past the caches measured 2% faster over the layer (the
// fp32 weight gradients most, and the LayerNorm backward that reads a GEMM
// output next).
constexpr int kEpiRows = 64;

template <Epi EPI, int BM, int BN, int WM, int WN>
__device__ __forceinline__ void store_tile_lds(const GemmArgs &p, const f32x16_t (&acc)[BM / WM / 32][BN / WN / 32],
                                               int m0, int n0, int wm, int wn, int lane, float *lds) {
  constexpr int NT = WM * WN * 64;
  constexpr int WTM = BM / WM, WTN = BN / WN, FM = WTM / 32, FN = WTN / 32;
  constexpr int LDR = BN + 4;  // floats per LDS row (16-byte pad)
  constexpr int NCH = BM / kEpiRows;
  static_assert(BM % kEpiRows == 0 && kEpiRows % 32 == 0, "epilogue chunking");
  constexpr bool kHasBias = EPI == Epi::kBias || EPI == Epi::kBiasResid || EPI == Epi::kBiasGelu;
  // a second per-element input: the residual, or the saved pre-activation u
  constexpr bool kHasR = EPI == Epi::kBiasResid || EPI == Epi::kResid || EPI == Epi::kGeluGrad;
  constexpr int PRB = BN / 8;                        // 16-byte bf16 segments per row
  constexpr int SEGS = (kEpiRows * PRB + NT - 1) / NT;  // per thread and chunk
  const int tid = threadIdx.x;
  const int lrow = lane & 31;

  // Every load of the epilogue is issued before its first store: loads and
  // stores retire in issue order, so a load issued behind the stores of the
  // previous chunk would wait for them.
  // (the 256-wide tile with both a bias and a residual has no registers to
  // spare for the bias: it loads the bias per chunk instead)
  constexpr bool kPreBias = kHasBias && !(kHasR && BN > 192);
  u32x2_t bias_w[kPreBias ? FN : 1][4];
  if constexpr (kPreBias) {
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int nb = n0 + wn * WTN + j * 32 + q * 8 + (lane >> 5) * 4;
        bias_w[j][q] = nb < p.N ? *reinterpret_cast<const u32x2_t *>(p.bias + nb) : u32x2_t{0u, 0u};
      }
  }
  u32x4_t rin[kHasR ? NCH : 1][kHasR ? SEGS : 1];
  if constexpr (kHasR) {
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
      for (int sg = 0; sg < SEGS; ++sg) {
        const int it = tid + NT * sg;
        const int gm = m0 + c * kEpiRows + it / PRB, gn = n0 + (it % PRB) * 8;
        const bool in = it < kEpiRows * PRB && gm < p.M && gn < p.N;
        rin[c][sg] = in ? ldg16(p.R + static_cast<size_t>(gm) * p.ldy + gn) : u32x4_t{0u, 0u, 0u, 0u};
      }
  }

#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    __syncthreads();  // LDS free (k-loop reads or the previous chunk's readers done)
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int r0 = wm * WTM + i * 32;  // fragment's first tile row
      if (r0 < c * kEpiRows || r0 >= (c + 1) * kEpiRows) continue;
      const int rl = r0 - c * kEpiRows + lrow;
#pragma unroll
      for (int j = 0; j < FN; ++j) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int cl = wn * WTN + j * 32 + q * 8 + (lane >> 5) * 4;
          f32x4_t v{acc[i][j][q * 4], acc[i][j][q * 4 + 1], acc[i][j][q * 4 + 2], acc[i][j][q * 4 + 3]};
          if constexpr (kPreBias) {
            v[0] += lo_bf(bias_w[j][q][0]);
            v[1] += hi_bf(bias_w[j][q][0]);
            v[2] += lo_bf(bias_w[j][q][1]);
            v[3] += hi_bf(bias_w[j][q][1]);
          } else if constexpr (kHasBias) {
            const int nb = n0 + cl;
            if (nb < p.N) {
              const u32x2_t bw = *reinterpret_cast<const u32x2_t *>(p.bias + nb);
              v[0] += lo_bf(bw[0]);
              v[1] += hi_bf(bw[0]);
              v[2] += lo_bf(bw[1]);
              v[3] += hi_bf(bw[1]);
            }
          }
          *reinterpret_cast<f32x4_t *>(lds + rl * LDR + cl) = v;
        }
      }
    }
    __syncthreads();
    if constexpr (EPI == Epi::kF32) {
      constexpr int PER_ROW = BN / 4;
      for (int it = tid; it < kEpiRows * PER_ROW; it += NT) {
        const int r = it / PER_ROW, cc = (it % PER_ROW) * 4;
        const int gm = m0 + c * kEpiRows + r, gn = n0 + cc;
        if (gm >= p.M || gn >= p.N) continue;
        f32x4_t v = *reinterpret_cast<const f32x4_t *>(lds + r * LDR + cc);
        const size_t off = static_cast<size_t>(gm) * p.ldy + gn;
        if (p.accumulate) v += *reinterpret_cast<const f32x4_t *>(p.Wf + off);
        stg16_nt(p.Wf + off, v);
      }
    } else {
#pragma unroll
      for (int sg = 0; sg < SEGS; ++sg) {
        const int it = tid + NT * sg;
        const int r = it / PRB, cc = (it % PRB) * 8;
        const int gm = m0 + c * kEpiRows + r, gn = n0 + cc;
        if (it >= kEpiRows * PRB || gm >= p.M || gn >= p.N) continue;
        const f32x4_t a = *reinterpret_cast<const f32x4_t *>(lds + r * LDR + cc);
        const f32x4_t b = *reinterpret_cast<const f32x4_t *>(lds + r * LDR + cc + 4);
        float v[8] = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
        const size_t off = static_cast<size_t>(gm) * p.ldy + gn;
        if constexpr (EPI == Epi::kBiasResid || EPI == Epi::kResid) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[2 * e] += lo_bf(rin[c][sg][e]);
            v[2 * e + 1] += hi_bf(rin[c][sg][e]);
          }
        }
        if constexpr (EPI == Epi::kGeluGrad) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[2 * e] *= gelu_grad_f(lo_bf(rin[c][sg][e]));
            v[2 * e + 1] *= gelu_grad_f(hi_bf(rin[c][sg][e]));
          }
        }
        u32x4_t o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = pack2(v[2 * e], v[2 * e + 1]);
        stg16_nt(p.Y + off, o);
        if constexpr (EPI == Epi::kBiasGelu) {
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = pack2(gelu_f(v[2 * e]), gelu_f(v[2 * e + 1]));
          stg16_nt(p.Y2 + off, o);
        }
      }
    }
  }
}

// Global -> register -> LDS staging of one [ROWS x BK] operand tile.
template <int ROWS, int BK, int NT, bool TRANS>
struct TileLoader;

// Contraction-contiguous operand: X(r, k) = X[r * ld + k].
template <int ROWS, int BK, int NT>
struct TileLoader<ROWS, BK, NT, false> {
  static constexpr int KC = BK / 8;  // 16-byte chunks per row
  static constexpr int CH = ROWS * KC / NT;
  static_assert(ROWS * KC % NT == 0, "tile chunks must divide the threads");
  u32x4_t r[CH];

  __device__ __forceinline__ void load(const bf16_t *__restrict__ X, int ld, int rows, int K, int r0, int k0,
                                       int tid) {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = tid + NT * i;
      const int row = c / KC, kc = c % KC;
      const int gr = r0 + row, gk = k0 + kc * 8;
      if (gr < rows && gk < K)
        r[i] = ldg16(X + static_cast<size_t>(gr) * ld + gk);
      else
        r[i] = u32x4_t{0u, 0u, 0u, 0u};
    }
  }
  template <int LDK>
  __device__ __forceinline__ void store(bf16_t *lds, int tid) {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = tid + NT * i;
      const int row = c / KC, kc = c % KC;
      *reinterpret_cast<u32x4_t *>(lds + row * LDK + kc * 8) = r[i];
    }
  }
};

// Contraction-strided operand: X(r, k) = X[k * ld + r]; rows come in whole
// groups of 8 (every row count here is a multiple of 8).
template <int ROWS, int BK, int NT>
struct TileLoader<ROWS, BK, NT, true> {
  static constexpr int KB = BK / 8;
  static constexpr int NBLK = (ROWS / 8) * KB;
  static constexpr int TB = (NBLK + NT - 1) / NT;
  u32x4_t r[TB][8];

  __device__ __forceinline__ void load(const bf16_t *__restrict__ X, int ld, int rows, int K, int r0, int k0,
                                       int tid) {
#pragma unroll
    for (int t = 0; t < TB; ++t) {
      const int b = tid + NT * t;
      const int kb = b % KB, rb = b / KB;
      const int gr = r0 + rb * 8;
      const bool rok = (NBLK % NT == 0 || b < NBLK) && gr < rows;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int gk = k0 + kb * 8 + j;
        if (rok && gk < K)
          r[t][j] = ldg16(X + static_cast<size_t>(gk) * ld + gr);
        else
          r[t][j] = u32x4_t{0u, 0u, 0u, 0u};
      }
    }
  }
  template <int LDK>
  __device__ __forceinline__ void store(bf16_t *lds, int tid) {
#pragma unroll
    for (int t = 0; t < TB; ++t) {
      const int b = tid + NT * t;
      if (NBLK % NT != 0 && b >= NBLK) continue;
      const int kb = b % KB, rb = b / KB;
      u32x4_t o[8];
      transpose8x8(r[t], o);
#pragma unroll
      for (int i = 0; i < 8; ++i) *reinterpret_cast<u32x4_t *>(lds + (rb * 8 + i) * LDK + kb * 8) = o[i];
    }
  }
  // Row sums over the 8 staged k values of each of the 8 rows of block t.
  __device__ __forceinline__ void rowsum(float acc[TB][8]) const {
#pragma unroll
    for (int t = 0; t < TB; ++t)
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[t][i] += (i & 1) ? hi_bf(r[t][j][i >> 1]) : lo_bf(r[t][j][i >> 1]);
  }
};

template <int BM, int BN, int BK, int WM, int WN, bool AT, bool BT, Epi EPI>
__global__ __launch_bounds__(WM *WN * 64) void gemm_kernel(GemmArgs p) {
  constexpr int NT = WM * WN * 64;
  constexpr int LDK = BK + 8;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  constexpr int STAGE = (BM + BN) * LDK;
  static_assert(WTM % 32 == 0 && WTN % 32 == 0 && BK % 16 == 0, "tile shape");
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid / WN, wn = wid % WN;
  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN;
  int tm, tn;
  tile_of(tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;

  TileLoader<BM, BK, NT, AT> la;
  TileLoader<BN, BK, NT, BT> lb;
  constexpr bool kDb = (EPI == Epi::kF32) && AT;
  constexpr int DB_TB = AT ? TileLoader<BM, BK, NT, true>::TB : 1;
  float dbacc[DB_TB][8];
  const bool do_db = kDb && p.db != nullptr && tn == 0;
  if constexpr (kDb) {
#pragma unroll
    for (int t = 0; t < DB_TB; ++t)
#pragma unroll
      for (int i = 0; i < 8; ++i) dbacc[t][i] = 0.f;
  }

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16_t{};

  const int nk = (p.K + BK - 1) / BK;
  la.load(p.A, p.lda, p.M, p.K, m0, 0, tid);
  lb.load(p.B, p.ldb, p.N, p.K, n0, 0, tid);
  if constexpr (kDb) {
    if (do_db) la.rowsum(dbacc);
  }
  la.template store<LDK>(smem, tid);
  lb.template store<LDK>(smem + BM * LDK, tid);
  __syncthreads();

  const int lrow = lane & 31, lk = (lane >> 5) * 8;
  for (int t = 0; t < nk; ++t) {
    const bf16_t *As = smem + (t & 1) * STAGE;
    const bf16_t *Bs = As + BM * LDK;
    const bool more = (t + 1) < nk;
    if (more) {
      la.load(p.A, p.lda, p.M, p.K, m0, (t + 1) * BK, tid);
      lb.load(p.B, p.ldb, p.N, p.K, n0, (t + 1) * BK, tid);
    }
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8_t af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t *>(As + (wm * WTM + i * 32 + lrow) * LDK + kk * 16 + lk);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8_t *>(Bs + (wn * WTN + j * 32 + lrow) * LDK + kk * 16 + lk);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32(bfr[j], af[i], acc[i][j]);
    }
    if (more) {
      if constexpr (kDb) {
        if (do_db) la.rowsum(dbacc);
      }
      bf16_t *Ns = smem + ((t + 1) & 1) * STAGE;
      la.template store<LDK>(Ns, tid);
      lb.template store<LDK>(Ns + BM * LDK, tid);
    }
    __syncthreads();
  }

  store_tile<EPI, FM, FN, WTM, WTN>(p, acc, m0, n0, wm, wn, lane);

  // ---- fused bias gradient: row sums of A over all k (column tile 0 only)
  if constexpr (kDb) {
    if (do_db) {
      constexpr int KB = BK / 8;
#pragma unroll
      for (int t = 0; t < DB_TB; ++t) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          float s = dbacc[t][i];
#pragma unroll
          for (int o = 1; o < KB; o <<= 1) s += __shfl_xor(s, o, kWave);
          dbacc[t][i] = s;
        }
        const int b = tid + NT * t;
        const int rb = b / KB;
        const int gr = m0 + rb * 8;
        if ((b % KB) == 0 && b < TileLoader<BM, BK, NT, true>::NBLK && gr < p.M) {
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            float s = dbacc[t][i];
            if (p.accumulate) s += p.db[gr + i];
            p.db[gr + i] = s;
          }
        }
      }
    }
  }
}

// ===========================================================================
// Direct-to-LDS pipeline (the large-problem path).
//
// Tiles go from HBM straight into LDS with buffer_load_dwordx4 ... lds (no
// staging registers), STAGES deep, so the loads for k-step t+STAGES-1 are in
// flight while k-step t runs on the MFMAs.  The buffer resource bounds every
// operand tensor: rows past its end (tokens past M, weight rows past N, or
// contraction rows past K of a transposed operand) read as zero.
//
// LDS tile layouts (16-byte chunks, XOR-swizzled against bank conflicts):
//  - contraction-contiguous operand: [row][BK], chunk c of row r stored at
//    c ^ ((r / RP) % CPR) (RP rows share one 128-byte line); MFMA operands
//    are single ds_read_b128.
//  - contraction-strided operand: [BK][ROWS] exactly as in memory, chunk j of
//    k-row k stored at j ^ 2*(k % 4); MFMA operands are two
//    ds_read_b64_tr_b16, whose 16-lane transpose delivers lane l the column
//    (l % 32) of k-rows 8*(l/32) + 0..7.
// ===========================================================================

// LDS is 64 banks x 4 bytes (256 bytes per cycle); a 16-lane quarter-wave
// of ds_read_b128 and a half-wave of ds_read_b64_tr_b16 must hit distinct
// banks.  nt tiles: RP rows share one 256-byte bank line, so chunk c of row
// r goes to c ^ ((r / RP) % CPR).  Transposed tiles: k-rows are padded to a
// power of two (TROWS) and chunk j of k-row k goes to j ^ 4 * (k % 4), which
// spreads the four k-rows read together over four disjoint 64-byte ranges.
template <int BK>
struct NtTile {
  static constexpr int RB = BK * 2;                          // bytes per row
  static constexpr int RP = (256 / RB) > 0 ? (256 / RB) : 1;  // rows per bank line
  static constexpr int CPR = BK / 8;                         // 16-byte chunks per row
  __device__ static __forceinline__ int off(int r, int c) { return r * RB + ((c ^ ((r / RP) % CPR)) << 4); }
};

template <int ROWS>
struct TTile {
  static constexpr int TROWS = ROWS <= 128 ? 128 : 256;  // padded k-row length
  static_assert(ROWS <= 256 && ROWS % 32 == 0, "transposed tile width");
  __device__ static __forceinline__ int off(int k, int j) { return k * (TROWS * 2) + ((j ^ ((k & 3) << 2)) << 4); }
};

template <int ROWS, int BK, int NW, bool TRANS>
struct DirectLoader {
  // LDS bytes of one stage of this operand (transposed tiles are padded)
  static constexpr int BYTES = TRANS ? TTile<ROWS>::TROWS * BK * 2 : ROWS * BK * 2;
  static constexpr int NI = BYTES / (1024 * NW);
  static_assert(BYTES % (1024 * NW) == 0, "tile bytes must split into whole wave loads");
  uint32_t voff[NI];
  uint32_t live;  // bit i: this lane's chunk of load i is real data (not padding)
  u32x4_t rsrc;

  // base/nbytes: the operand tensor; ld its leading dimension (elements);
  // r0 the first tile row (output row of this operand).
  __device__ __forceinline__ void init(const bf16_t *base, uint32_t nbytes, int ld, int r0, int wid, int lane) {
    rsrc = make_rsrc(base, nbytes);
    live = 0;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int o = (wid * NI + i) * 1024 + lane * 16;
      if constexpr (!TRANS) {
        using T = NtTile<BK>;
        const int r = o / T::RB, pch = (o % T::RB) >> 4;
        const int c = pch ^ ((r / T::RP) % T::CPR);
        voff[i] = static_cast<uint32_t>(((r0 + r) * static_cast<long>(ld) + c * 8) * 2);
        live |= 1u << i;
      } else {
        constexpr int TR = TTile<ROWS>::TROWS;
        const int k = o / (TR * 2), pch = (o % (TR * 2)) >> 4;
        const int j = pch ^ ((k & 3) << 2);
        voff[i] = static_cast<uint32_t>((k * static_cast<long>(ld) + r0 + j * 8) * 2);
        if (j * 8 < ROWS) live |= 1u << i;
      }
    }
  }
  // Enqueue this wave's share of one stage: soff is the k-step's byte offset.
  __device__ __forceinline__ void issue(uint32_t tile_addr, uint32_t soff, int wid) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const uint32_t dst = __builtin_amdgcn_readfirstlane(tile_addr + static_cast<uint32_t>((wid * NI + i) * 1024));
      const uint32_t so = __builtin_amdgcn_readfirstlane(soff);
      if (!TRANS || TTile<ROWS>::TROWS == ROWS || ((live >> i) & 1u)) buffer_load_lds16(rsrc, dst, voff[i], so);
    }
  }
};

// Per-lane LDS byte offsets of one operand's MFMA fragments (stage-relative).
template <int ROWS, int BK, int F, bool TRANS>
struct FragAddr {
  static constexpr int KS = BK / 16;
  // non-transposed: one address per k-step (fragments add 32 rows);
  // transposed: two per fragment (k-steps add 16 k-rows).
  static constexpr int N = TRANS ? 2 * F : KS;
  int off[N];
  __device__ __forceinline__ void init(int rbase, int lane) {
    if constexpr (!TRANS) {
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) off[kk] = NtTile<BK>::off(rbase + (lane & 31), kk * 2 + (lane >> 5));
    } else {
      const int k = 8 * (lane >> 5) + ((lane & 15) >> 2);
#pragma unroll
      for (int f = 0; f < F; ++f) {
        const int n = rbase + f * 32 + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
        off[2 * f] = TTile<ROWS>::off(k, n >> 3) + (n & 7) * 2;
        off[2 * f + 1] = TTile<ROWS>::off(k + 4, n >> 3) + (n & 7) * 2;
      }
    }
  }
  __device__ __forceinline__ bf16x8_t get(const lds_char *tile, int f, int kk) const {
    if constexpr (!TRANS) {
      return *reinterpret_cast<const __attribute__((address_space(3))) bf16x8_t *>(tile + off[kk] +
                                                                                     f * 32 * BK * 2);
    } else {
      constexpr int TR = TTile<ROWS>::TROWS;
      return lds_read_tr(tile + off[2 * f] + kk * 16 * TR * 2, tile + off[2 * f + 1] + kk * 16 * TR * 2);
    }
  }
};

// Scheduling hint for one k-step: spread the NR LDS reads of the next
// k-step's fragments evenly between the NM MFMAs of this k-step, so that the
// reads have a whole k-step of MFMA work to land in.
template <int NM, int NR, int M = 0>
__device__ __forceinline__ void interleave_reads() {
  if constexpr (M < NM) {
    constexpr int per = (NR + NM - 1) / NM;
    constexpr int done = M * per < NR ? M * per : NR;
    constexpr int r = (NR - done) < per ? (NR - done) : per;
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
    if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(0x100, r, 0);  // then r LDS reads
    interleave_reads<NM, NR, M + 1>();
  }
}

template <int BM, int BN, int BK, int WM, int WN, int STAGES, bool AT, bool BT, Epi EPI>
__global__ __launch_bounds__(WM *WN * 64, 1) void gemm_lds_kernel(GemmArgs p, uint32_t a_bytes, uint32_t b_bytes) {
  constexpr int NW = WM * WN;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  constexpr int KS = BK / 16;
  constexpr int A_BYTES = DirectLoader<BM, BK, NW, AT>::BYTES, B_BYTES = DirectLoader<BN, BK, NW, BT>::BYTES;
  constexpr int STAGE = A_BYTES + B_BYTES;
  static_assert(STAGES >= 2 && BK % 16 == 0, "pipeline shape");
  extern __shared__ __attribute__((aligned(1024))) char smem_raw[];
  const lds_char *smem = (const lds_char *)(smem_raw);  // generic -> LDS address space

  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int wm = wid / WN, wn = wid % WN;
  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN;
  int tm, tn, kbeg, klen;
  const int split = split_of(p, tiles_m, tiles_n, tm, tn, kbeg, klen);
  const int m0 = tm * BM, n0 = tn * BN;

  DirectLoader<BM, BK, NW, AT> la;
  DirectLoader<BN, BK, NW, BT> lb;
  la.init(p.A, a_bytes, p.lda, m0, wid, lane);
  lb.init(p.B, b_bytes, p.ldb, n0, wid, lane);
  // byte step of one k-step along each operand, and of the split's first k
  const uint32_t a_step = AT ? static_cast<uint32_t>(BK) * p.lda * 2 : BK * 2;
  const uint32_t b_step = BT ? static_cast<uint32_t>(BK) * p.ldb * 2 : BK * 2;
  const uint32_t a_k0 = AT ? static_cast<uint32_t>(kbeg) * p.lda * 2 : static_cast<uint32_t>(kbeg) * 2;
  const uint32_t b_k0 = BT ? static_cast<uint32_t>(kbeg) * p.ldb * 2 : static_cast<uint32_t>(kbeg) * 2;

  FragAddr<BM, BK, FM, AT> fa;
  FragAddr<BN, BK, FN, BT> fb;
  fa.init(wm * WTM, lane);
  fb.init(wn * WTN, lane);

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16_t{};

  // Weight gradient: the bias gradient db[m] = sum_k A(m, k) is summed from
  // the A fragments already in registers by the first wave column of the
  // first column tile (fixed order: deterministic).
  constexpr bool kDb = (EPI == Epi::kF32);
  const bool do_db = kDb && p.db != nullptr && tn == 0 && wn == 0;
  float dbacc[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) dbacc[i] = 0.f;

  const int nk = (klen + BK - 1) / BK;
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(smem));
  constexpr int PER_STAGE = DirectLoader<BM, BK, NW, AT>::NI + DirectLoader<BN, BK, NW, BT>::NI;
#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s) {
    if (s < nk) {
      la.issue(lds0 + s * STAGE, a_k0 + s * a_step, wid);
      lb.issue(lds0 + s * STAGE + A_BYTES, b_k0 + s * b_step, wid);
    }
  }
  // k-step 0 resident for every wave
  if (STAGES - 1 < nk)
    wait_vmcnt<PER_STAGE * (STAGES - 2)>();
  else
    wait_vmcnt<0>();
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");

  // Fragments are double-buffered in registers: the next k-step's LDS reads
  // are issued behind the current k-step's MFMAs.  The stage barrier sits
  // after the last k-step's MFMAs are issued, so their execution covers the
  // barrier and the first reads of the next stage.
  bf16x8_t af[2][FM], bfr[2][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i) af[0][i] = fa.get(smem, i, 0);
#pragma unroll
  for (int j = 0; j < FN; ++j) bfr[0][j] = fb.get(smem + A_BYTES, j, 0);

  for (int t = 0; t < nk; ++t) {
    // refill the buffer of k-step t-1 (every wave finished reading it
    // before the barrier that ended k-step t-1)
    const int tl = t + STAGES - 1;
    const uint32_t st_l = lds0 + (tl % STAGES) * STAGE;
    // One operand's refill goes out a sub-step after the other's: the
    // activations (A) second in the forward layout (256x192 and 256x256
    // tiles, contraction up to 8192), the weights (B) second in the
    // input-gradient layout (256x192).  Measured on the ViT-22B layer: QKV
    // forward 8%, MLP-up forward 2% and the out-projection forward and input
    // gradient 5% faster; the forward with K = 24576 (MLP down) was 2% faster
    // without it; later (two sub-steps) or both operands split in halves was
    // slower.
    constexpr bool kSpread = !AT && (BT ? BN == 192 : BN >= 192);
    constexpr bool kALate = kSpread && !BT;
    const bool spread = kSpread && (BT || p.K <= 8192);
    if (tl < nk) {
      if (!kALate || !spread) la.issue(st_l, a_k0 + tl * a_step, wid);
      if (!kSpread || kALate || !spread) lb.issue(st_l + A_BYTES, b_k0 + tl * b_step, wid);
    }
    const lds_char *As = smem + (t % STAGES) * STAGE;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const int c = kk & 1, n = c ^ 1;
      if constexpr (kSpread) {
        if (kk == 1 && tl < nk && spread) {
          if constexpr (kALate)
            la.issue(st_l, a_k0 + tl * a_step, wid);
          else
            lb.issue(st_l + A_BYTES, b_k0 + tl * b_step, wid);
        }
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32(bfr[c][j], af[c][i], acc[i][j]);
      if constexpr (kDb) {
        if (do_db) {
#pragma unroll
          for (int i = 0; i < FM; ++i) {
            const u32x4_t w = __builtin_bit_cast(u32x4_t, af[c][i]);
#pragma unroll
            for (int e = 0; e < 4; ++e) dbacc[i] += lo_bf(w[e]) + hi_bf(w[e]);
          }
        }
      }
      if (kk + 1 < KS) {
#pragma unroll
        for (int i = 0; i < FM; ++i) af[n][i] = fa.get(As, i, kk + 1);
#pragma unroll
        for (int j = 0; j < FN; ++j) bfr[n][j] = fb.get(As + A_BYTES, j, kk + 1);
        interleave_reads<FM * FN, (FM + FN) * (AT || BT ? 2 : 1)>();
      } else if (t + 1 < nk) {
        // also retire this wave's LDS reads of k-step t before the barrier
        if (t + STAGES - 1 < nk)
          wait_vmcnt<PER_STAGE * (STAGES - 2), 0>();
        else
          wait_vmcnt<0, 0>();
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        const lds_char *Ns = smem + ((t + 1) % STAGES) * STAGE;
#pragma unroll
        for (int i = 0; i < FM; ++i) af[n][i] = fa.get(Ns, i, 0);
#pragma unroll
        for (int j = 0; j < FN; ++j) bfr[n][j] = fb.get(Ns + A_BYTES, j, 0);
      }
    }
    if constexpr (KS % 2 == 1) {
      // odd k-steps per stage: the next stage's fragments sit in buffer 1
#pragma unroll
      for (int i = 0; i < FM; ++i) af[0][i] = af[1][i];
#pragma unroll
      for (int j = 0; j < FN; ++j) bfr[0][j] = bfr[1][j];
    }
  }
  const GemmArgs q = split_outputs(p, split);
  store_tile_lds<EPI, BM, BN, WM, WN>(q, acc, m0, n0, wm, wn, lane, reinterpret_cast<float *>(smem_raw));
  if constexpr (kDb) {
    if (do_db) {
      // lane l and l ^ 32 hold the two token halves of row (l % 32)
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const float tot = dbacc[i] + __shfl_xor(dbacc[i], 32, kWave);
        const int row = m0 + wm * WTM + i * 32 + (lane & 31);
        if (lane < 32 && row < q.M) q.db[row] = q.accumulate ? q.db[row] + tot : tot;
      }
    }
  }
}

// Variant of the two-stage kernel with uneven operand rings: the deep
// operand (A when A_DEEP, else B) cycles through three LDS slots and is
// refilled two stages ahead, the other through two slots, one stage ahead.
// A 256x192x64 tile uses 3 x 32 + 2 x 24 KB = 144 KB (a 256x256 one would
// take all 160 KB).  Each stage issues the shallow operand's next stage
// first and the deep operand's stage a sub-step later, so the wait that ends
// the stage leaves exactly the latter in flight; one barrier per stage as in
// the two-stage kernel.  A stage's refill then has two stages of matrix work
// to land in instead of one.

template <int BM, int BN, int BK, int WM, int WN, bool A_DEEP, bool BT, Epi EPI>
__global__ __launch_bounds__(WM *WN * 64, 1) void gemm_deep_kernel(GemmArgs p, uint32_t a_bytes, uint32_t b_bytes) {
  constexpr int NW = WM * WN;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  constexpr int KS = BK / 16;
  using LA = DirectLoader<BM, BK, NW, false>;
  using LB = DirectLoader<BN, BK, NW, BT>;
  constexpr int A_BYTES = LA::BYTES, B_BYTES = LB::BYTES;
  constexpr int SA = A_DEEP ? 3 : 2, SB = A_DEEP ? 2 : 3;
  constexpr int B_BASE = SA * A_BYTES;
  constexpr int NX = A_DEEP ? LA::NI : LB::NI;  // loads per wave of one stage of the deep operand
  static_assert(KS % 2 == 0, "fragment double-buffering needs an even number of k-steps per stage");
  extern __shared__ __attribute__((aligned(1024))) char smem_raw[];
  const lds_char *smem = (const lds_char *)(smem_raw);

  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wid / WN, wn = wid % WN;
  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN;
  int tm, tn, kbeg, klen;
  const int split = split_of(p, tiles_m, tiles_n, tm, tn, kbeg, klen);
  const int m0 = tm * BM, n0 = tn * BN;

  LA la;
  LB lb;
  la.init(p.A, a_bytes, p.lda, m0, wid, lane);
  lb.init(p.B, b_bytes, p.ldb, n0, wid, lane);
  const uint32_t a_k0 = static_cast<uint32_t>(kbeg) * 2;
  const uint32_t b_step = BT ? static_cast<uint32_t>(BK) * p.ldb * 2 : BK * 2;
  const uint32_t b_k0 = BT ? static_cast<uint32_t>(kbeg) * p.ldb * 2 : static_cast<uint32_t>(kbeg) * 2;
  FragAddr<BM, BK, FM, false> fa;
  FragAddr<BN, BK, FN, BT> fb;
  fa.init(wm * WTM, lane);
  fb.init(wn * WTN, lane);

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16_t{};

  const int nk = (klen + BK - 1) / BK;
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(smem));
  auto issue_a = [&](int t) { la.issue(lds0 + (t % SA) * A_BYTES, a_k0 + t * BK * 2, wid); };
  auto issue_b = [&](int t) { lb.issue(lds0 + B_BASE + (t % SB) * B_BYTES, b_k0 + t * b_step, wid); };
  auto issue_deep = [&](int t) {
    if constexpr (A_DEEP)
      issue_a(t);
    else
      issue_b(t);
  };
  auto issue_shallow = [&](int t) {
    if constexpr (A_DEEP)
      issue_b(t);
    else
      issue_a(t);
  };
  auto a_stage = [&](int t) { return smem + (t % SA) * A_BYTES; };
  auto b_stage = [&](int t) { return smem + B_BASE + (t % SB) * B_BYTES; };

  // stage 0 of both operands, then stage 1 of the deep one
  issue_deep(0);
  issue_shallow(0);
  if (nk > 1) {
    issue_deep(1);
    wait_vmcnt<NX>();
  } else {
    wait_vmcnt<0>();
  }
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");

  bf16x8_t af[2][FM], bfr[2][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i) af[0][i] = fa.get(a_stage(0), i, 0);
#pragma unroll
  for (int j = 0; j < FN; ++j) bfr[0][j] = fb.get(b_stage(0), j, 0);

  for (int t = 0; t < nk; ++t) {
    // refill the slots stage t-1 used (every wave finished reading them
    // before the barrier that ended stage t-1): shallow operand first
    if (t + 1 < nk) issue_shallow(t + 1);
    const lds_char *As = a_stage(t), *Bs = b_stage(t);
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const int c = kk & 1, n = c ^ 1;
      // the deep operand has two stages of lead: its refill can go out a
      // sub-step after the shallow one's
      if (kk == 1 && t + 2 < nk) issue_deep(t + 2);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32(bfr[c][j], af[c][i], acc[i][j]);
      if (kk + 1 < KS) {
#pragma unroll
        for (int i = 0; i < FM; ++i) af[n][i] = fa.get(As, i, kk + 1);
#pragma unroll
        for (int j = 0; j < FN; ++j) bfr[n][j] = fb.get(Bs, j, kk + 1);
        interleave_reads<FM * FN, (FM + FN) * (BT ? 2 : 1)>();
      } else if (t + 1 < nk) {
        // stage t+1 of both operands landed for this wave (the deep
        // operand's stage t+2, issued last, may stay in flight); this
        // wave's LDS reads of stage t retired
        if (t + 2 < nk)
          wait_vmcnt<NX, 0>();
        else
          wait_vmcnt<0, 0>();
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
#pragma unroll
        for (int i = 0; i < FM; ++i) af[n][i] = fa.get(a_stage(t + 1), i, 0);
#pragma unroll
        for (int j = 0; j < FN; ++j) bfr[n][j] = fb.get(b_stage(t + 1), j, 0);
      }
    }
  }
  const GemmArgs q = split_outputs(p, split);
  store_tile_lds<EPI, BM, BN, WM, WN>(q, acc, m0, n0, wm, wn, lane, reinterpret_cast<float *>(smem_raw));
}

template <int BM, int BN, int BK, int WM, int WN, bool A_DEEP, bool BT, Epi EPI>
bool launch_deep_cfg(const GemmArgs &a, uint32_t a_bytes, uint32_t b_bytes, hipStream_t s) {
  constexpr int NW = WM * WN;
  constexpr size_t lds = static_cast<size_t>(A_DEEP ? 3 : 2) * DirectLoader<BM, BK, NW, false>::BYTES +
                         static_cast<size_t>(A_DEEP ? 2 : 3) * DirectLoader<BN, BK, NW, BT>::BYTES;
  static_assert(lds <= 160 * 1024, "LDS budget");
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN) * (a.splits > 1 ? a.splits : 1);
  hipLaunchKernelGGL((gemm_deep_kernel<BM, BN, BK, WM, WN, A_DEEP, BT, EPI>), dim3(tiles), dim3(NW * 64), lds, s, a,
                     a_bytes, b_bytes);
  return true;
}

// 256x192 products that take the uneven-ring kernel (A deep): forward-layout
// products with a contraction longer than kDeepFwdMinK.  Measured (same-box
// A/B, ViT-22B layer): MLP-down forward (K = 24576) 543 -> 508 us; at
// K = 6144 (QKV and out-projection forward) 1% slower than the two-stage
// kernel, whose refill spread applies there; input gradients 0-8% slower
// with A deep and equal to 8% slower with B deep, 256x256 forward tiles
// 1-5% slower.  So only the forward layout with A deep is instantiated.
constexpr int kDeepFwdMinK = 8192;

// 256x192 input gradients with a contraction longer than this take the
// ping-pong kernel.  Same-box A/B on the ViT-22B layer: alone, the MLP-up
// input gradient (K = 24576) went 531 -> 523 us and the QKV one
// (K = 18432) 402 -> 396 us; inside the layer chain the MLP-up one still
// gained (541 -> 535 us) but the QKV one lost (401 -> 409 us), and at
// K = 6144 (out-projection) it was no better.
constexpr int kPpDgradMinK = 20480;

template <int BM, int BN, int BK, int WM, int WN, int STAGES, bool AT, bool BT, Epi EPI>
bool launch_lds_cfg(const GemmArgs &a, uint32_t a_bytes, uint32_t b_bytes, hipStream_t s) {
  constexpr int NW = WM * WN;
  constexpr size_t lds = static_cast<size_t>(STAGES) *
                         (DirectLoader<BM, BK, NW, AT>::BYTES + DirectLoader<BN, BK, NW, BT>::BYTES);
  static_assert(lds <= 160 * 1024, "LDS budget");
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN) * (a.splits > 1 ? a.splits : 1);
  hipLaunchKernelGGL((gemm_lds_kernel<BM, BN, BK, WM, WN, STAGES, AT, BT, EPI>), dim3(tiles), dim3(WM * WN * 64),
                     lds, s, a, a_bytes, b_bytes);
  return true;
}

template <int BM, int BN, int BK, int WM, int WN, bool AT, bool BT, Epi EPI>
bool launch_cfg(const GemmArgs &a, hipStream_t s) {
  constexpr int NT = WM * WN * 64;
  constexpr size_t lds = 2 * static_cast<size_t>(BM + BN) * (BK + 8) * sizeof(bf16_t);
  auto kern = gemm_kernel<BM, BN, BK, WM, WN, AT, BT, EPI>;
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  hipLaunchKernelGGL(kern, dim3(tiles), dim3(NT), lds, s, a);
  return true;
}

// Tile choice: 256x128 tiles (4 waves of 128x64) when the problem yields at
// least two waves of such tiles on 256 CUs; else 128x128 (4 waves of 64x64).
template <bool AT, bool BT, Epi EPI>
bool launch_any(const GemmArgs &a, hipStream_t s) {
  if (any_tile(a.M, a.N).bm == 256) return launch_cfg<256, 128, 64, 2, 2, AT, BT, EPI>(a, s);
  return launch_cfg<128, 128, 64, 2, 2, AT, BT, EPI>(a, s);
}

// ---------------------------------------------------------------------------
// Ping-pong variant: 8 waves, two per SIMD (waves w and w + 4), in two groups
// offset by one phase.  Each k-step has a load phase (issue this wave's share
// of the DMA STAGES-1 k-steps ahead, read all of this k-step's fragments into
// registers, wait for them) and a compute phase (the k-step's MFMAs, operands
// already in registers); a workgroup barrier ends every phase.  While one
// group computes, the other loads, so each SIMD's MFMA pipe is fed by one of
// its two waves at a time.
//
// Buffer safety: k-step t is read by group 0 in phase 2t and by group 1 in
// phase 2t+1; its buffer is refilled (k-step t+STAGES) from phase 2t+2 on.
// Each wave waits for its own share of k-step t+1 in its load phase of t, so
// both groups' shares have landed by the barrier that ends phase 2t+1.
// ---------------------------------------------------------------------------
template <int BM, int BN, int BK, int WM, int WN, int STAGES, bool AT, bool BT, Epi EPI>
__global__ __launch_bounds__(WM *WN * 64, 1) void gemm_pp_kernel(GemmArgs p, uint32_t a_bytes, uint32_t b_bytes) {
  constexpr int NW = WM * WN;
  static_assert(NW == 8, "ping-pong needs two waves per SIMD");
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FM = WTM / 32, FN = WTN / 32;
  constexpr int KS = BK / 16;
  constexpr int A_BYTES = DirectLoader<BM, BK, NW, AT>::BYTES, B_BYTES = DirectLoader<BN, BK, NW, BT>::BYTES;
  constexpr int STAGE = A_BYTES + B_BYTES;
  static_assert(STAGES >= 3 && BK % 16 == 0, "pipeline shape");
  extern __shared__ __attribute__((aligned(1024))) char smem_raw[];
  const lds_char *smem = (const lds_char *)(smem_raw);  // generic -> LDS address space

  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int grp = wid >> 2;                                          // 0: waves 0-3, 1: waves 4-7
  const int wm = wid / WN, wn = wid % WN;
  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN;
  int tm, tn, kbeg, klen;
  const int split = split_of(p, tiles_m, tiles_n, tm, tn, kbeg, klen);
  const int m0 = tm * BM, n0 = tn * BN;

  DirectLoader<BM, BK, NW, AT> la;
  DirectLoader<BN, BK, NW, BT> lb;
  la.init(p.A, a_bytes, p.lda, m0, wid, lane);
  lb.init(p.B, b_bytes, p.ldb, n0, wid, lane);
  const uint32_t a_step = AT ? static_cast<uint32_t>(BK) * p.lda * 2 : BK * 2;
  const uint32_t b_step = BT ? static_cast<uint32_t>(BK) * p.ldb * 2 : BK * 2;
  const uint32_t a_k0 = AT ? static_cast<uint32_t>(kbeg) * p.lda * 2 : static_cast<uint32_t>(kbeg) * 2;
  const uint32_t b_k0 = BT ? static_cast<uint32_t>(kbeg) * p.ldb * 2 : static_cast<uint32_t>(kbeg) * 2;
  FragAddr<BM, BK, FM, AT> fa;
  FragAddr<BN, BK, FN, BT> fb;
  fa.init(wm * WTM, lane);
  fb.init(wn * WTN, lane);

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x16_t{};
  constexpr bool kDb = (EPI == Epi::kF32);
  const bool do_db = kDb && p.db != nullptr && tn == 0 && wn == 0;
  float dbacc[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) dbacc[i] = 0.f;

  const int nk = (klen + BK - 1) / BK;
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(smem));
  constexpr int PER_STAGE = DirectLoader<BM, BK, NW, AT>::NI + DirectLoader<BN, BK, NW, BT>::NI;
#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s) {
    if (s < nk) {
      la.issue(lds0 + s * STAGE, a_k0 + s * a_step, wid);
      lb.issue(lds0 + s * STAGE + A_BYTES, b_k0 + s * b_step, wid);
    }
  }
  // k-step 0 resident for every wave
  if (STAGES - 1 < nk)
    wait_vmcnt<PER_STAGE * (STAGES - 2)>();
  else
    wait_vmcnt<0>();
  auto barrier = [] {
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
  };
  barrier();
  if (grp == 1) barrier();  // group 1 runs one phase behind

  bf16x8_t af[KS][FM], bfr[KS][FN];
  for (int t = 0; t < nk; ++t) {
    // ---- load phase
    const int tl = t + STAGES - 1;
    if (tl < nk) {
      const uint32_t st = lds0 + (tl % STAGES) * STAGE;
      la.issue(st, a_k0 + tl * a_step, wid);
      lb.issue(st + A_BYTES, b_k0 + tl * b_step, wid);
    }
    const lds_char *As = smem + (t % STAGES) * STAGE;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
#pragma unroll
      for (int i = 0; i < FM; ++i) af[kk][i] = fa.get(As, i, kk);
#pragma unroll
      for (int j = 0; j < FN; ++j) bfr[kk][j] = fb.get(As + A_BYTES, j, kk);
    }
    // own share of k-step t+1 landed (k-steps t+2.. may still be in flight)
    if (t + STAGES - 1 < nk)
      wait_vmcnt<PER_STAGE * (STAGES - 2), 0>();
    else
      wait_vmcnt<0, 0>();
    barrier();
    // ---- compute phase
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32(bfr[kk][j], af[kk][i], acc[i][j]);
      if constexpr (kDb) {
        if (do_db) {
#pragma unroll
          for (int i = 0; i < FM; ++i) {
            const u32x4_t w = __builtin_bit_cast(u32x4_t, af[kk][i]);
#pragma unroll
            for (int e = 0; e < 4; ++e) dbacc[i] += lo_bf(w[e]) + hi_bf(w[e]);
          }
        }
      }
    }
    barrier();
  }
  if (grp == 0) barrier();  // match group 1's extra barrier

  const GemmArgs q = split_outputs(p, split);
  store_tile_lds<EPI, BM, BN, WM, WN>(q, acc, m0, n0, wm, wn, lane, reinterpret_cast<float *>(smem_raw));
  if constexpr (kDb) {
    if (do_db) {
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const float tot = dbacc[i] + __shfl_xor(dbacc[i], 32, kWave);
        const int row = m0 + wm * WTM + i * 32 + (lane & 31);
        if (lane < 32 && row < q.M) q.db[row] = q.accumulate ? q.db[row] + tot : tot;
      }
    }
  }
}

template <int BM, int BN, int BK, int WM, int WN, int STAGES, bool AT, bool BT, Epi EPI>
bool launch_pp_cfg(const GemmArgs &a, uint32_t a_bytes, uint32_t b_bytes, hipStream_t s) {
  constexpr int NW = WM * WN;
  constexpr size_t lds = static_cast<size_t>(STAGES) *
                         (DirectLoader<BM, BK, NW, AT>::BYTES + DirectLoader<BN, BK, NW, BT>::BYTES);
  static_assert(lds <= 160 * 1024, "LDS budget");
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN) * (a.splits > 1 ? a.splits : 1);
  hipLaunchKernelGGL((gemm_pp_kernel<BM, BN, BK, WM, WN, STAGES, AT, BT, EPI>), dim3(tiles), dim3(NW * 64), lds, s, a,
                     a_bytes, b_bytes);
  return true;
}

// Direct-to-LDS path: pick the tile that minimises (rounds of 256 CUs) x
// (tile area / per-tile efficiency).  Measured on MI355X at the ViT-22B layer
// shapes with random bf16 data: 256x256 tiles are the most efficient per
// tile, 256x192 tiles divide the 6144- and 18432-wide outputs into whole
// rounds, 128x128 tiles serve small problems.  Kernel per tile and layout:
//   tile      forward (A, B k-contiguous)  input gradient (B strided)  weight gradient (both strided)
//   256x256   gemm_lds_kernel BK64 2-stage  gemm_pp_kernel BK32 4-stage  gemm_pp_kernel BK32 4-stage
//   256x192   gemm_lds_kernel BK64 2-stage  gemm_lds_kernel BK64 2-stage  gemm_pp_kernel BK32 4-stage
//             (K > 8192: gemm_deep_kernel)  (K > 20480: gemm_pp_kernel)
//   128x128   gemm_lds_kernel BK64 2-stage  gemm_lds_kernel BK64 2-stage  gemm_lds_kernel BK64 2-stage
// The ping-pong schedule hides the transpose reads of strided operands
// better where it is used; on the 256x192 input gradients it helps only with
// long contractions.
// Returns false when the operands do not fit the path's constraints.
template <bool AT, bool BT, Epi EPI>
bool launch_lds(const GemmArgs &a, hipStream_t s, TileShape t) {
  constexpr int BK = 64;
  if (!lds_fits(a.M, a.N, a.K, a.lda, a.ldb, AT, BT)) return false;
  // operand extents (bytes) bound the buffer loads
  const uint32_t ab = static_cast<uint32_t>(static_cast<uint64_t>(AT ? a.K : a.M) * a.lda * 2);
  const uint32_t bb = static_cast<uint32_t>(static_cast<uint64_t>(BT ? a.K : a.N) * a.ldb * 2);
  if (t.bm == 256 && t.bn == 256) {
    if constexpr (BT) return launch_pp_cfg<256, 256, 32, 2, 4, 4, AT, BT, EPI>(a, ab, bb, s);
    return launch_lds_cfg<256, 256, BK, 2, 4, 2, AT, BT, EPI>(a, ab, bb, s);
  }
  if (t.bm == 256 && t.bn == 192) {
    if constexpr (AT && BT) return launch_pp_cfg<256, 192, 32, 4, 2, 4, AT, BT, EPI>(a, ab, bb, s);
    if constexpr (!AT && BT) {
      if (a.K > kPpDgradMinK) return launch_pp_cfg<256, 192, 32, 4, 2, 4, AT, BT, EPI>(a, ab, bb, s);
    }
    if constexpr (!AT && !BT) {
      if (a.K > kDeepFwdMinK) return launch_deep_cfg<256, 192, BK, 4, 2, true, false, EPI>(a, ab, bb, s);
    }
    return launch_lds_cfg<256, 192, BK, 4, 2, 2, AT, BT, EPI>(a, ab, bb, s);
  }
  if (t.bm == 256) return launch_lds_cfg<256, 128, BK, 4, 2, 2, AT, BT, EPI>(a, ab, bb, s);
  if (t.bn == 256) return launch_lds_cfg<128, 256, BK, 2, 4, 2, AT, BT, EPI>(a, ab, bb, s);
  return launch_lds_cfg<128, 128, BK, 2, 2, 2, AT, BT, EPI>(a, ab, bb, s);
}

template <bool AT, bool BT, Epi EPI>
bool launch_lds(const GemmArgs &a, hipStream_t s) {
  return launch_lds<AT, BT, EPI>(a, s, choose_tile(a.M, a.N, AT && BT));
}

}  // namespace

namespace {

// Sum of the fp32 partials [S][M][N] in split order, then the epilogue of
// the unsplit kernel: bias, residual, GELU (writing u and g) or GELU' (from
// the saved u in R), rounded once to bf16.  Eight outputs per thread and
// iteration (N is a multiple of 8).
template <Epi EPI>
__global__ __launch_bounds__(256) void splitk_epilogue_kernel(const float *__restrict__ part, int splits,
                                                              size_t stride, int M, int N,
                                                              const bf16_t *__restrict__ bias,
                                                              const bf16_t *__restrict__ R, bf16_t *__restrict__ Y,
                                                              bf16_t *__restrict__ Y2) {
  const long n8 = static_cast<long>(M) * N / 8;
  for (long i = blockIdx.x * 256L + threadIdx.x; i < n8; i += static_cast<long>(gridDim.x) * 256) {
    const size_t e0 = static_cast<size_t>(i) * 8;
    f32x4_t lo = *reinterpret_cast<const f32x4_t *>(part + e0);
    f32x4_t hi = *reinterpret_cast<const f32x4_t *>(part + e0 + 4);
    for (int sp = 1; sp < splits; ++sp) {
      lo += *reinterpret_cast<const f32x4_t *>(part + sp * stride + e0);
      hi += *reinterpret_cast<const f32x4_t *>(part + sp * stride + e0 + 4);
    }
    float v[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    if constexpr (EPI == Epi::kBias || EPI == Epi::kBiasResid || EPI == Epi::kBiasGelu) {
      const u32x4_t bw = ldg16(bias + e0 % N);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[2 * e] += lo_bf(bw[e]);
        v[2 * e + 1] += hi_bf(bw[e]);
      }
    }
    if constexpr (EPI == Epi::kBiasResid || EPI == Epi::kResid) {
      const u32x4_t rw = ldg16(R + e0);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[2 * e] += lo_bf(rw[e]);
        v[2 * e + 1] += hi_bf(rw[e]);
      }
    }
    if constexpr (EPI == Epi::kGeluGrad) {
      const u32x4_t uw = ldg16(R + e0);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[2 * e] *= gelu_grad_f(lo_bf(uw[e]));
        v[2 * e + 1] *= gelu_grad_f(hi_bf(uw[e]));
      }
    }
    u32x4_t o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = pack2(v[2 * e], v[2 * e + 1]);
    stg16_nt(Y + e0, o);
    if constexpr (EPI == Epi::kBiasGelu) {
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = pack2(gelu_f(v[2 * e]), gelu_f(v[2 * e + 1]));
      stg16_nt(Y2 + e0, o);
    }
  }
}

// Split launch of a forward (AT = false, BT = false) or input-gradient
// (BT = true) product: fp32 partials into ws, then the epilogue kernel.
// Returns false (nothing launched) when the plan does not split or ws is
// missing or too small.
template <bool BT, Epi EPI>
bool launch_split(const GemmArgs &a, void *ws, size_t ws_bytes, hipStream_t s) {
  const SplitPlan sp = gemm_split_plan(a.M, a.N, a.K);
  if (sp.splits <= 1 || ws == nullptr || ws_bytes < gemm_ws_bytes(a.M, a.N, a.K) || a.ldy != a.N || a.N % 8)
    return false;
  GemmArgs b = a;
  b.splits = sp.splits;
  b.k_chunk = sp.k_chunk;
  b.split_stride = static_cast<size_t>(a.M) * a.N;
  b.Wf = static_cast<float *>(ws);
  b.db = nullptr;
  b.accumulate = 0;
  if (!launch_lds<false, BT, Epi::kF32>(b, s, sp.tile)) return false;
  const long n8 = static_cast<long>(a.M) * a.N / 8;
  const int blocks = static_cast<int>(std::min<long>((n8 + 255) / 256, 2048));
  hipLaunchKernelGGL((splitk_epilogue_kernel<EPI>), dim3(blocks), dim3(256), 0, s, b.Wf, sp.splits, b.split_stride,
                     a.M, a.N, a.bias, a.R, a.Y, a.Y2);
  return true;
}

template <Epi EPI>
bool fwd_any(const GemmArgs &a, void *ws, size_t ws_bytes, hipStream_t s) {
  return launch_split<false, EPI>(a, ws, ws_bytes, s) || launch_lds<false, false, EPI>(a, s) ||
         launch_any<false, false, EPI>(a, s);
}

template <Epi EPI>
bool dgrad_any(const GemmArgs &a, void *ws, size_t ws_bytes, hipStream_t s) {
  return launch_split<true, EPI>(a, ws, ws_bytes, s) || launch_lds<false, true, EPI>(a, s) ||
         launch_any<false, true, EPI>(a, s);
}

}  // namespace

bool launch_gemm_fwd(const GemmArgs &a, Epi epi, void *ws, size_t ws_bytes, hipStream_t s) {
  switch (epi) {
    case Epi::kBias: return fwd_any<Epi::kBias>(a, ws, ws_bytes, s);
    case Epi::kBiasResid: return fwd_any<Epi::kBiasResid>(a, ws, ws_bytes, s);
    case Epi::kBiasGelu: return fwd_any<Epi::kBiasGelu>(a, ws, ws_bytes, s);
    case Epi::kPlain: return fwd_any<Epi::kPlain>(a, ws, ws_bytes, s);
    default: return false;
  }
}

bool launch_gemm_dgrad(const GemmArgs &a, Epi epi, void *ws, size_t ws_bytes, hipStream_t s) {
  switch (epi) {
    case Epi::kPlain: return dgrad_any<Epi::kPlain>(a, ws, ws_bytes, s);
    case Epi::kGeluGrad: return dgrad_any<Epi::kGeluGrad>(a, ws, ws_bytes, s);
    case Epi::kResid: return dgrad_any<Epi::kResid>(a, ws, ws_bytes, s);
    default: return false;
  }
}

namespace {

// out[i] = (accumulate ? out[i] : 0) + part[0][i] + part[1][i] + ... in split
// order (deterministic), over n4 float4s; blockIdx.y picks the dW or the db
// segment.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(float *__restrict__ w, const float *__restrict__ wp,
                                                            long w4, float *__restrict__ b,
                                                            const float *__restrict__ bp, long b4, int splits,
                                                            int accumulate) {
  float *out = blockIdx.y == 0 ? w : b;
  const float *part = blockIdx.y == 0 ? wp : bp;
  const long n4 = blockIdx.y == 0 ? w4 : b4;
  for (long i = blockIdx.x * 256L + threadIdx.x; i < n4; i += static_cast<long>(gridDim.x) * 256) {
    f32x4_t v = accumulate ? reinterpret_cast<const f32x4_t *>(out)[i] : f32x4_t{0.f, 0.f, 0.f, 0.f};
    for (int sp = 0; sp < splits; ++sp) v += reinterpret_cast<const f32x4_t *>(part)[sp * n4 + i];
    reinterpret_cast<f32x4_t *>(out)[i] = v;
  }
}

}  // namespace

bool launch_gemm_wgrad(const GemmArgs &a, void *ws, size_t ws_bytes, hipStream_t s) {
  // both paths fuse the bias gradient into the weight-gradient kernel
  const SplitPlan sp = wgrad_split_plan(a.M, a.N, a.K);
  if (sp.splits > 1 && ws != nullptr && ws_bytes >= gemm_wgrad_ws_bytes(a.M, a.N, a.K) && a.ldy == a.N &&
      a.M % 4 == 0 && a.N % 4 == 0) {
    GemmArgs b = a;
    b.splits = sp.splits;
    b.k_chunk = sp.k_chunk;
    b.split_stride = static_cast<size_t>(a.M) * a.N;
    b.Wf = static_cast<float *>(ws);
    b.db = a.db ? b.Wf + ws_round256(static_cast<size_t>(sp.splits) * a.M * a.N * sizeof(float)) / sizeof(float)
                : nullptr;
    b.accumulate = 0;
    if (launch_lds<true, true, Epi::kF32>(b, s, sp.tile)) {
      const long w4 = static_cast<long>(a.M) * a.N / 4, b4 = a.db ? a.M / 4 : 0;
      const int blocks = static_cast<int>(std::min<long>((w4 + 255) / 256, 2048));
      hipLaunchKernelGGL(splitk_reduce_kernel, dim3(blocks, a.db ? 2 : 1), dim3(256), 0, s, a.Wf, b.Wf, w4, a.db,
                         b.db, b4, sp.splits, a.accumulate);
      return true;
    }
  }
  return launch_lds<true, true, Epi::kF32>(a, s) || launch_any<true, true, Epi::kF32>(a, s);
}

}  // namespace optimus
