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
// so logical tile ids are remapped to give each XCD one contiguous range,
// ordered M-fastest in groups, which keeps each weight slab in one XCD's L2.
#include "common.hpp"
#include "kernels.hpp"

namespace optimus {

namespace {

__device__ __forceinline__ float gelu_f(float u) { return 0.5f * u * (1.0f + erff(u * 0.70710678118654752f)); }

__device__ __forceinline__ float gelu_grad_f(float u) {
  const float Phi = 0.5f * (1.0f + erff(u * 0.70710678118654752f));
  const float phi = expf(-0.5f * u * u) * 0.39894228040143268f;
  return Phi + u * phi;
}

// Logical tile id for this workgroup: contiguous per XCD, then grouped so
// that GROUP_M row tiles sweep one column tile before moving on.
__device__ __forceinline__ void tile_of(int tiles_m, int tiles_n, int &tm, int &tn) {
  const int pid = blockIdx.x, nb = gridDim.x;
  const int xcd = pid & 7, local = pid >> 3;
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

  // ---- epilogue: lane owns row m, columns nb..nb+3 of each 32x32 fragment
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
          if constexpr (EPI == Epi::kBiasResid) {
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
  const long big = static_cast<long>((a.M + 255) / 256) * ((a.N + 127) / 128);
  if (big >= 512) return launch_cfg<256, 128, 64, 2, 2, AT, BT, EPI>(a, s);
  return launch_cfg<128, 128, 64, 2, 2, AT, BT, EPI>(a, s);
}

}  // namespace

bool launch_gemm_fwd(const GemmArgs &a, Epi epi, hipStream_t s) {
  switch (epi) {
    case Epi::kBias: return launch_any<false, false, Epi::kBias>(a, s);
    case Epi::kBiasResid: return launch_any<false, false, Epi::kBiasResid>(a, s);
    case Epi::kBiasGelu: return launch_any<false, false, Epi::kBiasGelu>(a, s);
    default: return false;
  }
}

bool launch_gemm_dgrad(const GemmArgs &a, Epi epi, hipStream_t s) {
  switch (epi) {
    case Epi::kPlain: return launch_any<false, true, Epi::kPlain>(a, s);
    case Epi::kGeluGrad: return launch_any<false, true, Epi::kGeluGrad>(a, s);
    default: return false;
  }
}

bool launch_gemm_wgrad(const GemmArgs &a, hipStream_t s) { return launch_any<true, true, Epi::kF32>(a, s); }

}  // namespace optimus
