// Fused multi-head attention, forward and backward, for gfx950.
//
// Layout: qkv is [B*S, 3*heads*D] with columns [3][heads][D]; o, dO are
// [B*S, heads*D]; lse and the backward's D vector are [B, heads, S] fp32.
//
// Every product is a v_mfma_f32_32x32x16_bf16 with the *key/query-transposed*
// orientation: the forward computes S^T = K Q^T, so each lane of the 32x32
// result owns one query and holds that query's logits for 16 keys.  The row
// max and row sum of the online softmax are then in-lane reductions plus one
// exchange with lane^32, and the exponentiated tile is already laid out as
// the B operand of O^T += V^T P^T once the key order inside each 16-key step
// is permuted the same way in both operands (lane half h holds keys
// 4h..4h+3 and 8+4h..8+4h+3).  V^T is staged in LDS as [d][key] through an
// 8x8 register transpose, so the A operand is two 8-byte LDS reads.  Head
// dims 64, 80 and 128 contract in 16-wide steps; the O^T rows are padded to
// a multiple of 32 (80 -> 96) and the padding rows are never stored.
//
// The backward is two kernels and uses no atomics: one per query tile that
// recomputes P^T and dP^T and accumulates dQ^T = K^T dS^T over all keys (and
// writes D_i = dO_i . O_i), then one per key tile that recomputes P and dP
// and accumulates dV^T = dO^T P and dK^T = Q^T dS over all queries.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace optimus {

namespace {

constexpr int kKT = 64;     // keys (forward, dQ) or queries (dK/dV) per LDS tile
constexpr int kRows = 128;  // queries (or keys) per workgroup: 4 waves x 32
constexpr float kLog2e = 1.4426950408889634f;

template <int D>
struct Head {
  static constexpr int KS = D / 16;              // 16-wide contraction steps over d
  static constexpr int NF = (D + 31) / 32;       // 32-row fragments of a d-major result
  static constexpr int DP = NF * 32;             // padded d rows
  static constexpr int LDR = D + 8;              // LDS row stride of [token][d] tiles
  static constexpr int LDT = kKT + 8;            // LDS row stride of [d][token] tiles
};

__device__ __forceinline__ bf16x8_t lds_b128(const bf16_t *p) { return *reinterpret_cast<const bf16x8_t *>(p); }

// Two 8-byte LDS reads forming one MFMA operand in the permuted key order.
__device__ __forceinline__ bf16x8_t lds_perm(const bf16_t *row, int step, int hf) {
  const u32x2_t a = *reinterpret_cast<const u32x2_t *>(row + step * 16 + 4 * hf);
  const u32x2_t b = *reinterpret_cast<const u32x2_t *>(row + step * 16 + 8 + 4 * hf);
  return as_bf16x8(u32x4_t{a[0], a[1], b[0], b[1]});
}

// Pack eight fp32 (registers 8*half .. 8*half+7 of a 32x32 result) to bf16.
__device__ __forceinline__ bf16x8_t pack8(const f32x16_t &v, int half) {
  u32x4_t r;
#pragma unroll
  for (int e = 0; e < 4; ++e) r[e] = pack2(v[8 * half + 2 * e], v[8 * half + 2 * e + 1]);
  return as_bf16x8(r);
}

// Row-major [kKT][D] tile of tokens t0.. (rows >= S zero-filled).
template <int D>
__device__ __forceinline__ void stage_rows(bf16_t *dst, const bf16_t *src, int ld, int t0, int S, int tid) {
  constexpr int C = D / 8;
  for (int c = tid; c < kKT * C; c += 256) {
    const int t = c / C, dc = c % C;
    u32x4_t v{0u, 0u, 0u, 0u};
    if (t0 + t < S) v = ldg16(src + static_cast<size_t>(t0 + t) * ld + dc * 8);
    *reinterpret_cast<u32x4_t *>(dst + t * Head<D>::LDR + dc * 8) = v;
  }
}

// Transposed [D][kKT] tile (d-major, tokens contiguous) via 8x8 register blocks.
template <int D>
__device__ __forceinline__ void stage_cols(bf16_t *dst, const bf16_t *src, int ld, int t0, int S, int tid) {
  constexpr int NB = (kKT / 8) * (D / 8);
  if (tid < NB) {
    const int tb = tid % (kKT / 8), db = tid / (kKT / 8);
    u32x4_t in[8], out[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int t = t0 + tb * 8 + j;
      in[j] = (t < S) ? ldg16(src + static_cast<size_t>(t) * ld + db * 8) : u32x4_t{0u, 0u, 0u, 0u};
    }
    transpose8x8(in, out);
#pragma unroll
    for (int i = 0; i < 8; ++i)
      *reinterpret_cast<u32x4_t *>(dst + (db * 8 + i) * Head<D>::LDT + tb * 8) = out[i];
  }
}

// Load this lane's token row (d values 16*kk + 8*hf .. +7 for each step kk)
// as B operands; zero for tokens >= S.
template <int D>
__device__ __forceinline__ void load_row_operand(bf16x8_t (&f)[Head<D>::KS], const bf16_t *src, bool valid,
                                                 int hf) {
#pragma unroll
  for (int kk = 0; kk < Head<D>::KS; ++kk)
    f[kk] = valid ? as_bf16x8(ldg16(src + kk * 16 + hf * 8)) : as_bf16x8(u32x4_t{0u, 0u, 0u, 0u});
}

// Store a d-major 32x32 fragment set (rows d, lane = token) scaled by s.
template <int D>
__device__ __forceinline__ void store_dmajor(bf16_t *dst, const f32x16_t (&acc)[Head<D>::NF], float s, int hf) {
#pragma unroll
  for (int nf = 0; nf < Head<D>::NF; ++nf) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int d0 = nf * 32 + q * 8 + hf * 4;
      if (d0 < D) {
        *reinterpret_cast<u32x2_t *>(dst + d0) =
            u32x2_t{pack2(acc[nf][4 * q] * s, acc[nf][4 * q + 1] * s), pack2(acc[nf][4 * q + 2] * s, acc[nf][4 * q + 3] * s)};
      }
    }
  }
}

// ------------------------------------------------------------------ forward

template <int D>
__global__ __launch_bounds__(256) void attn_fwd_kernel(int B, int S, int heads, const bf16_t *__restrict__ qkv,
                                                       bf16_t *__restrict__ o, float *__restrict__ lse) {
  using H = Head<D>;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[kKT * H::LDR];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[H::DP * H::LDT];

  const int nqt = (S + kRows - 1) / kRows;
  const int qt = blockIdx.x % nqt;
  const int bh = blockIdx.x / nqt;
  const int b = bh / heads, h = bh % heads;
  const int A = heads * D, ld = 3 * A;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, hf = lane >> 5;
  const int q = qt * kRows + wid * 32 + (lane & 31);
  const bool qvalid = q < S;
  const bf16_t *base = qkv + static_cast<size_t>(b) * S * ld;
  const bf16_t *kbase = base + A + h * D;
  const bf16_t *vbase = base + 2 * A + h * D;

  bf16x8_t qf[H::KS];
  load_row_operand<D>(qf, base + static_cast<size_t>(q) * ld + h * D, qvalid, hf);

  f32x16_t acc[H::NF];
#pragma unroll
  for (int i = 0; i < H::NF; ++i) acc[i] = f32x16_t{};
  float m = -INFINITY, l = 0.f;
  const float c = kLog2e / sqrtf(static_cast<float>(D));

  for (int k0 = 0; k0 < S; k0 += kKT) {
    __syncthreads();
    stage_rows<D>(Ks, kbase, ld, k0, S, tid);
    stage_cols<D>(Vt, vbase, ld, k0, S, tid);
    __syncthreads();

    f32x16_t s[2];
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      s[f] = f32x16_t{};
#pragma unroll
      for (int kk = 0; kk < H::KS; ++kk)
        s[f] = mfma32(lds_b128(Ks + (f * 32 + (lane & 31)) * H::LDR + kk * 16 + hf * 8), qf[kk], s[f]);
    }
    float mt = m;
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = k0 + f * 32 + (i >> 2) * 8 + hf * 4 + (i & 3);
        const float x = (key < S) ? s[f][i] * c : -INFINITY;
        s[f][i] = x;
        mt = fmaxf(mt, x);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 32, kWave));
    const float alpha = exp2f(m - mt);
    m = mt;
    float ls = 0.f;
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = exp2f(s[f][i] - mt);
        s[f][i] = p;
        ls += p;
      }
    l = l * alpha + ls;
#pragma unroll
    for (int nf = 0; nf < H::NF; ++nf) acc[nf] *= alpha;
#pragma unroll
    for (int st = 0; st < kKT / 16; ++st) {
      const bf16x8_t pb = pack8(s[st >> 1], st & 1);
#pragma unroll
      for (int nf = 0; nf < H::NF; ++nf)
        acc[nf] = mfma32(lds_perm(Vt + (nf * 32 + (lane & 31)) * H::LDT, st, hf), pb, acc[nf]);
    }
  }

  const float lt = l + __shfl_xor(l, 32, kWave);
  if (qvalid) {
    store_dmajor<D>(o + (static_cast<size_t>(b) * S + q) * A + h * D, acc, 1.0f / lt, hf);
    if (hf == 0) lse[static_cast<size_t>(bh) * S + q] = (m + log2f(lt)) / kLog2e;
  }
}

// ------------------------------------------------------------------ backward: dQ and D

template <int D>
__global__ __launch_bounds__(256) void attn_bwd_dq_kernel(int B, int S, int heads, const bf16_t *__restrict__ qkv,
                                                          const bf16_t *__restrict__ o, const float *__restrict__ lse,
                                                          const bf16_t *__restrict__ dO, bf16_t *__restrict__ dqkv,
                                                          float *__restrict__ dvec) {
  using H = Head<D>;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[kKT * H::LDR];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[kKT * H::LDR];
  __shared__ __attribute__((aligned(16))) bf16_t Kt[H::DP * H::LDT];

  const int nqt = (S + kRows - 1) / kRows;
  const int qt = blockIdx.x % nqt;
  const int bh = blockIdx.x / nqt;
  const int b = bh / heads, h = bh % heads;
  const int A = heads * D, ld = 3 * A;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, hf = lane >> 5;
  const int q = qt * kRows + wid * 32 + (lane & 31);
  const bool qvalid = q < S;
  const bf16_t *base = qkv + static_cast<size_t>(b) * S * ld;
  const bf16_t *kbase = base + A + h * D;
  const bf16_t *vbase = base + 2 * A + h * D;
  const size_t orow = (static_cast<size_t>(b) * S + q) * A + h * D;

  bf16x8_t qf[H::KS], df[H::KS];
  load_row_operand<D>(qf, base + static_cast<size_t>(q) * ld + h * D, qvalid, hf);
  load_row_operand<D>(df, dO + orow, qvalid, hf);

  // D_i = dO_i . O_i (this lane holds half of the d values of its query)
  float dd = 0.f;
  if (qvalid) {
#pragma unroll
    for (int kk = 0; kk < H::KS; ++kk) {
      const u32x4_t ow = ldg16(o + orow + kk * 16 + hf * 8);
      const u32x4_t dw = __builtin_bit_cast(u32x4_t, df[kk]);
#pragma unroll
      for (int e = 0; e < 4; ++e) dd += lo_bf(ow[e]) * lo_bf(dw[e]) + hi_bf(ow[e]) * hi_bf(dw[e]);
    }
  }
  dd += __shfl_xor(dd, 32, kWave);
  const float c = kLog2e / sqrtf(static_cast<float>(D));
  const float lse2 = qvalid ? lse[static_cast<size_t>(bh) * S + q] * kLog2e : 0.f;
  if (qvalid && hf == 0) dvec[static_cast<size_t>(bh) * S + q] = dd;

  f32x16_t acc[H::NF];
#pragma unroll
  for (int i = 0; i < H::NF; ++i) acc[i] = f32x16_t{};

  for (int k0 = 0; k0 < S; k0 += kKT) {
    __syncthreads();
    stage_rows<D>(Ks, kbase, ld, k0, S, tid);
    stage_rows<D>(Vs, vbase, ld, k0, S, tid);
    stage_cols<D>(Kt, kbase, ld, k0, S, tid);
    __syncthreads();

    f32x16_t s[2], dp[2];
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      s[f] = f32x16_t{};
      dp[f] = f32x16_t{};
#pragma unroll
      for (int kk = 0; kk < H::KS; ++kk) {
        s[f] = mfma32(lds_b128(Ks + (f * 32 + (lane & 31)) * H::LDR + kk * 16 + hf * 8), qf[kk], s[f]);
        dp[f] = mfma32(lds_b128(Vs + (f * 32 + (lane & 31)) * H::LDR + kk * 16 + hf * 8), df[kk], dp[f]);
      }
    }
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = k0 + f * 32 + (i >> 2) * 8 + hf * 4 + (i & 3);
        const float p = (key < S) ? exp2f(s[f][i] * c - lse2) : 0.f;
        s[f][i] = p * (dp[f][i] - dd);  // dS^T
      }
#pragma unroll
    for (int st = 0; st < kKT / 16; ++st) {
      const bf16x8_t pb = pack8(s[st >> 1], st & 1);
#pragma unroll
      for (int nf = 0; nf < H::NF; ++nf)
        acc[nf] = mfma32(lds_perm(Kt + (nf * 32 + (lane & 31)) * H::LDT, st, hf), pb, acc[nf]);
    }
  }
  if (qvalid)
    store_dmajor<D>(dqkv + (static_cast<size_t>(b) * S + q) * ld + h * D, acc, 1.0f / sqrtf(static_cast<float>(D)),
                    hf);
}

// ------------------------------------------------------------------ backward: dK, dV

template <int D>
__global__ __launch_bounds__(256) void attn_bwd_dkdv_kernel(int B, int S, int heads, const bf16_t *__restrict__ qkv,
                                                            const float *__restrict__ lse,
                                                            const bf16_t *__restrict__ dO,
                                                            const float *__restrict__ dvec,
                                                            bf16_t *__restrict__ dqkv) {
  using H = Head<D>;
  __shared__ __attribute__((aligned(16))) bf16_t Qs[kKT * H::LDR];
  __shared__ __attribute__((aligned(16))) bf16_t Ds[kKT * H::LDR];
  __shared__ __attribute__((aligned(16))) bf16_t Qt[H::DP * H::LDT];
  __shared__ __attribute__((aligned(16))) bf16_t Dt[H::DP * H::LDT];
  __shared__ __attribute__((aligned(16))) float Ls[kKT];
  __shared__ __attribute__((aligned(16))) float Dv[kKT];

  const int nkt = (S + kRows - 1) / kRows;
  const int kt = blockIdx.x % nkt;
  const int bh = blockIdx.x / nkt;
  const int b = bh / heads, h = bh % heads;
  const int A = heads * D, ld = 3 * A;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, hf = lane >> 5;
  const int key = kt * kRows + wid * 32 + (lane & 31);
  const bool kvalid = key < S;
  const bf16_t *base = qkv + static_cast<size_t>(b) * S * ld;
  const bf16_t *qbase = base + h * D;
  const bf16_t *dobase = dO + static_cast<size_t>(b) * S * A + h * D;

  bf16x8_t kf[H::KS], vf[H::KS];
  load_row_operand<D>(kf, base + static_cast<size_t>(key) * ld + A + h * D, kvalid, hf);
  load_row_operand<D>(vf, base + static_cast<size_t>(key) * ld + 2 * A + h * D, kvalid, hf);

  f32x16_t dk[H::NF], dv[H::NF];
#pragma unroll
  for (int i = 0; i < H::NF; ++i) dk[i] = dv[i] = f32x16_t{};
  const float c = kLog2e / sqrtf(static_cast<float>(D));

  for (int q0 = 0; q0 < S; q0 += kKT) {
    __syncthreads();
    stage_rows<D>(Qs, qbase, ld, q0, S, tid);
    stage_rows<D>(Ds, dobase, A, q0, S, tid);
    stage_cols<D>(Qt, qbase, ld, q0, S, tid);
    stage_cols<D>(Dt, dobase, A, q0, S, tid);
    if (tid < kKT) {
      const int qq = q0 + tid;
      // queries past the end get lse = +inf (P = 0) and D = 0
      Ls[tid] = (qq < S) ? lse[static_cast<size_t>(bh) * S + qq] * kLog2e : INFINITY;
      Dv[tid] = (qq < S) ? dvec[static_cast<size_t>(bh) * S + qq] : 0.f;
    }
    __syncthreads();

    f32x16_t s[2], dp[2];
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      s[f] = f32x16_t{};
      dp[f] = f32x16_t{};
#pragma unroll
      for (int kk = 0; kk < H::KS; ++kk) {
        s[f] = mfma32(lds_b128(Qs + (f * 32 + (lane & 31)) * H::LDR + kk * 16 + hf * 8), kf[kk], s[f]);
        dp[f] = mfma32(lds_b128(Ds + (f * 32 + (lane & 31)) * H::LDR + kk * 16 + hf * 8), vf[kk], dp[f]);
      }
    }
    // s[f][i] is query f*32 + 8*(i/4) + 4*hf + i%4 of this tile, key = this lane
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int qi = f * 32 + g * 8 + hf * 4;
        const f32x4_t l4 = *reinterpret_cast<const f32x4_t *>(Ls + qi);
        const f32x4_t d4 = *reinterpret_cast<const f32x4_t *>(Dv + qi);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p = exp2f(s[f][4 * g + e] * c - l4[e]);
          s[f][4 * g + e] = p;
          dp[f][4 * g + e] = p * (dp[f][4 * g + e] - d4[e]);
        }
      }
#pragma unroll
    for (int st = 0; st < kKT / 16; ++st) {
      const bf16x8_t pb = pack8(s[st >> 1], st & 1);
      const bf16x8_t sb = pack8(dp[st >> 1], st & 1);
#pragma unroll
      for (int nf = 0; nf < H::NF; ++nf) {
        dv[nf] = mfma32(lds_perm(Dt + (nf * 32 + (lane & 31)) * H::LDT, st, hf), pb, dv[nf]);
        dk[nf] = mfma32(lds_perm(Qt + (nf * 32 + (lane & 31)) * H::LDT, st, hf), sb, dk[nf]);
      }
    }
  }
  if (kvalid) {
    bf16_t *row = dqkv + (static_cast<size_t>(b) * S + key) * ld + h * D;
    store_dmajor<D>(row + A, dk, 1.0f / sqrtf(static_cast<float>(D)), hf);
    store_dmajor<D>(row + 2 * A, dv, 1.0f, hf);
  }
}

template <int D>
void launch_fwd_d(int B, int S, int heads, const bf16_t *qkv, bf16_t *o, float *lse, hipStream_t s) {
  const int blocks = B * heads * ((S + kRows - 1) / kRows);
  hipLaunchKernelGGL(attn_fwd_kernel<D>, dim3(blocks), dim3(256), 0, s, B, S, heads, qkv, o, lse);
}

template <int D>
void launch_bwd_d(int B, int S, int heads, const bf16_t *qkv, const bf16_t *o, const float *lse, const bf16_t *dO,
                  bf16_t *dqkv, float *dvec, hipStream_t s) {
  const int blocks = B * heads * ((S + kRows - 1) / kRows);
  hipLaunchKernelGGL(attn_bwd_dq_kernel<D>, dim3(blocks), dim3(256), 0, s, B, S, heads, qkv, o, lse, dO, dqkv, dvec);
  hipLaunchKernelGGL(attn_bwd_dkdv_kernel<D>, dim3(blocks), dim3(256), 0, s, B, S, heads, qkv, lse, dO, dvec, dqkv);
}

}  // namespace

size_t attn_bwd_ws_bytes(int B, int S, int heads) {
  return static_cast<size_t>(B) * heads * S * sizeof(float);
}

bool launch_attn_fwd(int B, int S, int heads, int d, const bf16_t *qkv, bf16_t *o, float *lse, hipStream_t s) {
  switch (d) {
    case 64: launch_fwd_d<64>(B, S, heads, qkv, o, lse, s); return true;
    case 80: launch_fwd_d<80>(B, S, heads, qkv, o, lse, s); return true;
    case 128: launch_fwd_d<128>(B, S, heads, qkv, o, lse, s); return true;
    default: return false;
  }
}

bool launch_attn_bwd(int B, int S, int heads, int d, const bf16_t *qkv, const bf16_t *o, const float *lse,
                     const bf16_t *dO, bf16_t *dqkv, float *dvec, hipStream_t s) {
  switch (d) {
    case 64: launch_bwd_d<64>(B, S, heads, qkv, o, lse, dO, dqkv, dvec, s); return true;
    case 80: launch_bwd_d<80>(B, S, heads, qkv, o, lse, dO, dqkv, dvec, s); return true;
    case 128: launch_bwd_d<128>(B, S, heads, qkv, o, lse, dO, dqkv, dvec, s); return true;
    default: return false;
  }
}

}  // namespace optimus
