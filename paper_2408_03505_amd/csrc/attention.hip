// Fused multi-head attention, forward and backward, for gfx950.
//
// Layout: qkv is [B*S, 3*heads*D] with columns [3][heads][D]; o, dO are
// [B*S, heads*D]; lse and the backward's D vector are [B, heads, S] fp32.
//
// Every product is a v_mfma_f32_32x32x16_bf16 with the *key/query-transposed*
// orientation: the forward computes S^T = K Q^T, so each lane of the 32x32
// result owns one query and holds that query's logits for 16 keys.  The row
// max and row sum of the online softmax are then in-lane reductions plus one
// exchange with lane^32, and the exponentiated tile is already the B operand
// of O^T += V^T P^T.  Token tiles of K, V (forward, dQ) or Q, dO (dK/dV) go
// HBM -> LDS by DMA, double-buffered, and the token-contracting products read
// their A operand with the LDS transpose read.  Head dims 64, 80 and 128
// contract in 16-wide steps; d-major results are padded to a multiple of 32
// rows (80 -> 96) and the padding rows are never stored.
//
// The backward is two kernels and uses no atomics: one per query tile that
// recomputes P^T and dP^T and accumulates dQ^T = K^T dS^T over all keys (and
// writes D_i = dO_i . O_i), then one per key tile that recomputes P and dP
// and accumulates dV^T = dO^T P and dK^T = Q^T dS over all queries.
#include <math.h>

#include <algorithm>
#include <atomic>
#include <mutex>

#include "common.hpp"
#include "kernels.hpp"
#include "lds_dma.hpp"

// Scratch of the allocation-free backward entry point: the D vector
// (D_i = dO_i . O_i per sequence, head and query, fp32) of calls whose caller
// cannot allocate a workspace.  Each GPU the library runs on holds its own
// copy until the process ends.  Host code never passes this name to a kernel
// (on the host it is a stand-in, not a device address): it uses the address
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) float scratch[optimus::kAttnScratchFloats];

namespace optimus {

namespace {

constexpr int kRows = 128;  // queries per forward workgroup: 4 waves x 32
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLazyRescale = 8.0f;  // forward: rescale when a query's maximum grows by more than 2^8
constexpr int kPrefetchMaxD = 80;     // head dims whose registers hold a tile's operands read ahead

// 2^x on the hardware exponential (v_exp_f32).  Every argument here is a
// logit minus a running maximum or the log-sum-exp, so x <= 0 up to rounding
// and -inf for masked keys: results lie in [0, 1] and those below the fp32
// normal range flush to zero, which only drops weights under 2^-126.
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// Work item (sequence-head bh, tile sub) of this workgroup.  The nsub blocks
// of one sequence-head read the same K/V (or Q/dO) tiles, so they are placed
// on one XCD (workgroup i runs on XCD i % 8) to share its L2: each XCD takes
// a contiguous range of items when the grid splits evenly over the 8 XCDs.
__device__ __forceinline__ void block_item(int nsub, int &bh, int &sub) {
  const int pid = blockIdx.x, nb = gridDim.x;
  const int item = (nb & 7) ? pid : (pid & 7) * (nb >> 3) + (pid >> 3);
  bh = item / nsub;
  sub = item % nsub;
}

template <int D>
struct Head {
  static constexpr int KS = D / 16;              // 16-wide contraction steps over d
  static constexpr int NF = (D + 31) / 32;       // 32-row fragments of a d-major result
};

// Pack eight fp32 (registers 8*half .. 8*half+7 of a 32x32 result) to bf16.
__device__ __forceinline__ bf16x8_t pack8(const f32x16_t &v, int half) {
  u32x4_t r;
#pragma unroll
  for (int e = 0; e < 4; ++e) r[e] = pack2(v[8 * half + 2 * e], v[8 * half + 2 * e + 1]);
  return as_bf16x8(r);
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

// Store a d-major result through this wave's 8 KB LDS slot.  The lane of
// token t holds d values in 8-byte runs, so direct stores would touch 32 rows
// per instruction; here the runs go to LDS row t (256-byte rows, 16-byte
// chunk c stored at c ^ (t % 16)), and each lane then writes whole 16-byte
// row segments: a quarter-wave covers one row, four rows per instruction.
// dst is the row of the wave's first token, ld the row stride (elements),
// ntok the wave's tokens inside the sequence (the rest are not stored).
template <int D>
__device__ __forceinline__ void store_dmajor_lds(bf16_t *dst, size_t ld, const f32x16_t (&acc)[Head<D>::NF], float s,
                                                 int lane, lds_char *slot, int ntok) {
  const int t = lane & 31, hf = lane >> 5;
#pragma unroll
  for (int nf = 0; nf < Head<D>::NF; ++nf) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int d0 = nf * 32 + q * 8 + hf * 4;
      if (d0 < D) {
        const int c = d0 >> 3;
        *reinterpret_cast<__attribute__((address_space(3))) u32x2_t *>(slot + t * 256 + ((c ^ (t & 15)) << 4) +
                                                                        hf * 8) =
            u32x2_t{pack2(acc[nf][4 * q] * s, acc[nf][4 * q + 1] * s), pack2(acc[nf][4 * q + 2] * s, acc[nf][4 * q + 3] * s)};
      }
    }
  }
  // LDS accesses of one wave run in order: the reads below see the writes
  const int j = lane & 15;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int r = i * 4 + (lane >> 4);
    if (j * 8 < D && r < ntok) {
      const u32x4_t v =
          *reinterpret_cast<const __attribute__((address_space(3))) u32x4_t *>(slot + r * 256 + ((j ^ (r & 15)) << 4));
      stg16(dst + r * ld + j * 8, v);
    }
  }
}

// ------------------------------------------------------------------ forward
//
// K and V tiles of KT tokens (32, or 64 on grids that leave CUs idle) go
// HBM -> LDS by DMA (double-buffered, no staging registers), rows of
// kDL = 128 columns taken from the head's first column (columns past
// head_dim belong to the neighbouring data and are never contracted; rows
// past the sequence re-read the tile's first row and are masked out of the
// softmax).  K is
// read as the A operand of S^T = K Q^T with ds_read_b128; V is read as the A
// operand of O^T += V^T P^T with ds_read_b64_tr_b16.  The transpose read
// delivers tokens in natural order while the P^T registers hold them with
// bits 2 and 3 of the token index swapped, so V rows are stored with that
// swap (perm23).  One XOR swizzle serves both read patterns: chunk c of tile
// row r sits at c ^ tsw(r), distinct over any 16 consecutive rows (the
// ds_read_b128 pattern) and spreading any 4 consecutive rows over disjoint
// 64-byte ranges (the transpose-read pattern).

constexpr int kDL = 128;  // LDS row length (elements)
constexpr int kMaxKT = 64;  // longest token tile of any kernel (bounds the DMA overhang past a tensor)

// Bytes of one tile of KT tokens (KT = 32: 8 KB; KT = 64: 16 KB).
template <int KT>
constexpr int tile_bytes() {
  return KT * kDL * 2;
}

__device__ __forceinline__ int tsw(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }
__device__ __forceinline__ int tile_off(int r, int c) { return r * (kDL * 2) + ((c ^ tsw(r)) << 4); }
__device__ __forceinline__ int perm23(int r) { return (r & ~0xC) | ((r & 4) << 1) | ((r & 8) >> 1); }

// Per-lane byte offsets of this wave's DMA loads of one tile (KT/4 loads of
// 1 KB per tile, split over NW waves; tile-relative: the tile's first row and
// column go in the scalar offset).  perm stores token perm23(r) in row r.
template <int KT, int NW>
struct TileLoads {
  static constexpr int N = KT / 4 / NW;  // 1 KB loads per wave per tile
  static_assert(N >= 1 && N * NW * 4 == KT, "tile rows must split evenly over the waves");
};

template <int KT, int NW, int N>
__device__ __forceinline__ void tile_voff(uint32_t (&v)[N], int wid, int lane, int ld, bool perm) {
  static_assert(N == TileLoads<KT, NW>::N, "one offset per load");
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const int o = (wid * N + i) * 1024 + lane * 16;
    const int pr = o >> 8, c = ((o & 255) >> 4) ^ tsw(pr);
    v[i] = static_cast<uint32_t>(((perm ? perm23(pr) : pr) * ld + c * 8) * 2);
  }
}

// Issue one tile's DMA loads.  In the last tile of a sequence (rem < KT
// rows left) the rows past the sequence re-read the tile's first row: every
// product with those rows carries a zero weight, but a non-finite value in
// the next sequence would still turn that zero into NaN.
template <int KT, int NW, int N>
__device__ __forceinline__ void tile_issue(const u32x4_t &rsrc, uint32_t lds_tile, const uint32_t (&voff)[N],
                                           uint32_t soff, int wid, int lane, int rem, int ld, bool perm) {
  static_assert(N == TileLoads<KT, NW>::N, "one offset per load");
  const uint32_t sl = __builtin_amdgcn_readfirstlane(soff);
  if (rem >= KT) {
#pragma unroll
    for (int i = 0; i < N; ++i)
      buffer_load_lds16(rsrc, __builtin_amdgcn_readfirstlane(lds_tile + (wid * N + i) * 1024), voff[i], sl);
  } else {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int pr = (wid * N + i) * 4 + (lane >> 4);
      const int tok = perm ? perm23(pr) : pr;
      const uint32_t v = tok < rem ? voff[i] : voff[i] - static_cast<uint32_t>(tok * ld * 2);
      buffer_load_lds16(rsrc, __builtin_amdgcn_readfirstlane(lds_tile + (wid * N + i) * 1024), v, sl);
    }
  }
}

// Wait for the oldest tile in flight: with `ahead` later tiles already issued
// (each L loads per wave) those may stay outstanding.
template <int L>
__device__ __forceinline__ void wait_tiles(int ahead) {
  if (ahead >= 2)
    wait_vmcnt<2 * L>();
  else if (ahead == 1)
    wait_vmcnt<L>();
  else
    wait_vmcnt<0>();
}

__device__ __forceinline__ void block_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// MFMA A operand (rows = tile rows rbase.., contraction = columns 16kk..) by ds_read_b128.
__device__ __forceinline__ bf16x8_t tile_rows(const lds_char *t, int rbase, int kk, int lane) {
  return *reinterpret_cast<const __attribute__((address_space(3))) bf16x8_t *>(
      t + tile_off(rbase + (lane & 31), kk * 2 + (lane >> 5)));
}

// MFMA A operand (rows = columns nbase.., contraction = tile rows 16st..) by
// two ds_read_b64_tr_b16.
__device__ __forceinline__ bf16x8_t tile_cols(const lds_char *t, int nbase, int st, int lane) {
  const int k = st * 16 + 8 * (lane >> 5) + ((lane & 15) >> 2);
  const int n = nbase + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const int in = (n & 7) * 2;
  return lds_read_tr(t + tile_off(k, n >> 3) + in, t + tile_off(k + 4, n >> 3) + in);
}

// As tile_cols, but contraction index kk reads tile row 16st + perm23(kk):
// the operand then meets registers whose tokens come in the order a
// 32x32 MFMA result leaves them (bits 2 and 3 of the token index swapped),
// so one natural-order tile serves both the row reads and this read.  The
// transpose read takes each source lane's row address; lane half h (lanes
// 32h..) supplies rows 4h + (lane % 16) / 4 for elements 0..3 and those
// rows + 8 for elements 4..7.
__device__ __forceinline__ bf16x8_t tile_cols_perm(const lds_char *t, int nbase, int st, int lane) {
  const int k = st * 16 + 4 * (lane >> 5) + ((lane & 15) >> 2);
  const int n = nbase + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const int in = (n & 7) * 2;
  return lds_read_tr(t + tile_off(k, n >> 3) + in, t + tile_off(k + 8, n >> 3) + in);
}

// A operands of a token-contracting product (columns nf*32.. of a tile,
// contraction over its rows), read ahead of the work they wait on when the
// head is small enough for the registers (PRE); otherwise read at use.
template <int D, int KT, bool PRE, bool PERM>
struct ColOperands {
  bf16x8_t v[PRE ? KT / 16 : 1][PRE ? Head<D>::NF : 1];
  __device__ __forceinline__ void fetch(const lds_char *t, int lane) {
    if constexpr (PRE) {
#pragma unroll
      for (int st = 0; st < KT / 16; ++st)
#pragma unroll
        for (int nf = 0; nf < Head<D>::NF; ++nf)
          v[st][nf] = PERM ? tile_cols_perm(t, nf * 32, st, lane) : tile_cols(t, nf * 32, st, lane);
    }
  }
  __device__ __forceinline__ bf16x8_t get(const lds_char *t, int nf, int st, int lane) const {
    if constexpr (PRE)
      return v[st][nf];
    else
      return PERM ? tile_cols_perm(t, nf * 32, st, lane) : tile_cols(t, nf * 32, st, lane);
  }
};

template <int D, int KT, int ST, int MINB>
__global__ __launch_bounds__(256, MINB) void attn_fwd_kernel(int B, int S, int heads, const bf16_t *__restrict__ qkv,
                                                          uint32_t qkv_bytes, bf16_t *__restrict__ o,
                                                          float *__restrict__ lse) {
  using H = Head<D>;
  constexpr int TB = tile_bytes<KT>(), NL = TileLoads<KT, 4>::N;
  static_assert(ST == 2 || ST == 3, "two or three tile stages");
  extern __shared__ __attribute__((aligned(1024))) char smem_raw[];  // ST x (K tile, V tile)
  const lds_char *smem = (const lds_char *)(smem_raw);
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(smem));

  const int nqt = (S + kRows - 1) / kRows;
  int bh, qt;
  block_item(nqt, bh, qt);
  const int b = bh / heads, h = bh % heads;
  const int A = heads * D, ld = 3 * A;
  const int lane = threadIdx.x & 63, hf = lane >> 5;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int q = qt * kRows + wid * 32 + (lane & 31);
  const bool qvalid = q < S;
  const bool active = qt * kRows + wid * 32 < S;  // wave-uniform
  const bf16_t *base = qkv + static_cast<size_t>(b) * S * ld;

  const u32x4_t rsrc = make_rsrc(qkv, qkv_bytes);
  uint32_t voff_k[NL], voff_v[NL];
  tile_voff<KT, 4>(voff_k, wid, lane, ld, false);
  tile_voff<KT, 4>(voff_v, wid, lane, ld, true);
  const uint32_t k_base = static_cast<uint32_t>((static_cast<size_t>(b) * S * ld + A + h * D) * 2);
  const uint32_t v_base = k_base + static_cast<uint32_t>(A * 2);
  const uint32_t tile_step = static_cast<uint32_t>(KT * ld * 2);
  auto issue = [&](int t) {
    const uint32_t buf = lds0 + (t % ST) * 2 * TB;
    const int rem = S - t * KT;
    tile_issue<KT, 4>(rsrc, buf, voff_k, k_base + t * tile_step, wid, lane, rem, ld, false);
    tile_issue<KT, 4>(rsrc, buf + TB, voff_v, v_base + t * tile_step, wid, lane, rem, ld, true);
  };

  bf16x8_t qf[H::KS];
  load_row_operand<D>(qf, base + static_cast<size_t>(q) * ld + h * D, qvalid, hf);

  f32x16_t acc[H::NF];
#pragma unroll
  for (int i = 0; i < H::NF; ++i) acc[i] = f32x16_t{};
  float m = -INFINITY, l = 0.f;
  const float c = kLog2e / sqrtf(static_cast<float>(D));

  const int nk = (S + KT - 1) / KT;
  for (int t = 0; t < ST - 1 && t < nk; ++t) issue(t);
  for (int t = 0; t < nk; ++t) {
    // this wave's loads of tile t have landed (those of later tiles may stay in flight)
    wait_tiles<2 * NL>(min(nk - 1 - t, ST - 2));
    // every wave's loads of tile t have landed, and every wave is done with
    // tile t - 1, whose buffer the next issue refills
    block_barrier();
    if (t + ST - 1 < nk) issue(t + ST - 1);
    const lds_char *Ks = smem + (t % ST) * 2 * TB;
    const lds_char *Vs = Ks + TB;
    const int k0 = t * KT;
    if (active) {  // waves whose queries all lie past the sequence only load and synchronise
    constexpr int NS = KT / 32;  // 32-key fragments per tile
    f32x16_t s[NS];
#pragma unroll
    for (int f = 0; f < NS; ++f) {
      s[f] = f32x16_t{};
#pragma unroll
      for (int kk = 0; kk < H::KS; ++kk) s[f] = mfma32(tile_rows(Ks, f * 32, kk, lane), qf[kk], s[f]);
    }
    ColOperands<D, KT, (D <= kPrefetchMaxD), false> vop;  // V^T operands, read under the softmax
    vop.fetch(Vs, lane);
    if (k0 + KT > S) {  // the sequence's last, partial tile: keys past it get no weight
#pragma unroll
      for (int f = 0; f < NS; ++f)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (k0 + f * 32 + (i >> 2) * 8 + hf * 4 + (i & 3) >= S) s[f][i] = -INFINITY;
    }
    // Raw logits are scaled by c > 0, so the scaled maximum is c times the
    // raw one.  The reference maximum m of a query moves only when its
    // maximum exceeds m by more than kLazyRescale (log2 units); otherwise the
    // weights, up to 2^kLazyRescale, stay relative to the old m and the
    // accumulator needs no rescaling.  O = acc / l and lse = m + log2 l hold
    // for any such m.
    float ms = -INFINITY;
#pragma unroll
    for (int f = 0; f < NS; ++f)
#pragma unroll
      for (int i = 0; i < 16; ++i) ms = fmaxf(ms, s[f][i]);
    ms = fmaxf(ms, __shfl_xor(ms, 32, kWave));
    const float mt = ms * c;
    const bool grow = mt > m + kLazyRescale;
    if (__any(grow)) {
      const float mn = grow ? mt : m;
      const float alpha = exp2_hw(m - mn);  // 0 on the first tile (m = -inf), 1 where m stays
      m = mn;
      l *= alpha;
#pragma unroll
      for (int nf = 0; nf < H::NF; ++nf) acc[nf] *= alpha;
    }
    float ls = 0.f;
#pragma unroll
    for (int f = 0; f < NS; ++f)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float pv = exp2_hw(__builtin_fmaf(s[f][i], c, -m));
        s[f][i] = pv;
        ls += pv;
      }
    l += ls;
#pragma unroll
    for (int st = 0; st < KT / 16; ++st) {
      const bf16x8_t pb = pack8(s[st >> 1], st & 1);
#pragma unroll
      for (int nf = 0; nf < H::NF; ++nf) acc[nf] = mfma32(vop.get(Vs, nf, st, lane), pb, acc[nf]);
    }
    }
  }
  block_barrier();  // every wave is done with the tile buffers, which the output slots reuse

  const float lt = l + __shfl_xor(l, 32, kWave);
  if (qvalid && hf == 0) lse[static_cast<size_t>(bh) * S + q] = (m + log2f(lt)) / kLog2e;
  const int q0 = qt * kRows + wid * 32;
  store_dmajor_lds<D>(o + (static_cast<size_t>(b) * S + q0) * A + h * D, A, acc, 1.0f / lt, lane,
                      const_cast<lds_char *>(smem) + wid * 8192, S - q0);
}

// ------------------------------------------------------------------ backward: dQ and D
//
// Per query tile: S^T = K Q^T and dP^T = V dO^T read natural-order K and V
// tiles with ds_read_b128; dQ^T += K^T dS^T reads the same K tile with the
// permuted transpose read, which matches the token order of the dS^T
// registers.  This kernel also writes D_i = dO_i . O_i for the dK/dV kernel.

template <int D, int NW, int KT, int ST, int MINB>
__global__ __launch_bounds__(NW * 64, MINB) void attn_bwd_dq_kernel(int B, int S, int heads,
                                                                    const bf16_t *__restrict__ qkv, uint32_t qkv_bytes,
                                                                    const bf16_t *__restrict__ o,
                                                                    const float *__restrict__ lse,
                                                                    const bf16_t *__restrict__ dO,
                                                                    bf16_t *__restrict__ dqkv, float *__restrict__ dvec) {
  using H = Head<D>;
  constexpr int TB = tile_bytes<KT>(), NL = TileLoads<KT, NW>::N;
  constexpr int ROWS = 32 * NW, STAGE = 2 * TB;  // K, V
  static_assert(ST == 2 || ST == 3, "two or three tile stages");
  extern __shared__ __attribute__((aligned(1024))) char smem_raw[];
  const lds_char *smem = (const lds_char *)(smem_raw);
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(smem));

  const int nqt = (S + ROWS - 1) / ROWS;
  int bh, qt;
  block_item(nqt, bh, qt);
  const int b = bh / heads, h = bh % heads;
  const int A = heads * D, ld = 3 * A;
  const int lane = threadIdx.x & 63, hf = lane >> 5;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int q = qt * ROWS + wid * 32 + (lane & 31);
  const bool qvalid = q < S;
  const bool active = qt * ROWS + wid * 32 < S;  // wave-uniform
  const bf16_t *base = qkv + static_cast<size_t>(b) * S * ld;
  const size_t orow = (static_cast<size_t>(b) * S + q) * A + h * D;

  const u32x4_t rsrc = make_rsrc(qkv, qkv_bytes);
  uint32_t voff[NL];
  tile_voff<KT, NW>(voff, wid, lane, ld, false);
  const uint32_t k_base = static_cast<uint32_t>((static_cast<size_t>(b) * S * ld + A + h * D) * 2);
  const uint32_t v_base = k_base + static_cast<uint32_t>(A * 2);
  const uint32_t tile_step = static_cast<uint32_t>(KT * ld * 2);
  auto issue = [&](int t) {
    const uint32_t buf = lds0 + (t % ST) * STAGE;
    const int rem = S - t * KT;
    tile_issue<KT, NW>(rsrc, buf, voff, k_base + t * tile_step, wid, lane, rem, ld, false);
    tile_issue<KT, NW>(rsrc, buf + TB, voff, v_base + t * tile_step, wid, lane, rem, ld, false);
  };

  bf16x8_t qf[H::KS], df[H::KS];
  load_row_operand<D>(qf, base + static_cast<size_t>(q) * ld + h * D, qvalid, hf);
  load_row_operand<D>(df, dO + orow, qvalid, hf);
  float dd = 0.f;  // D_i (this lane holds half of the d values of its query)
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
  constexpr int LOADS = 2 * NL;
  constexpr int NS = KT / 32;  // 32-key fragments per tile
  const int nk = (S + KT - 1) / KT;
  for (int t = 0; t < ST - 1 && t < nk; ++t) issue(t);
  for (int t = 0; t < nk; ++t) {
    wait_tiles<LOADS>(min(nk - 1 - t, ST - 2));  // this wave's loads of tile t
    block_barrier();  // everyone's loads of tile t landed; tile t - 1's buffer is free
    if (t + ST - 1 < nk) issue(t + ST - 1);
    const lds_char *Ks = smem + (t % ST) * STAGE, *Vs = Ks + TB;
    const int k0 = t * KT;
    if (active) {  // waves whose queries all lie past the sequence only load and synchronise
    f32x16_t sv[NS], dp[NS];
#pragma unroll
    for (int f = 0; f < NS; ++f) {
      sv[f] = f32x16_t{};
      dp[f] = f32x16_t{};
#pragma unroll
      for (int kk = 0; kk < H::KS; ++kk) {
        sv[f] = mfma32(tile_rows(Ks, f * 32, kk, lane), qf[kk], sv[f]);
        dp[f] = mfma32(tile_rows(Vs, f * 32, kk, lane), df[kk], dp[f]);
      }
    }
#pragma unroll
    for (int f = 0; f < NS; ++f)
#pragma unroll
      for (int i = 0; i < 16; ++i) sv[f][i] = exp2_hw(__builtin_fmaf(sv[f][i], c, -lse2)) * (dp[f][i] - dd);  // dS^T
    if (k0 + KT > S) {  // the sequence's last, partial tile: keys past it get no weight
      // register i of fragment f is key k0 + f*32 + 8(i/4) + 4 hf + i%4
#pragma unroll
      for (int f = 0; f < NS; ++f)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (k0 + f * 32 + (i >> 2) * 8 + hf * 4 + (i & 3) >= S) sv[f][i] = 0.f;
    }
#pragma unroll
    for (int st = 0; st < KT / 16; ++st) {
      const bf16x8_t sb = pack8(sv[st >> 1], st & 1);
#pragma unroll
      for (int nf = 0; nf < H::NF; ++nf) acc[nf] = mfma32(tile_cols_perm(Ks, nf * 32, st, lane), sb, acc[nf]);
    }
    }
  }
  block_barrier();  // the output slots reuse the tile buffers
  const int q0 = qt * ROWS + wid * 32;
  store_dmajor_lds<D>(dqkv + (static_cast<size_t>(b) * S + q0) * ld + h * D, ld, acc,
                      1.0f / sqrtf(static_cast<float>(D)), lane, const_cast<lds_char *>(smem) + wid * 8192, S - q0);
}

// ------------------------------------------------------------------ backward: dK, dV
//
// Per block of 32·NG keys, two waves share each group of 32 keys.  Wave A
// (waves 0..NG-1) computes S = Q K^T, P = exp(S - lse) and dV^T += dO^T P;
// wave B (waves NG..2NG-1) computes dP = dO V^T, dS = P ∘ (dP - D) and
// dK^T += Q^T dS.  P goes from A to B through LDS in fp32, in the MFMA
// result layout both waves hold (lane = key, registers = queries), so dS is
// exactly what one wave computing both would get.  Each wave keeps one row
// operand and one d-major accumulator, which fits two waves per SIMD.  The
// Q and dO tiles are natural-order; S and dP read them with ds_read_b128,
// the dV and dK products with the permuted transpose read.  lse and D of the
// tile's queries come in by DMA; queries past the sequence are masked out.

// LDS of one dK/dV stage: the Q and dO tiles, then lse and D of up to 64
// queries each (a 64-lane DMA; entries past the tile are never read).
template <int KT>
constexpr int dkdv_stage_bytes() {
  return 2 * tile_bytes<KT>() + 2 * 64 * 4;
}

template <int D, int NG, int KT, int MINB>
__global__ __launch_bounds__(NG * 128, MINB) void attn_bwd_dkdv_kernel(int B, int S, int heads,
                                                                       const bf16_t *__restrict__ qkv,
                                                                       uint32_t qkv_bytes,
                                                                       const float *__restrict__ lse,
                                                                       const bf16_t *__restrict__ dO,
                                                                       uint32_t do_bytes,
                                                                       const float *__restrict__ dvec,
                                                                       bf16_t *__restrict__ dqkv) {
  using H = Head<D>;
  constexpr int TB = tile_bytes<KT>(), NL = TileLoads<KT, 2 * NG>::N;
  constexpr int NW = 2 * NG, ROWS = 32 * NG, TILES = 2 * TB;  // Q, dO
  constexpr int STAGE = dkdv_stage_bytes<KT>();                // + lse, D
  constexpr int PX = 2 * STAGE;  // P hand-over: one 32 x KT fp32 slot per key group
  extern __shared__ __attribute__((aligned(1024))) char smem_raw[];
  const lds_char *smem = (const lds_char *)(smem_raw);
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(smem));

  const int nkt = (S + ROWS - 1) / ROWS;
  int bh, kt;
  block_item(nkt, bh, kt);
  const int b = bh / heads, h = bh % heads;
  const int A = heads * D, ld = 3 * A;
  const int lane = threadIdx.x & 63, hf = lane >> 5;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool role_a = wid < NG;  // wave-uniform
  const int grp = role_a ? wid : wid - NG;
  const int k0w = kt * ROWS + grp * 32;
  const bool active = k0w < S;  // wave-uniform
  const int key = k0w + (lane & 31);
  const bool kvalid = key < S;
  const bf16_t *base = qkv + static_cast<size_t>(b) * S * ld;

  const u32x4_t rq = make_rsrc(qkv, qkv_bytes), rd = make_rsrc(dO, do_bytes);
  uint32_t vq[NL], vd[NL];
  tile_voff<KT, NW>(vq, wid, lane, ld, false);
  tile_voff<KT, NW>(vd, wid, lane, A, false);
  const uint32_t q_base = static_cast<uint32_t>((static_cast<size_t>(b) * S * ld + h * D) * 2);
  const uint32_t d_base = static_cast<uint32_t>((static_cast<size_t>(b) * S * A + h * D) * 2);
  const uint32_t q_step = static_cast<uint32_t>(KT * ld * 2), d_step = static_cast<uint32_t>(KT * A * 2);
  const uint32_t vec_bytes = static_cast<uint32_t>(static_cast<size_t>(B) * heads * S * 4);
  const u32x4_t rl = make_rsrc(lse, vec_bytes), rv = make_rsrc(dvec, vec_bytes);
  auto issue = [&](int t) {
    const uint32_t buf = lds0 + (t & 1) * STAGE;
    const int rem = S - t * KT;
    tile_issue<KT, NW>(rq, buf, vq, q_base + t * q_step, wid, lane, rem, ld, false);
    tile_issue<KT, NW>(rd, buf + TB, vd, d_base + t * d_step, wid, lane, rem, A, false);
    // lse (wave 0) and D (wave 1) of 64 queries from the tile's first; entries
    // past the tile or the sequence are never used (masked out of P below)
    const uint32_t vs = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>((bh * S + t * KT) * 4));
    if (wid == 0) buffer_load_lds4(rl, __builtin_amdgcn_readfirstlane(buf + TILES), lane * 4, vs);
    if (wid == 1) buffer_load_lds4(rv, __builtin_amdgcn_readfirstlane(buf + TILES + 64 * 4), lane * 4, vs);
  };

  // K rows (wave A) or V rows (wave B) of this lane's key
  bf16x8_t rf[H::KS];
  load_row_operand<D>(rf, base + static_cast<size_t>(key) * ld + (role_a ? A : 2 * A) + h * D, kvalid, hf);

  f32x16_t acc[H::NF];  // dV^T (wave A) or dK^T (wave B)
#pragma unroll
  for (int i = 0; i < H::NF; ++i) acc[i] = f32x16_t{};
  constexpr int NS = KT / 32;  // 32-query fragments per tile
  // P hand-over slot of this key group: lane l's 16 NS values as 16-byte
  // chunks, chunk j at position j ^ pswz(l); over any 16 consecutive lanes
  // the positions hit distinct banks, so ds_write_b128 / ds_read_b128 run
  // without conflicts
  f32x4_t *pxl = reinterpret_cast<f32x4_t *>(smem_raw + PX) + grp * (8 * KT) + lane * (4 * NS);
  const int pswz = (lane >> (NS == 1 ? 2 : 1)) & (4 * NS - 1);
  const float c = kLog2e / sqrtf(static_cast<float>(D));
  const int nq = (S + KT - 1) / KT;
  issue(0);
  for (int t = 0; t < nq; ++t) {
    wait_vmcnt<0>();  // this wave's loads of tile t
    // every wave's loads of tile t have landed, and every wave is done with
    // tile t - 1: its buffer is refilled next and its P slots rewritten
    block_barrier();
    if (t + 1 < nq) issue(t + 1);
    const lds_char *Qs = smem + (t & 1) * STAGE, *Ds = Qs + TB;
    const float *Ls = reinterpret_cast<const float *>(smem_raw + (t & 1) * STAGE + TILES);
    const int q0 = t * KT;
    // S^T (wave A) or dP^T (wave B): register 4g+e of fragment f is query
    // f*32 + 8g + 4hf + e (four consecutive queries)
    const lds_char *Rs = role_a ? Qs : Ds;
    const lds_char *Cs = role_a ? Ds : Qs;
    // dO^T (wave A) or Q^T (wave B) operands of the token-contracting
    // product, read while S or dP and the P hand-over run
    ColOperands<D, KT, (D <= kPrefetchMaxD), true> cop;
    if (active) cop.fetch(Cs, lane);
    f32x16_t sv[NS];
    // waves whose keys all lie past the sequence only load and synchronise
    // (both waves of a key group agree)
    if (active) {
#pragma unroll
    for (int f = 0; f < NS; ++f) {
      sv[f] = f32x16_t{};
#pragma unroll
      for (int kk = 0; kk < H::KS; ++kk) sv[f] = mfma32(tile_rows(Rs, f * 32, kk, lane), rf[kk], sv[f]);
    }
    if (role_a) {
      // lse and D of queries past the sequence are not this sequence's: the
      // last, partial tile zeroes their weights by selection
      const bool ragged = q0 + KT > S;
#pragma unroll
      for (int f = 0; f < NS; ++f)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int qi = f * 32 + 8 * g + 4 * hf;
          const f32x4_t l4 = *reinterpret_cast<const f32x4_t *>(Ls + qi) * kLog2e;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float pv = exp2_hw(__builtin_fmaf(sv[f][4 * g + e], c, -l4[e]));
            if (ragged && q0 + qi + e >= S) pv = 0.f;
            sv[f][4 * g + e] = pv;
          }
          pxl[(f * 4 + g) ^ pswz] = f32x4_t{sv[f][4 * g], sv[f][4 * g + 1], sv[f][4 * g + 2], sv[f][4 * g + 3]};
        }
    }
    }
    lds_barrier();  // P of every group is in LDS
    if (active) {
    if (!role_a) {
      const bool ragged = q0 + KT > S;
#pragma unroll
      for (int f = 0; f < NS; ++f)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int qi = f * 32 + 8 * g + 4 * hf;
          const f32x4_t d4 = *reinterpret_cast<const f32x4_t *>(Ls + 64 + qi);
          const f32x4_t p4 = pxl[(f * 4 + g) ^ pswz];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float ds = p4[e] * (sv[f][4 * g + e] - d4[e]);  // dS^T
            if (ragged && q0 + qi + e >= S) ds = 0.f;
            sv[f][4 * g + e] = ds;
          }
        }
    }
    // dV^T += dO^T P (wave A) or dK^T += Q^T dS (wave B)
#pragma unroll
    for (int st = 0; st < KT / 16; ++st) {
      const bf16x8_t pb = pack8(sv[st >> 1], st & 1);
#pragma unroll
      for (int nf = 0; nf < H::NF; ++nf) acc[nf] = mfma32(cop.get(Cs, nf, st, lane), pb, acc[nf]);
    }
    }
  }
  block_barrier();  // the output slots reuse the tile buffers
  // wave A holds dV, wave B dK
  bf16_t *row = dqkv + (static_cast<size_t>(b) * S + k0w) * ld + h * D + (role_a ? 2 * A : A);
  store_dmajor_lds<D>(row, ld, acc, role_a ? 1.0f : 1.0f / sqrtf(static_cast<float>(D)), lane,
                      const_cast<lds_char *>(smem) + wid * 8192, S - k0w);
}

// Launch shapes.  Forward and dQ: 4 waves of 32 queries per workgroup; dK/dV:
// NG groups of 32 keys, two waves each.  KT is the token tile streamed
// through LDS, MINB the workgroups each CU must hold at once (it caps the
// registers per wave: 512 / (waves per SIMD)).
constexpr int kFwdKT = 32, kFwdStages = 2, kFwdMinBlocks = 3, kFwdSmallGrid = 256;
constexpr int kDqWaves = 4, kDqKT = 32, kDqStages = 2, kDqMinBlocks = 2;
constexpr int kDkvGroups = 2, kDkvKT = 32, kDkvMinBlocks = 3;

template <int D, int KT, int ST, int MINB>
void launch_fwd_cfg(int B, int S, int heads, const bf16_t *qkv, bf16_t *o, float *lse, hipStream_t s) {
  const int blocks = B * heads * ((S + kRows - 1) / kRows);
  const uint32_t bytes = static_cast<uint32_t>(static_cast<size_t>(B) * S * 3 * heads * D * 2);
  // ST stages of (K, V) tiles; the per-wave 8 KB output slots reuse them
  constexpr int lds = std::max(2 * ST * tile_bytes<KT>(), 4 * 8192);
  hipLaunchKernelGGL((attn_fwd_kernel<D, KT, ST, MINB>), dim3(blocks), dim3(256), lds, s, B, S, heads, qkv, bytes, o,
                     lse);
}

// A grid that leaves CUs idle runs each block's tiles back to back with no
// other block to hide their latency: there fewer, longer tiles win (64
// tokens, two blocks per CU); larger grids take 32-token tiles and three
// blocks per CU.
template <int D>
void launch_fwd_d(int B, int S, int heads, const bf16_t *qkv, bf16_t *o, float *lse, hipStream_t s) {
  const long blocks = static_cast<long>(B) * heads * ((S + kRows - 1) / kRows);
  if (blocks <= kFwdSmallGrid)
    launch_fwd_cfg<D, 64, 2, 2>(B, S, heads, qkv, o, lse, s);
  else
    launch_fwd_cfg<D, kFwdKT, kFwdStages, kFwdMinBlocks>(B, S, heads, qkv, o, lse, s);
}

template <int D>
void launch_bwd_d(int B, int S, int heads, const bf16_t *qkv, const bf16_t *o, const float *lse, const bf16_t *dO,
                  bf16_t *dqkv, float *dvec, hipStream_t s) {
  const uint32_t qkv_bytes = static_cast<uint32_t>(static_cast<size_t>(B) * S * 3 * heads * D * 2);
  const uint32_t do_bytes = static_cast<uint32_t>(static_cast<size_t>(B) * S * heads * D * 2);
  const int qblocks = B * heads * ((S + 32 * kDqWaves - 1) / (32 * kDqWaves));
  const int kblocks = B * heads * ((S + 32 * kDkvGroups - 1) / (32 * kDkvGroups));
  // dQ: kDqStages stages of (K, V) tiles, reused by the per-wave output slots.
  // dK/dV: two stages of (Q, dO, lse, D) and one 32 x KT fp32 P slot per key
  // group, or the per-wave output slots if those need more.
  constexpr int kDqLds = std::max(2 * kDqStages * tile_bytes<kDqKT>(), kDqWaves * 8192);
  constexpr int kDkvLds = std::max(2 * dkdv_stage_bytes<kDkvKT>() + kDkvGroups * 32 * kDkvKT * 4,
                                   2 * kDkvGroups * 8192);
  hipLaunchKernelGGL((attn_bwd_dq_kernel<D, kDqWaves, kDqKT, kDqStages, kDqMinBlocks>), dim3(qblocks), dim3(kDqWaves * 64),
                     kDqLds, s, B, S, heads, qkv, qkv_bytes, o, lse, dO, dqkv, dvec);
  hipLaunchKernelGGL((attn_bwd_dkdv_kernel<D, kDkvGroups, kDkvKT, kDkvMinBlocks>), dim3(kblocks),
                     dim3(kDkvGroups * 128), kDkvLds, s, B, S, heads, qkv, qkv_bytes, lse, dO, do_bytes, dvec, dqkv);
}

}  // namespace

bool launch_attn_fwd(int B, int S, int heads, int d, const bf16_t *qkv, bf16_t *o, float *lse, hipStream_t s) {
  // every tile address (up to one tile past the tensor) must stay a 32-bit buffer offset
  const uint64_t ld = 3ull * heads * d;
  if ((static_cast<uint64_t>(B) * S + kMaxKT) * ld * 2 + kDL * 2 >= (1ull << 32)) return false;
  switch (d) {
    case 64: launch_fwd_d<64>(B, S, heads, qkv, o, lse, s); return true;
    case 80: launch_fwd_d<80>(B, S, heads, qkv, o, lse, s); return true;
    case 128: launch_fwd_d<128>(B, S, heads, qkv, o, lse, s); return true;
    default: return false;
  }
}

bool launch_attn_bwd(int B, int S, int heads, int d, const bf16_t *qkv, const bf16_t *o, const float *lse,
                     const bf16_t *dO, bf16_t *dqkv, float *dvec, hipStream_t s) {
  const uint64_t ld = 3ull * heads * d;
  if ((static_cast<uint64_t>(B) * S + kMaxKT) * ld * 2 + kDL * 2 >= (1ull << 32)) return false;
  switch (d) {
    case 64: launch_bwd_d<64>(B, S, heads, qkv, o, lse, dO, dqkv, dvec, s); return true;
    case 80: launch_bwd_d<80>(B, S, heads, qkv, o, lse, dO, dqkv, dvec, s); return true;
    case 128: launch_bwd_d<128>(B, S, heads, qkv, o, lse, dO, dqkv, dvec, s); return true;
    default: return false;
  }
}

namespace {
constexpr int kMaxDevices = 64;
std::atomic<float *> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;
}  // namespace

hipError_t attn_bwd_scratch(float **ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  float *p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    // first call on this device: look the array up with the device current
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      void *addr = nullptr;
      e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
      if (e != hipSuccess) return e;
      if (!addr) return hipErrorInvalidSymbol;
      p = static_cast<float *>(addr);
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *ptr = p;
  return hipSuccess;
}

}  // namespace optimus
