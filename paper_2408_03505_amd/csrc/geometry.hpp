// Host-side launch geometry that fixes workspace sizes: shared by the kernel
// launchers and the C-ABI size queries (plain C++, no device code).
#pragma once

#include <stddef.h>

#include <algorithm>

namespace optimus {

// ---- LayerNorm backward: 256-thread blocks, up to kLnBwdBlocks of them, each
// writing one row of fp32 column partials per gradient (dgamma, dbeta).
constexpr int kLnThreads = 256;
constexpr int kLnBwdBlocks = 256;

// Threads per row: one wave up to 2048 columns (four rows in flight per
// block), the whole block beyond.
inline int ln_bwd_tpr(int cols) { return (cols >> 3) > 256 ? 256 : 64; }

// Rows per block (a multiple of the rows in flight).
inline int ln_bwd_rows_per_block(int rows, int cols) {
  const int rg = kLnThreads / ln_bwd_tpr(cols);
  int rpb = (rows + kLnBwdBlocks - 1) / kLnBwdBlocks;
  rpb = (rpb + rg - 1) / rg * rg;
  return rpb < rg ? rg : rpb;
}

inline int ln_bwd_blocks(int rows, int cols) {
  const int rpb = ln_bwd_rows_per_block(rows, cols);
  return (rows + rpb - 1) / rpb;
}

inline size_t ln_bwd_ws_bytes(int rows, int cols) {
  return static_cast<size_t>(ln_bwd_blocks(rows, cols)) * static_cast<size_t>(cols) * 2 * sizeof(float);
}

// ---- QK-norm backward: 16-lane groups, 16 per 256-thread block, at most
// 1024 blocks, each writing 4 x head_dim fp32 partials.
constexpr int kQkGroups = 16;

inline int qk_norm_bwd_blocks(int M, int heads) {
  const long pairs = static_cast<long>(M) * heads;
  const long want = (pairs + kQkGroups - 1) / kQkGroups;
  return static_cast<int>(want < 1024 ? want : 1024);
}

inline size_t qk_norm_bwd_ws_bytes(int M, int heads, int d) {
  return static_cast<size_t>(qk_norm_bwd_blocks(M, heads)) * 4 * d * sizeof(float);
}

// ---- Attention backward: the D vector, one fp32 per (sequence, head, query).
inline size_t attn_bwd_ws_bytes(int B, int S, int heads) {
  return static_cast<size_t>(B) * heads * S * sizeof(float);
}

// ---- GEMM tile shape.  Relative work per unit of time of each tile shape on
// one CU (256x256 = 1; 0 = never chosen).  256x128 and 128x256 tiles
// measured 5-15% slower per GEMM than the shapes below on the ViT-22B
// tensor-parallel shard, where they would fill more CUs, so they stay off.
// 128x128 tiles (two workgroups per CU) count 0.9 in the forward and
// input-gradient layouts: at 0.9 the ViT-Base MLP-up forward and MLP-down
// input gradient take them and ran 11% faster (58 -> 52 and 61 -> 53 us),
// while no other product of the five workloads changed tile.  The weight
// gradients keep 0.75: at 0.9 the ViT-22B shard's MLP weight gradients would
// take them, and one of the two ran 3% slower.
constexpr double kEff256x256 = 1.0, kEff256x192 = 0.95, kEff256x128 = 0.0, kEff128x256 = 0.0;
constexpr double kEff128x128 = 0.9, kEff128x128Wgrad = 0.75;

struct TileShape {
  int bm, bn;
};

// The tile that minimises (rounds of 256 CUs) x (tile area / efficiency);
// wgrad selects the weight-gradient layout's efficiencies.
inline TileShape choose_tile(int M, int N, bool wgrad) {
  auto cost = [&](int bm, int bn, double eff) {
    if (eff <= 0.0) return 1e300;
    const long tiles = static_cast<long>((M + bm - 1) / bm) * ((N + bn - 1) / bn);
    return static_cast<double>((tiles + 255) / 256) * bm * bn / eff;
  };
  const TileShape shapes[5] = {{256, 256}, {256, 192}, {256, 128}, {128, 256}, {128, 128}};
  const double eff[5] = {kEff256x256, kEff256x192, kEff256x128, kEff128x256, wgrad ? kEff128x128Wgrad : kEff128x128};
  int best = 0;
  for (int i = 1; i < 5; ++i)
    if (cost(shapes[i].bm, shapes[i].bn, eff[i]) < cost(shapes[best].bm, shapes[best].bn, eff[best])) best = i;
  return shapes[best];
}

// ---- Split of the contraction.  A product whose output is a small grid of
// 256 x 256 tiles is split over its contraction (the tokens, for a weight
// gradient): each split writes fp32 partials and a second kernel adds them
// in split order (deterministic).  Splits run 128 x 128 tiles, as many splits
// as fill two workgroups on each of the 256 CUs, each covering at least
// kMinSplitTokens of the contraction in a whole number of 64-wide k-steps
// (the last split takes the remainder).  Same-box A/B of the split kernels
// alone (us): with 256 x 256 tiles split to fill the CUs once, the ViT-Base
// weight gradients took 60, 58, 35 and 47 (MLP-down, MLP-up, out-projection,
// QKV); with the 128 x 128 splits 53, 56, 26 and 40, the ViT-Huge
// out-projection weight gradient 39 -> 30 and the ViT-22B shard's
// out-projection input gradient 44 -> 36.  In the layer chain ViT-Base went
// from 0.665 to 0.631 ms per step; ViT-Huge and the shard were unchanged.
constexpr int kMinSplitTokens = 512, kMaxSplits = 16;

struct SplitPlan {
  int splits, k_chunk;
  TileShape tile;
};

inline SplitPlan split_128(int M, int N, int K) {
  const long tiles = static_cast<long>((M + 127) / 128) * ((N + 127) / 128);
  int S = static_cast<int>(std::min<long>(512 / tiles, std::min(K / kMinSplitTokens, kMaxSplits)));
  if (S > 1) {
    const int kc = ((K + S - 1) / S + 63) / 64 * 64;
    S = (K + kc - 1) / kc;
    if (S > 1) return {S, kc, {128, 128}};
  }
  return {1, K, {0, 0}};
}

// Weight gradient (M output rows, N output columns, K tokens): split when
// the output has at most 64 tiles of 256 x 256 (a quarter of the CUs).
// Measured per layer with the earlier 256 x 256 splits (ViT-Base / ViT-Huge /
// ViT-22B shard, four weight gradients): 351 -> 201 us, 287 -> 268 us,
// 299 -> 299 us against no split; splitting outputs of up to 128 tiles lost
// 10-20 us on the ViT-Huge MLP and shard out-projection gradients.
inline SplitPlan wgrad_split_plan(int M, int N, int K) {
  const long tiles = static_cast<long>((M + 255) / 256) * ((N + 255) / 256);
  if (tiles * 4 <= 256) {
    const SplitPlan sp = split_128(M, N, K);
    if (sp.splits > 1) return sp;
  }
  return {1, K, choose_tile(M, N, true)};
}

// Forward / input-gradient product (output [M, N], contraction K over
// k-contiguous rows, so K a multiple of 64): split when the output has at
// most 32 tiles of 256 x 256 (an eighth of the CUs).  The partials' round
// trip and the separate epilogue pay off only for such very small grids:
// with up to 128 tiles the ViT-Base and ViT-Huge forward and input-gradient
// products with 75-96 tiles ran 5-14 us slower split.
inline SplitPlan gemm_split_plan(int M, int N, int K) {
  const long tiles = static_cast<long>((M + 255) / 256) * ((N + 255) / 256);
  if (K % 64 == 0 && tiles * 8 <= 256) {
    const SplitPlan sp = split_128(M, N, K);
    if (sp.splits > 1) return sp;
  }
  return {1, K, choose_tile(M, N, false)};
}

// Whether the direct-to-LDS kernels take a product (operands A(m, k) and
// B(n, k) with leading dimensions lda, ldb; AT / BT: stored k-major):
// contiguous-k operands need whole 64-wide k-steps, and the operand extents
// that bound the buffer loads keep every offset below 2^32.  The others run
// the register-staged kernel.
inline bool lds_fits(int M, int N, int K, int lda, int ldb, bool AT, bool BT) {
  if ((!AT || !BT) && K % 64 != 0) return false;
  const unsigned long long lim = (1ull << 32) - 1;
  const unsigned long long a_bytes = static_cast<unsigned long long>(AT ? K : M) * lda * 2;
  const unsigned long long b_bytes = static_cast<unsigned long long>(BT ? K : N) * ldb * 2;
  return a_bytes + 600ull * lda * 2 <= lim && b_bytes + 600ull * ldb * 2 <= lim;
}

// Tile of the register-staged kernel: 256x128 once that grid has 512 tiles,
// else 128x128.
inline TileShape any_tile(int M, int N) {
  const long big = static_cast<long>((M + 255) / 256) * ((N + 127) / 128);
  return big >= 512 ? TileShape{256, 128} : TileShape{128, 128};
}

// Output tile and contraction splits of a product as the launchers take it
// when given a workspace of the queried size (forward: AT = BT = false;
// input gradient: BT; weight gradient: AT and BT, M output rows, N output
// columns, K tokens).
struct GemmPlan {
  TileShape tile;
  int splits;
};

inline GemmPlan gemm_plan(int M, int N, int K, int lda, int ldb, bool AT, bool BT) {
  const bool wgrad = AT && BT;
  const bool fits = lds_fits(M, N, K, lda, ldb, AT, BT);
  const SplitPlan sp = wgrad ? wgrad_split_plan(M, N, K) : gemm_split_plan(M, N, K);
  const bool split_ok = wgrad ? M % 4 == 0 && N % 4 == 0 : N % 8 == 0;
  if (sp.splits > 1 && split_ok && fits) return {sp.tile, sp.splits};
  if (fits) return {choose_tile(M, N, wgrad), 1};
  return {any_tile(M, N), 1};
}

inline size_t ws_round256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

// Workspace of a split forward or input-gradient product: the fp32 partials
// [S][M][N]; 0 when the plan does not split.
inline size_t gemm_ws_bytes(int M, int N, int K) {
  const SplitPlan sp = gemm_split_plan(M, N, K);
  return sp.splits > 1 ? ws_round256(static_cast<size_t>(sp.splits) * M * N * sizeof(float)) : 0;
}

// Workspace of a split weight gradient: the fp32 partials of dW [S][M][N]
// and of db [S][M], each 256-byte aligned; 0 when the plan does not split.
inline size_t gemm_wgrad_ws_bytes(int M, int N, int K) {
  const SplitPlan sp = wgrad_split_plan(M, N, K);
  if (sp.splits <= 1) return 0;
  return ws_round256(static_cast<size_t>(sp.splits) * M * N * sizeof(float)) +
         ws_round256(static_cast<size_t>(sp.splits) * M * sizeof(float));
}

}  // namespace optimus
