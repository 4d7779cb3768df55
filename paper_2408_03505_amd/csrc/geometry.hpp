// Host-side launch geometry that fixes workspace sizes: shared by the kernel
// launchers and the C-ABI size queries (plain C++, no device code).
#pragma once

#include <stddef.h>

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

}  // namespace optimus
