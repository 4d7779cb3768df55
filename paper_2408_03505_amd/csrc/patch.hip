// Patch embedding of a ViT encoder: non-overlapping p x p patches of the
// input images become rows of a matrix (the stride-p convolution written as
// a matrix product), a GEMM with bias turns them into tokens, and the
// tokens -- after an optional class token -- get the position embedding.
//
//   patches[b*N + n, c*p*p + i*p + j] = images[b, c, py*p + i, px*p + j]
//     (n = py*gw + px; columns C*p*p .. Kp-1 are zero, Kp = C*p*p rounded
//      up to a multiple of 8)
//   x0[b*S + s] = (s == 0 and has_cls ? cls : tok[b*N + s - has_cls]) + pos[s]
#include "common.hpp"
#include "kernels.hpp"

namespace optimus {

namespace {

__global__ __launch_bounds__(256) void patchify_kernel(int B, int C, int img_h, int img_w, int p, int Kp,
                                                       const bf16_t *__restrict__ images,
                                                       bf16_t *__restrict__ patches) {
  const int gw = img_w / p, gh = img_h / p, K = C * p * p;
  const size_t total = static_cast<size_t>(B) * gh * gw * Kp;
  for (size_t t = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x; t < total;
       t += static_cast<size_t>(gridDim.x) * 256) {
    const int col = static_cast<int>(t % Kp);
    const size_t row = t / Kp;
    bf16_t v = 0;
    if (col < K) {
      const int n = static_cast<int>(row % (static_cast<size_t>(gh) * gw));
      const int b = static_cast<int>(row / (static_cast<size_t>(gh) * gw));
      const int c = col / (p * p), i = (col / p) % p, j = col % p;
      const int y = (n / gw) * p + i, x = (n % gw) * p + j;
      v = images[((static_cast<size_t>(b) * C + c) * img_h + y) * img_w + x];
    }
    patches[t] = v;
  }
}

// 8 columns per thread, fp32 add, one rounding.
__global__ __launch_bounds__(256) void assemble_kernel(int B, int N, int S, int H, int has_cls,
                                                       const bf16_t *__restrict__ tok, const bf16_t *__restrict__ cls,
                                                       const bf16_t *__restrict__ pos, bf16_t *__restrict__ x0) {
  const int CH = H / 8;
  const size_t total = static_cast<size_t>(B) * S * CH;
  for (size_t t = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x; t < total;
       t += static_cast<size_t>(gridDim.x) * 256) {
    const int ch = static_cast<int>(t % CH);
    const size_t r = t / CH;
    const int s = static_cast<int>(r % S), b = static_cast<int>(r / S);
    const u32x4_t src = (has_cls && s == 0) ? ldg16(cls + ch * 8)
                                            : ldg16(tok + (static_cast<size_t>(b) * N + s - has_cls) * H + ch * 8);
    const u32x4_t pw = ldg16(pos + static_cast<size_t>(s) * H + ch * 8);
    u32x4_t o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = pack2(lo_bf(src[e]) + lo_bf(pw[e]), hi_bf(src[e]) + hi_bf(pw[e]));
    stg16(x0 + r * H + ch * 8, o);
  }
}

// dpos[s, h] (+)= sum_b dx0[b*S + s, h] in order b = 0..B-1; dcls = dpos[0].
__global__ __launch_bounds__(256) void pos_grad_kernel(int B, int S, int H, const bf16_t *__restrict__ dx0,
                                                       float *__restrict__ dpos, float *__restrict__ dcls,
                                                       int accumulate) {
  const size_t total = static_cast<size_t>(S) * H;
  for (size_t t = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x; t < total;
       t += static_cast<size_t>(gridDim.x) * 256) {
    float s = 0.f;
    for (int b = 0; b < B; ++b) s += bf2f(dx0[static_cast<size_t>(b) * total + t]);
    dpos[t] = accumulate ? dpos[t] + s : s;
    if (dcls && t < static_cast<size_t>(H)) dcls[t] = accumulate ? dcls[t] + s : s;
  }
}

// dtok[b*N + n] = dx0[b*S + n + 1] (rows after each sequence's class token).
__global__ __launch_bounds__(256) void token_rows_kernel(int B, int N, int S, int H, const bf16_t *__restrict__ dx0,
                                                         bf16_t *__restrict__ dtok) {
  const int CH = H / 8;
  const size_t total = static_cast<size_t>(B) * N * CH;
  for (size_t t = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x; t < total;
       t += static_cast<size_t>(gridDim.x) * 256) {
    const int ch = static_cast<int>(t % CH);
    const size_t r = t / CH;
    const int n = static_cast<int>(r % N), b = static_cast<int>(r / N);
    stg16(dtok + r * H + ch * 8, ldg16(dx0 + (static_cast<size_t>(b) * S + n + 1) * H + ch * 8));
  }
}

int grid_for(size_t work) {
  const size_t blocks = (work + 255) / 256;
  return static_cast<int>(blocks < 8192 ? (blocks > 0 ? blocks : 1) : 8192);
}

}  // namespace

bool launch_patchify(int B, int C, int img_h, int img_w, int p, int Kp, const bf16_t *images, bf16_t *patches,
                     hipStream_t s) {
  const size_t total = static_cast<size_t>(B) * (img_h / p) * (img_w / p) * Kp;
  hipLaunchKernelGGL(patchify_kernel, dim3(grid_for(total)), dim3(256), 0, s, B, C, img_h, img_w, p, Kp, images,
                     patches);
  return true;
}

bool launch_patch_assemble(int B, int N, int S, int H, int has_cls, const bf16_t *tok, const bf16_t *cls,
                           const bf16_t *pos, bf16_t *x0, hipStream_t s) {
  hipLaunchKernelGGL(assemble_kernel, dim3(grid_for(static_cast<size_t>(B) * S * (H / 8))), dim3(256), 0, s, B, N,
                     S, H, has_cls, tok, cls, pos, x0);
  return true;
}

bool launch_patch_pos_grad(int B, int S, int H, const bf16_t *dx0, float *dpos, float *dcls, int accumulate,
                           hipStream_t s) {
  hipLaunchKernelGGL(pos_grad_kernel, dim3(grid_for(static_cast<size_t>(S) * H)), dim3(256), 0, s, B, S, H, dx0,
                     dpos, dcls, accumulate);
  return true;
}

bool launch_patch_token_rows(int B, int N, int S, int H, const bf16_t *dx0, bf16_t *dtok, hipStream_t s) {
  hipLaunchKernelGGL(token_rows_kernel, dim3(grid_for(static_cast<size_t>(B) * N * (H / 8))), dim3(256), 0, s, B, N,
                     S, H, dx0, dtok);
  return true;
}

}  // namespace optimus
