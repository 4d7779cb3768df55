// Stand-ins for the device side of the library, for a host-only build of the
// C-ABI layer (argument checks, layouts, composites, the kernel packer) under
// AddressSanitizer and UndefinedBehaviorSanitizer on a machine without a GPU.
// Every launcher accepts and does nothing; the HIP calls the C-ABI layer
// makes report success.  Never part of the product library.
#include <hip/hip_runtime_api.h>

#include "../kernels.hpp"

namespace optimus {

bool launch_ln_fwd(int, int, const bf16_t *, const bf16_t *, const bf16_t *, float, bf16_t *, float *, float *,
                   hipStream_t) {
  return true;
}
bool launch_ln_bwd(int, int, const bf16_t *, const bf16_t *, const float *, const float *, const bf16_t *,
                   const bf16_t *, bf16_t *, float *, float *, int, float *, hipStream_t) {
  return true;
}
bool launch_gemm_fwd(const GemmArgs &, Epi, void *, size_t, hipStream_t) { return true; }
bool launch_gemm_dgrad(const GemmArgs &, Epi, void *, size_t, hipStream_t) { return true; }
bool launch_gemm_wgrad(const GemmArgs &, void *, size_t, hipStream_t) { return true; }
bool launch_qk_norm_fwd(int, int, int, const bf16_t *, const bf16_t *, const bf16_t *, const bf16_t *,
                        const bf16_t *, float, bf16_t *, float *, hipStream_t) {
  return true;
}
bool launch_qk_norm_bwd(int, int, int, const bf16_t *, const bf16_t *, const float *, const bf16_t *,
                        const bf16_t *, bf16_t *, float *, float *, float *, float *, int, float *, hipStream_t) {
  return true;
}
bool launch_attn_fwd(int, int, int, int, const bf16_t *, bf16_t *, float *, hipStream_t) { return true; }
bool launch_attn_bwd(int, int, int, int, const bf16_t *, const bf16_t *, const float *, const bf16_t *, bf16_t *,
                     float *, hipStream_t) {
  return true;
}
hipError_t attn_bwd_scratch(float **ptr) {
  static float stand_in[16];
  *ptr = stand_in;
  return hipSuccess;
}
bool launch_patchify(int, int, int, int, int, int, const bf16_t *, bf16_t *, hipStream_t) { return true; }
bool launch_patch_assemble(int, int, int, int, int, const bf16_t *, const bf16_t *, const bf16_t *, bf16_t *,
                           hipStream_t) {
  return true;
}
bool launch_patch_pos_grad(int, int, int, const bf16_t *, float *, float *, int, hipStream_t) { return true; }
bool launch_patch_token_rows(int, int, int, int, const bf16_t *, bf16_t *, hipStream_t) { return true; }
bool launch_calib_mfma(int, int, float *, hipStream_t) { return true; }
bool launch_calib_copy(const void *, void *, size_t, hipStream_t) { return true; }

}  // namespace optimus

extern "C" {
hipError_t hipGetLastError(void) { return hipSuccess; }
const char *hipGetErrorString(hipError_t) { return "no error (host-only build)"; }
// Marks this build: tests that pass fake device pointers to entry points that
// would launch kernels run only against a library exporting this symbol.
int enc_host_stub_build(void) { return 1; }
}
