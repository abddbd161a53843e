// Training-step kernels (train.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace auvm {

// AdamW constants of one step, precomputed on the host: decay = 1 - lr*wd,
// step_size = lr / (1 - b1^t), inv_bc2 = 1 / (1 - b2^t).
struct AdamArgs {
  float b1, b2, eps, decay, step_size, inv_bc2;
};

hipError_t launch_transpose(const void* a, void* b, int64_t R, int64_t C, bool bf16, hipStream_t s);
// operands as the SWIGLU_ACT / SWIGLU_BWD ops list them
hipError_t launch_swiglu(bool bwd, uint8_t* const* p, int64_t n, bool bf16, hipStream_t s);
hipError_t launch_rmsnorm_bwd(uint8_t* const* p, int64_t T, int64_t H, int acc, bool g_bf16, hipStream_t s);
hipError_t launch_attn_bwd(uint8_t* const* p, int64_t B, int64_t S, int64_t nH, hipStream_t s);
hipError_t launch_rope_bwd(uint8_t* const* p, int64_t B, int64_t S, int64_t nH, int64_t d, bool bf16, hipStream_t s);
hipError_t launch_xent(uint8_t* const* p, int64_t T, int64_t V, bool bf16, hipStream_t s);
hipError_t launch_embed_bwd(uint8_t* const* p, int64_t T, int64_t H, int64_t V, hipStream_t s);
hipError_t launch_adam(uint8_t* const* p, int64_t n, const AdamArgs& a, bool bf16, hipStream_t s);

}  // namespace auvm
