// Kernel launch entry used by the executor: one call per traced kernel.
#pragma once

#include <hip/hip_runtime_api.h>

#include <vector>

#include "core.h"

namespace auvm {

// Launch kernel `k` with operand device pointers `ptrs` (positional order)
// on stream `s`.  Shapes were validated when the kernel was added.
hipError_t launch_op(const Kernel& k, const std::vector<Tensor>& T, uint8_t* const* ptrs,
                     hipStream_t s);

// Fill `bytes` at `p` with 0xFF (NaN for f32/bf16) on stream s.
hipError_t launch_poison(uint8_t* p, uint64_t bytes, hipStream_t s);

// The static device scratch (kernels/scratch.hip): its size, and its address
// on `device` (looked up once per device, with the device made current).
uint64_t scratch_capacity();
hipError_t scratch_address(int device, void** out);

}  // namespace auvm
