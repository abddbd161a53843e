// Routed-expert routing kernels (moe.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace auvm {

// rte/rtw [M,K]: the K largest router logits of each row of h [M,H] against
// wr [E,H] (ties: lower expert index) and the softmax over them.
hipError_t launch_moe_route(const void* h, const void* wr, int32_t* rte, float* rtw, int64_t M, int64_t H, int E,
                            int K, bool bf16, hipStream_t s);
// lists [E, M+1]: per expert the count, then the entries j (rte[j] == e) in
// increasing j; log[log_row*E + e] = count.
hipError_t launch_moe_dispatch(const int32_t* rte, int32_t* lists, int32_t* log, int64_t M, int K, int E,
                               int64_t log_row, hipStream_t s);

}  // namespace auvm
