// GEMM entry: C[M,N] (epilogue) = A[M,K] * W[N,K]^T, fp32 accumulation.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace auvm {

struct GemmArgs {
  int64_t M, N, K;
  const uint8_t* a;   // [M,K] f32 or bf16
  const uint8_t* w;   // [N,K] same dtype as a
  const uint8_t* w2;  // second weight for the SwiGLU epilogue (else null)
  uint8_t* c;         // [M,N]: f32 or bf16 output, f32 residual for EPI_RESID
  int epi;            // dev::Epi
  bool in_bf16, out_bf16;
};

// Dispatch: bf16 with M <= 16 -> matrix-core GEMV (gemv.hip); bf16 with
// M >= 512 and K % 64 == 0 -> 256 x 256 matrix-core GEMM fed by direct LDS
// loads (gemm_big.hip); other bf16 -> 128 x 128 matrix-core GEMM
// (gemm_mfma.hip); fp32 -> LDS-tiled FMA GEMM.
hipError_t launch_gemm(const GemmArgs& g, hipStream_t s);
hipError_t launch_gemv_bf16(const GemmArgs& g, hipStream_t s);
hipError_t launch_gemm_mfma_bf16(const GemmArgs& g, hipStream_t s);
hipError_t launch_gemm_big_bf16(const GemmArgs& g, hipStream_t s);

}  // namespace auvm
