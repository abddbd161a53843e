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
  // Routed rows (bf16 only): list[0] = count, list[1 + i] = entry j of GEMM
  // row i, token j / topk.  Rows i >= min(count, M) are skipped.  With
  // EPI_SWIGLU row i reads A row token(i) and writes C row i; with EPI_MOE it
  // reads A row i and adds rw[j] * result into row token(i) of the fp32 C.
  const int32_t* list = nullptr;
  const float* rw = nullptr;
  int topk = 1;
  // Grouped products of one A (EPI_STORE, no list): groups > 1 computes
  // C_i = A W_i^T for i < groups with W_i = gw[i], C_i = gc[i] (w and c
  // unused).  The GEMV runs them as one grid; other routes launch once per
  // product.  Each C_i equals the ungrouped product bit for bit.
  int groups = 1;
  const uint8_t* gw[3] = {};
  uint8_t* gc[3] = {};
};

// Dispatch: bf16 with M <= 16 -> matrix-core GEMV (gemv.hip); bf16 with
// M >= 512 and K % 64 == 0 -> 256 x 256 matrix-core GEMM fed by direct LDS
// loads (gemm_big.hip); other bf16 -> 128 x 128 matrix-core GEMM
// (gemm_mfma.hip); fp32 -> LDS-tiled FMA GEMM.  With a routed-row list:
// M <= 16 -> the GEMV, else the 256 x 256 GEMM (K % 64 == 0).  Groups of up
// to three products as described above.
hipError_t launch_gemm(const GemmArgs& g, hipStream_t s);
hipError_t launch_gemv_bf16(const GemmArgs& g, hipStream_t s);
hipError_t launch_gemm_mfma_bf16(const GemmArgs& g, hipStream_t s);
hipError_t launch_gemm_big_bf16(const GemmArgs& g, hipStream_t s);

}  // namespace auvm
