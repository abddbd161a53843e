// fp32 GEMM with fused epilogues (store, exact GELU, residual add, SwiGLU),
// and the GEMM dispatch.
//
// C[m,n] = sum_k A[m,k] W[n,k]: both operands are K-contiguous ("[out,in]"
// weights).  Tiles of A and W are staged through LDS as fp32 and each thread
// accumulates a TM x TN block in registers.  Used for fp32 decoders; bf16
// work goes to the matrix-core kernels.
#include <hip/hip_runtime.h>

#include "common.h"
#include "gemm.h"

namespace auvm {

using namespace dev;

namespace {

constexpr int BK = 16;

template <int BM, int BN, int TM, int TN, class TA, class TC, int EPI>
__global__ void __launch_bounds__(256) gemm_tiled(const TA* __restrict__ A, const TA* __restrict__ W,
                                                  const TA* __restrict__ W2, TC* __restrict__ C,
                                                  int64_t M, int64_t N, int64_t K) {
  constexpr int TY = BM / TM, TX = BN / TN;
  static_assert(TX * TY == 256, "256 threads per block");
  constexpr bool DUAL = EPI == EPI_SWIGLU;
  __shared__ float As[BK][BM + 1];
  __shared__ float Ws[BK][BN + 1];
  __shared__ float W2s[DUAL ? BK : 1][DUAL ? BN + 1 : 1];
  const int tid = threadIdx.x, tx = tid % TX, ty = tid / TX;
  const int64_t m0 = int64_t(blockIdx.y) * BM, n0 = int64_t(blockIdx.x) * BN;
  float acc[TM][TN], acc2[DUAL ? TM : 1][DUAL ? TN : 1];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = 0.f;
  if constexpr (DUAL) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc2[i][j] = 0.f;
  }
  for (int64_t k0 = 0; k0 < K; k0 += BK) {
    for (int e = tid; e < BM * BK; e += 256) {
      int r = e / BK, kk = e % BK;
      int64_t m = m0 + r, k = k0 + kk;
      As[kk][r] = (m < M && k < K) ? ld(A, m * K + k) : 0.f;
    }
    for (int e = tid; e < BN * BK; e += 256) {
      int r = e / BK, kk = e % BK;
      int64_t n = n0 + r, k = k0 + kk;
      bool in = n < N && k < K;
      Ws[kk][r] = in ? ld(W, n * K + k) : 0.f;
      if constexpr (DUAL) W2s[kk][r] = in ? ld(W2, n * K + k) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float av[TM], wv[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) av[i] = As[kk][ty + TY * i];
#pragma unroll
      for (int j = 0; j < TN; ++j) wv[j] = Ws[kk][tx + TX * j];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = fmaf(av[i], wv[j], acc[i][j]);
      if constexpr (DUAL) {
#pragma unroll
        for (int j = 0; j < TN; ++j) wv[j] = W2s[kk][tx + TX * j];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) acc2[i][j] = fmaf(av[i], wv[j], acc2[i][j]);
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    int64_t m = m0 + ty + TY * i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      int64_t n = n0 + tx + TX * j;
      if (n >= N) continue;
      float v = acc[i][j];
      if constexpr (EPI == EPI_GELU) v = gelu_erf(v);
      if constexpr (EPI == EPI_SWIGLU) v = silu(v) * acc2[i][j];
      if constexpr (EPI == EPI_RESID) {
        float* x = reinterpret_cast<float*>(C);
        x[m * N + n] += v;
      } else {
        st(C, m * N + n, v);
      }
    }
  }
}

template <class TA, class TC, int EPI>
hipError_t run(const GemmArgs& g, hipStream_t s) {
  const TA* A = reinterpret_cast<const TA*>(g.a);
  const TA* W = reinterpret_cast<const TA*>(g.w);
  const TA* W2 = reinterpret_cast<const TA*>(g.w2);
  TC* C = reinterpret_cast<TC*>(g.c);
  if (g.M <= 16) {
    dim3 grid(unsigned((g.N + 255) / 256), unsigned((g.M + 15) / 16));
    hipLaunchKernelGGL((gemm_tiled<16, 256, 1, 16, TA, TC, EPI>), grid, dim3(256), 0, s, A, W, W2, C,
                       g.M, g.N, g.K);
  } else {
    dim3 grid(unsigned((g.N + 63) / 64), unsigned((g.M + 63) / 64));
    hipLaunchKernelGGL((gemm_tiled<64, 64, 4, 4, TA, TC, EPI>), grid, dim3(256), 0, s, A, W, W2, C,
                       g.M, g.N, g.K);
  }
  return hipGetLastError();
}

template <class TA, class TC>
hipError_t by_epi(const GemmArgs& g, hipStream_t s) {
  switch (g.epi) {
    case EPI_STORE: return run<TA, TC, EPI_STORE>(g, s);
    case EPI_GELU: return run<TA, TC, EPI_GELU>(g, s);
    case EPI_RESID: return run<TA, float, EPI_RESID>(g, s);
    case EPI_SWIGLU: return run<TA, TC, EPI_SWIGLU>(g, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& g, hipStream_t s) {
  if (g.groups != 1) {
    if (g.groups < 1 || g.groups > 3 || g.list || g.epi != EPI_STORE) return hipErrorInvalidValue;
    if (g.in_bf16 && g.M <= 16) return launch_gemv_bf16(g, s);
    for (int i = 0; i < g.groups; ++i) {
      GemmArgs one = g;
      one.groups = 1;
      one.w = g.gw[i];
      one.c = g.gc[i];
      const hipError_t e = launch_gemm(one, s);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  if (g.list) {
    if (!g.in_bf16 || g.topk < 1) return hipErrorInvalidValue;
    return g.M <= 16 ? launch_gemv_bf16(g, s) : launch_gemm_big_bf16(g, s);
  }
  if (g.in_bf16) {
    if (g.M <= 16) return launch_gemv_bf16(g, s);
    if (g.M >= 512 && g.K % 64 == 0) return launch_gemm_big_bf16(g, s);
    return launch_gemm_mfma_bf16(g, s);
  }
  return by_epi<float, float>(g, s);
}

}  // namespace auvm
