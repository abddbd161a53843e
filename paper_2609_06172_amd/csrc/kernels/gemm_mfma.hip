// Prefill GEMM on bf16 matrix cores: C[M,N] (epilogue) = A[M,K] W[N,K]^T.
//
// Workgroup tile 128 x 128, K step 64, four waves in a 2 x 2 grid each owning
// a 64 x 64 block = 2 x 2 tiles of v_mfma_f32_32x32x16_bf16.  A and W tiles are
// staged through LDS (rows padded by 16 bytes so the 32 row reads of one
// ds_read_b128 spread over the banks) with two buffers: the next K step is
// loaded into registers while the current one feeds the matrix cores.
// Tiles are ordered so that the workgroups resident on one XCD (dispatch is
// round-robin over the 8 XCDs) share A row-blocks and W column-blocks in L2.
#include <hip/hip_runtime.h>

#include "common.h"
#include "gemm.h"

namespace auvm {

using namespace dev;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128, BN = 128, BK = 64, LDK = BK + 8;  // LDS row pitch in elements
constexpr int kXcd = 8;
constexpr int kGroupM = 8;

struct Frag {
  u32x4 v[4];  // 4 x 16 B per thread per 128 x 64 tile
};

__device__ __forceinline__ void load_tile(Frag& f, const bf16_t* __restrict__ P, int64_t rows, int64_t K,
                                          int64_t r0, int64_t k0, int tid) {
  const int kc = (tid & 7) * 8;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t r = r0 + (tid >> 3) + 32 * i, k = k0 + kc;
    if (r < rows && k < K)
      f.v[i] = *reinterpret_cast<const u32x4*>(P + r * K + k);
    else
      f.v[i] = u32x4{0u, 0u, 0u, 0u};
  }
}

__device__ __forceinline__ void store_tile(const Frag& f, bf16_t* lds, int tid) {
  const int kc = (tid & 7) * 8;
#pragma unroll
  for (int i = 0; i < 4; ++i) *reinterpret_cast<u32x4*>(lds + ((tid >> 3) + 32 * i) * LDK + kc) = f.v[i];
}

template <int EPI, class TC>
__global__ void __launch_bounds__(256) gemm_mfma(const bf16_t* __restrict__ A, const bf16_t* __restrict__ W,
                                                 const bf16_t* __restrict__ W2, TC* __restrict__ C,
                                                 int64_t M, int64_t N, int64_t K, int tilesN) {
  constexpr bool DUAL = EPI == EPI_SWIGLU;
  extern __shared__ __align__(16) bf16_t smem[];
  bf16_t* As = smem;                                   // [2][BM][LDK]
  bf16_t* Ws = As + 2 * BM * LDK;                      // [2][BN][LDK]
  bf16_t* W2s = Ws + 2 * BN * LDK;                     // [2][BN][LDK] (DUAL only)
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int wm = wv >> 1, wn = wv & 1;

  // Tile order.  Dispatch sends workgroup i to XCD i % 8, so the remap gives
  // each XCD a contiguous run of the tile sequence; the sequence walks groups
  // of kGroupM row-blocks column by column, so the ~64 tiles resident on one
  // XCD span about 8 row-blocks x 8 column-blocks and share both A and W in
  // that XCD's L2.
  const int nwg = gridDim.x, per = nwg / kXcd;
  int id = blockIdx.x;
  if (per > 0 && id < per * kXcd) id = (id % kXcd) * per + id / kXcd;
  const int tilesM = nwg / tilesN;
  const int gsize = kGroupM * tilesN, grp = id / gsize, first = grp * kGroupM;
  const int gm = (tilesM - first) < kGroupM ? (tilesM - first) : kGroupM;
  const int in = id - grp * gsize;
  const int64_t m0 = int64_t(first + in % gm) * BM, n0 = int64_t(in / gm) * BN;

  f32x16 acc[2][2], acc2[DUAL ? 2 : 1][DUAL ? 2 : 1];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
  if constexpr (DUAL) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc2[i][j] = f32x16{};
  }

  const int64_t nk = (K + BK - 1) / BK;
  Frag fa, fw, fw2;
  load_tile(fa, A, M, K, m0, 0, tid);
  load_tile(fw, W, N, K, n0, 0, tid);
  if constexpr (DUAL) load_tile(fw2, W2, N, K, n0, 0, tid);
  store_tile(fa, As, tid);
  store_tile(fw, Ws, tid);
  if constexpr (DUAL) store_tile(fw2, W2s, tid);
  __syncthreads();

  // lane's operand rows inside a 32-row MFMA tile and its 8-wide K slice
  const int lr = lane & 31, lk = (lane >> 5) * 8;
  for (int64_t kt = 0; kt < nk; ++kt) {
    const int buf = int(kt & 1);
    if (kt + 1 < nk) {
      load_tile(fa, A, M, K, m0, (kt + 1) * BK, tid);
      load_tile(fw, W, N, K, n0, (kt + 1) * BK, tid);
      if constexpr (DUAL) load_tile(fw2, W2, N, K, n0, (kt + 1) * BK, tid);
    }
    const bf16_t* as = As + buf * BM * LDK;
    const bf16_t* ws = Ws + buf * BN * LDK;
    const bf16_t* w2s = W2s + buf * BN * LDK;
#pragma unroll
    for (int ks = 0; ks < BK; ks += 16) {
      bf16x8 a[2], b[2], b2[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[i] = *reinterpret_cast<const bf16x8*>(as + (wm * 64 + i * 32 + lr) * LDK + ks + lk);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        b[j] = *reinterpret_cast<const bf16x8*>(ws + (wn * 64 + j * 32 + lr) * LDK + ks + lk);
        if constexpr (DUAL) b2[j] = *reinterpret_cast<const bf16x8*>(w2s + (wn * 64 + j * 32 + lr) * LDK + ks + lk);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
          if constexpr (DUAL) acc2[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b2[j], acc2[i][j], 0, 0, 0);
        }
    }
    if (kt + 1 < nk) {
      store_tile(fa, As + (buf ^ 1) * BM * LDK, tid);
      store_tile(fw, Ws + (buf ^ 1) * BN * LDK, tid);
      if constexpr (DUAL) store_tile(fw2, W2s + (buf ^ 1) * BN * LDK, tid);
    }
    __syncthreads();
  }

  // accumulator layout: element e of lane l is row 8*(e/4) + 4*(l/32) + e%4, column l%32
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t col = n0 + wn * 64 + j * 32 + (lane & 31);
      if (col >= N) continue;
      const int64_t r0 = m0 + wm * 64 + i * 32;   // first row of the 32-row tile
      if constexpr (EPI == EPI_RESID) {
        // every residual load of a full tile before its stores: one wait for
        // memory per tile rather than one per element
        if (r0 + 32 <= M) {
          float* x = reinterpret_cast<float*>(C) + (r0 + 4 * (lane >> 5)) * N + col;
          float xv[16];
#pragma unroll
          for (int e = 0; e < 16; ++e) xv[e] = x[(8 * (e >> 2) + (e & 3)) * N];
#pragma unroll
          for (int e = 0; e < 16; ++e) x[(8 * (e >> 2) + (e & 3)) * N] = xv[e] + acc[i][j][e];
          continue;
        }
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int64_t row = r0 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (row >= M) continue;
        float v = acc[i][j][e];
        if constexpr (EPI == EPI_GELU) v = gelu_erf(v);
        if constexpr (EPI == EPI_SWIGLU) v = silu(v) * acc2[i][j][e];
        if constexpr (EPI == EPI_RESID) {
          float* x = reinterpret_cast<float*>(C);
          x[row * N + col] += v;
        } else {
          st(C, row * N + col, v);
        }
      }
    }
}

template <int EPI, class TC>
hipError_t go(const GemmArgs& g, hipStream_t s) {
  const int tilesM = int((g.M + BM - 1) / BM), tilesN = int((g.N + BN - 1) / BN);
  const size_t lds = size_t(2) * (BM + BN + (EPI == EPI_SWIGLU ? BN : 0)) * LDK * sizeof(bf16_t);
  hipLaunchKernelGGL((gemm_mfma<EPI, TC>), dim3(unsigned(tilesM * tilesN)), dim3(256), lds, s,
                     reinterpret_cast<const bf16_t*>(g.a), reinterpret_cast<const bf16_t*>(g.w),
                     reinterpret_cast<const bf16_t*>(g.w2), reinterpret_cast<TC*>(g.c), g.M, g.N, g.K,
                     tilesN);
  return hipGetLastError();
}

template <class TC>
hipError_t by_epi(const GemmArgs& g, hipStream_t s) {
  switch (g.epi) {
    case EPI_STORE: return go<EPI_STORE, TC>(g, s);
    case EPI_GELU: return go<EPI_GELU, TC>(g, s);
    case EPI_RESID: return go<EPI_RESID, float>(g, s);
    case EPI_SWIGLU: return go<EPI_SWIGLU, TC>(g, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

// bf16 operands, K % 32 == 0 (checked when the kernel was added).
hipError_t launch_gemm_mfma_bf16(const GemmArgs& g, hipStream_t s) {
  return g.out_bf16 ? by_epi<bf16_t>(g, s) : by_epi<float>(g, s);
}

}  // namespace auvm
