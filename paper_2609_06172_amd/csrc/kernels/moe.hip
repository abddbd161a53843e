// Routed-expert (MoE) routing: router top-K and per-expert row lists.
//
// moe_route: one wave per token row.  Each lane accumulates the E router dot
// products over its 8-element slices of the row (fp32), the wave reduces them
// with a fixed butterfly, and lane 0 picks the K largest logits (a larger
// logit first, the lower expert index on equal logits) and their softmax.
// Reads the activation row once: HBM-bound, M*H*2 bytes for bf16.
//
// moe_dispatch: one 1024-thread workgroup per expert.  The routing entries
// j = K*token + slot are scanned in increasing j, 1024 at a time; a wave
// ballot gives each lane its rank among the wave's hits and a workgroup
// prefix over the 16 wave counts (LDS) places them, so every list comes out
// in increasing j, the same on every run.
#include <hip/hip_runtime.h>

#include "common.h"
#include "moe.h"

namespace auvm {

using namespace dev;

namespace {

constexpr int kMaxE = 16;

__device__ __forceinline__ void load8(const bf16_t* p, float* v) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

__device__ __forceinline__ void load8(const float* p, float* v) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

template <class T>
__global__ void __launch_bounds__(256) moe_route_kernel(const T* __restrict__ h, const T* __restrict__ wr,
                                                        int32_t* __restrict__ rte, float* __restrict__ rtw,
                                                        int64_t M, int64_t H, int E, int K) {
  const int lane = threadIdx.x & 63;
  const int64_t row = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  float acc[kMaxE];
#pragma unroll
  for (int e = 0; e < kMaxE; ++e) acc[e] = 0.f;
  const T* hr = h + row * H;
  for (int64_t c = 8 * lane; c < H; c += 8 * 64) {
    float hv[8];
    load8(hr + c, hv);
#pragma unroll
    for (int e = 0; e < kMaxE; ++e) {
      if (e < E) {
        float wv[8];
        load8(wr + e * H + c, wv);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[e] = fmaf(hv[i], wv[i], acc[e]);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < kMaxE; ++e)
    if (e < E) acc[e] = wave_sum(acc[e]);
  if (lane != 0) return;
  uint32_t taken = 0;
  int idx[kMaxE];
  float sel[kMaxE];
  for (int j = 0; j < K; ++j) {
    int best = -1;
    float bv = 0.f;
#pragma unroll
    for (int e = 0; e < kMaxE; ++e)
      if (e < E && !((taken >> e) & 1u) && (best < 0 || acc[e] > bv)) {
        best = e;
        bv = acc[e];
      }
    taken |= 1u << best;
    idx[j] = best;
    sel[j] = bv;
  }
  const float top = sel[0];
  float s = 0.f;
  for (int j = 0; j < K; ++j) {
    sel[j] = expf(sel[j] - top);
    s += sel[j];
  }
  for (int j = 0; j < K; ++j) {
    rte[row * K + j] = idx[j];
    rtw[row * K + j] = sel[j] / s;
  }
}

__global__ void __launch_bounds__(1024) moe_dispatch_kernel(const int32_t* __restrict__ rte,
                                                            int32_t* __restrict__ lists,
                                                            int32_t* __restrict__ log, int64_t M, int K,
                                                            int E, int64_t log_row) {
  __shared__ int wcount[16];
  const int e = blockIdx.x;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int32_t* out = lists + int64_t(e) * (M + 1);
  const int64_t n = M * K;
  const uint64_t below = (uint64_t(1) << lane) - 1;
  int64_t base = 0;
  for (int64_t j0 = 0; j0 < n; j0 += 1024) {
    const int64_t j = j0 + threadIdx.x;
    const bool hit = j < n && rte[j] == e;
    const uint64_t b = __ballot(hit);
    if (lane == 0) wcount[wv] = __popcll(b);
    __syncthreads();
    int off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < 16; ++w) {
      const int c = wcount[w];
      off += w < wv ? c : 0;
      tot += c;
    }
    // a token lists an expert at most once, so a list holds at most M rows;
    // the bound only guards against malformed routing
    const int64_t at = base + off + __popcll(b & below);
    if (hit && at < M) out[1 + at] = int32_t(j);
    base += tot;
    __syncthreads();   // wcount is rewritten by the next chunk
  }
  if (threadIdx.x == 0) {
    const int32_t cnt = int32_t(base < M ? base : M);
    out[0] = cnt;
    log[log_row * E + e] = cnt;
  }
}

}  // namespace

hipError_t launch_moe_route(const void* h, const void* wr, int32_t* rte, float* rtw, int64_t M, int64_t H, int E,
                            int K, bool bf16, hipStream_t s) {
  dim3 grid(unsigned((M + 3) / 4));
  if (bf16)
    hipLaunchKernelGGL(moe_route_kernel<bf16_t>, grid, dim3(256), 0, s, static_cast<const bf16_t*>(h),
                       static_cast<const bf16_t*>(wr), rte, rtw, M, H, E, K);
  else
    hipLaunchKernelGGL(moe_route_kernel<float>, grid, dim3(256), 0, s, static_cast<const float*>(h),
                       static_cast<const float*>(wr), rte, rtw, M, H, E, K);
  return hipGetLastError();
}

hipError_t launch_moe_dispatch(const int32_t* rte, int32_t* lists, int32_t* log, int64_t M, int K, int E,
                               int64_t log_row, hipStream_t s) {
  hipLaunchKernelGGL(moe_dispatch_kernel, dim3(unsigned(E)), dim3(1024), 0, s, rte, lists, log, M, K, E, log_row);
  return hipGetLastError();
}

}  // namespace auvm
