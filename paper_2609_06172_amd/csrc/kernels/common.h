// Device helpers shared by the HIP kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace auvm {
namespace dev {

typedef uint16_t bf16_t;  // storage of a bfloat16 value

__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// round to nearest even; NaN stays NaN
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return bf16_t((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return bf16_t(u >> 16);
}

__device__ __forceinline__ float ld(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ld(const bf16_t* p, int64_t i) { return bf2f(p[i]); }
__device__ __forceinline__ void st(float* p, int64_t i, float v) { p[i] = v; }
__device__ __forceinline__ void st(bf16_t* p, int64_t i, float v) { p[i] = f2bf(v); }

// Exact-erf GELU, 0.5 x (1 + erf(x / sqrt 2)), with erf from Abramowitz and
// Stegun's rational approximation 7.1.26 (|error| <= 1.5e-7).  It is written
// through erfc(z), z = |x| / sqrt 2, so one branch-free expression serves
// both signs: 1 + erf(x / sqrt 2) is 2 - erfc(z) for x >= 0 and erfc(z)
// otherwise, with erfc(z) ~= t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) e^(-z^2),
// t = 1 / (1 + p z).  About a third of the instructions of the library erff,
// which matters in GEMM epilogues (128 results per lane).
__device__ __forceinline__ float gelu_erf(float x) {
  const float z = fabsf(x) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, z, 1.0f));
  const float poly =
      t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, 1.061405429f, -1.453152027f), 1.421413741f), -0.284496736f), 0.254829592f);
  const float q = poly * __builtin_amdgcn_exp2f(-(z * z) * 1.4426950408889634f);
  return 0.5f * x * (x >= 0.f ? 2.0f - q : q);
}
__device__ __forceinline__ float silu(float x) { return x / (1.0f + __expf(-x)); }

// Rotate-half RoPE angle of pair i (of d/2) at position pos, base 10000, in
// fp32: 10000^(-2i/d) = 2^(-(2i/d) log2 10000).  The angle error at position
// 4096 is ~4e-4 rad, below the bf16 storage step.  Forward and backward
// kernels share it so that they rotate by identical angles.
__device__ __forceinline__ float rope_angle(int64_t pos, int64_t i, int64_t d) {
  const float lg = 13.287712379549449f;  // log2(10000)
  return float(pos) * exp2f(-2.f * float(i) / float(d) * lg);
}

// wave64 reductions
__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// block-wide sum over blockDim.x <= 1024 threads (wave64), result to all threads
__device__ __forceinline__ float block_sum(float v, float* scratch /* >= 16 floats */) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = (blockDim.x + 63) >> 6;
  __syncthreads();
  if (lane == 0) scratch[w] = v;
  __syncthreads();
  float r = 0.f;
  for (int i = 0; i < nw; ++i) r += scratch[i];
  return r;
}

// EPI_MOE: weighted scatter-add of routed rows into an fp32 residual (GEMMs
// driven by a routed-row list only).
enum Epi { EPI_STORE = 0, EPI_GELU = 1, EPI_RESID = 2, EPI_SWIGLU = 3, EPI_MOE = 4 };

}  // namespace dev
}  // namespace auvm
