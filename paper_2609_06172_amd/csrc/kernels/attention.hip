// Causal attention kernels.
//
// attn_rowwave (any head dim <= 128, f32 or bf16): one 64-lane wave per query
// row with an online softmax over 64-key tiles: each lane scores one key of
// the tile, the wave takes the tile maximum, and every lane accumulates two
// output dimensions of P*V.
// attn_decode_d128 (bf16, head dim 128, short query blocks): see below.
#include <hip/hip_runtime.h>

#include "attention.h"
#include "common.h"

namespace auvm {

using namespace dev;

namespace {

template <class T>
__global__ void __launch_bounds__(256) attn_rowwave(AttnArgs a) {
  __shared__ float qs[4][128];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t row = int64_t(blockIdx.x) * 4 + wv;  // over (b, h, i)
  const int64_t total = a.B * a.nH * a.S;
  if (row >= total) return;
  const int64_t i = row % a.S, bh = row / a.S, h = bh % a.nH, b = bh / a.nH;
  const int64_t d = a.d;
  const T* q = reinterpret_cast<const T*>(a.q) + (b * a.S + i) * a.q_rs + h * d;
  const T* kb = reinterpret_cast<const T*>(a.k) + b * a.kv_bstride + h * a.kv_hstride;
  const T* vb = reinterpret_cast<const T*>(a.v) + b * a.kv_bstride + h * a.kv_hstride;
  T* o = reinterpret_cast<T*>(a.o) + (b * a.S + i) * a.o_rs + h * d;
  const float scale = rsqrtf(float(d));
  for (int j = lane; j < d; j += 64) qs[wv][j] = ld(q, j) * scale;
  // the 64 lanes of a wave run in lockstep; the LDS row is private to the wave
  __builtin_amdgcn_wave_barrier();
  const int64_t last = a.pos0 + i;  // highest visible key
  float m = -INFINITY, l = 0.f, acc0 = 0.f, acc1 = 0.f;
  const int d0 = lane, d1 = lane + 64;
  for (int64_t j0 = 0; j0 <= last; j0 += 64) {
    const int64_t j = j0 + lane;
    float sc = -INFINITY;
    if (j <= last) {
      const T* kr = kb + j * a.kv_rs;
      float s = 0.f;
      for (int x = 0; x < d; ++x) s = fmaf(qs[wv][x], ld(kr, x), s);
      sc = s;
    }
    const float mt = wave_max(sc);
    const float mn = fmaxf(m, mt);
    const float p = j <= last ? __expf(sc - mn) : 0.f;
    const float corr = __expf(m - mn);
    l = l * corr + wave_sum(p);
    acc0 *= corr;
    acc1 *= corr;
    const int64_t nk = (last - j0 + 1) < 64 ? (last - j0 + 1) : 64;
    for (int t = 0; t < nk; ++t) {
      const float pt = __shfl(p, t, 64);
      const T* vr = vb + (j0 + t) * a.kv_rs;
      if (d0 < d) acc0 = fmaf(pt, ld(vr, d0), acc0);
      if (d1 < d) acc1 = fmaf(pt, ld(vr, d1), acc1);
    }
    m = mn;
  }
  const float inv = 1.f / l;
  if (d0 < d) st(o, d0, acc0 * inv);
  if (d1 < d) st(o, d1, acc1 * inv);
}

// Decode attention, head dim 128, bf16: one workgroup per query row.
// A key (or value) row is 256 B = 16 lanes x 16 B, so a wave loads four
// consecutive rows per instruction, fully coalesced.  Lane (grp, sub) =
// (l / 16, l % 16) holds dims 8*sub..8*sub+7; a wave takes blocks of 32 keys
// (key 32*blk + 4*u + grp for u = 0..7, eight loads of K and eight of V in
// flight), the four waves interleave blocks, each keeps an online softmax and
// the waves are merged through LDS.
constexpr int kDecU = 8;

__device__ __forceinline__ void load8(const bf16_t* p, float* f) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  u32x4 v = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(v[i] << 16);
    f[2 * i + 1] = __uint_as_float(v[i] & 0xffff0000u);
  }
}

__global__ void __launch_bounds__(256) attn_decode_d128(AttnArgs a) {
  __shared__ float sm[4], sl[4], sacc[4][128];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int grp = lane >> 4, sub = lane & 15;
  const int64_t row = blockIdx.x;
  const int64_t i = row % a.S, bh = row / a.S, h = bh % a.nH, b = bh / a.nH;
  const bf16_t* q = reinterpret_cast<const bf16_t*>(a.q) + (b * a.S + i) * a.q_rs + h * 128;
  const bf16_t* kb = reinterpret_cast<const bf16_t*>(a.k) + b * a.kv_bstride + h * a.kv_hstride + 8 * sub;
  const bf16_t* vb = reinterpret_cast<const bf16_t*>(a.v) + b * a.kv_bstride + h * a.kv_hstride + 8 * sub;
  bf16_t* o = reinterpret_cast<bf16_t*>(a.o) + (b * a.S + i) * a.o_rs + h * 128;
  float qf[8];
  load8(q + 8 * sub, qf);
  const float scale = 0.08838834764831845f;  // 1/sqrt(128)
#pragma unroll
  for (int e = 0; e < 8; ++e) qf[e] *= scale;
  const int64_t last = a.pos0 + i;
  float m = -INFINITY, l = 0.f, acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  for (int64_t j0 = int64_t(wv) * 32; j0 <= last; j0 += 4 * 32) {
    float kf[kDecU][8], vf[kDecU][8], sc[kDecU];
#pragma unroll
    for (int u = 0; u < kDecU; ++u) {
      const int64_t j = j0 + 4 * u + grp;
      if (j <= last) {
        load8(kb + j * a.kv_rs, kf[u]);
        load8(vb + j * a.kv_rs, vf[u]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) kf[u][e] = vf[u][e] = 0.f;
      }
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int u = 0; u < kDecU; ++u) {
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) s = fmaf(qf[e], kf[u][e], s);
      s += __shfl_xor(s, 8, 64);
      s += __shfl_xor(s, 4, 64);
      s += __shfl_xor(s, 2, 64);
      s += __shfl_xor(s, 1, 64);
      sc[u] = (j0 + 4 * u + grp <= last) ? s : -INFINITY;
      mloc = fmaxf(mloc, sc[u]);
    }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float mn = fmaxf(m, mloc);
    const float corr = __expf(m - mn);
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] *= corr;
#pragma unroll
    for (int u = 0; u < kDecU; ++u) {
      const float p = __expf(sc[u] - mn);
      psum += p;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = fmaf(p, vf[u][e], acc[e]);
    }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    l = l * corr + psum;
    m = mn;
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    acc[e] += __shfl_xor(acc[e], 16, 64);
    acc[e] += __shfl_xor(acc[e], 32, 64);
  }
  if (lane == 0) {
    sm[wv] = m;
    sl[wv] = l;
  }
  if (grp == 0)
#pragma unroll
    for (int e = 0; e < 8; ++e) sacc[wv][8 * sub + e] = acc[e];
  __syncthreads();
  if (threadIdx.x < 128) {
    const int dd = threadIdx.x;
    float M = sm[0];
    for (int w = 1; w < 4; ++w) M = fmaxf(M, sm[w]);
    float L = 0.f, r = 0.f;
    for (int w = 0; w < 4; ++w) {
      const float f = sm[w] == -INFINITY ? 0.f : __expf(sm[w] - M);
      L += sl[w] * f;
      r += sacc[w][dd] * f;
    }
    o[dd] = f2bf(r / L);
  }
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  const int64_t rows = a.B * a.nH * a.S;
  if (a.bf16 && a.d == 128 && a.S <= 16) {
    hipLaunchKernelGGL(attn_decode_d128, dim3(unsigned(rows)), dim3(256), 0, s, a);
    return hipGetLastError();
  }
  dim3 grid(unsigned((rows + 3) / 4));
  if (a.bf16)
    hipLaunchKernelGGL(attn_rowwave<bf16_t>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(attn_rowwave<float>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace auvm
