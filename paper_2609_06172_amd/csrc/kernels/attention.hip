// Causal attention, one 64-lane wave per query row with an online softmax
// over 64-key tiles: each lane scores one key of the tile, the wave takes the
// tile maximum, and every lane accumulates two output dimensions of P*V.
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

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  const int64_t rows = a.B * a.nH * a.S;
  dim3 grid(unsigned((rows + 3) / 4));
  if (a.bf16)
    hipLaunchKernelGGL(attn_rowwave<bf16_t>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(attn_rowwave<float>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace auvm
