// Causal attention kernels.
//
// attn_rowwave (any head dim <= 128, f32 or bf16): one 64-lane wave per query
// row with an online softmax over 64-key tiles: each lane scores one key of
// the tile, the wave takes the tile maximum, and every lane accumulates two
// output dimensions of P*V.
// attn_decode_d128 (bf16, head dim 128, short query blocks) and
// attn_prefill_d128 (bf16, head dim 128, matrix cores): see below.
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

// Prefill attention, head dim 128, bf16, on matrix cores (flash-style).
// One workgroup per (b, h, block of 64 queries); wave w owns queries
// 16w..16w+15 with its Q fragments in registers.  For each block of 64 keys:
//   K is staged in LDS row-major and V transposed (dims x keys), so every
//   MFMA operand is one 16-byte LDS read;
//   S = Q K^T: 4 key tiles x 4 dim steps of v_mfma_f32_16x16x32_bf16;
//   online softmax on the accumulators (a lane holds 4 query rows);
//   P goes through a per-wave LDS tile to become the A operand of
//   O += P V: 2 key steps x 8 dim tiles of the same MFMA.
// Blocks past the diagonal are skipped; only diagonal blocks are masked.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));

constexpr int FQ = 64, FK = 64, FD = 128;
constexpr int KP = FD + 8;   // K tile pitch (elements)
constexpr int VP = FK + 8;   // transposed V tile pitch
constexpr int PP = FK + 8;   // P tile pitch

__global__ void __launch_bounds__(256) attn_prefill_d128(AttnArgs a, int64_t nqb) {
  __shared__ __align__(16) bf16_t Ks[FK * KP];
  __shared__ __align__(16) bf16_t Vt[FD * VP];
  __shared__ __align__(16) bf16_t Ps[4][16 * PP];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  // heaviest query blocks first
  const int64_t wg = blockIdx.x;
  const int64_t qb = nqb - 1 - wg % nqb, bh = wg / nqb;
  const int64_t h = bh % a.nH, b = bh / a.nH;
  const int64_t q0 = qb * FQ;
  const bf16_t* Q = reinterpret_cast<const bf16_t*>(a.q) + (b * a.S) * a.q_rs + h * FD;
  const bf16_t* Kg = reinterpret_cast<const bf16_t*>(a.k) + b * a.kv_bstride + h * a.kv_hstride;
  const bf16_t* Vg = reinterpret_cast<const bf16_t*>(a.v) + b * a.kv_bstride + h * a.kv_hstride;
  bf16_t* O = reinterpret_cast<bf16_t*>(a.o) + (b * a.S) * a.o_rs + h * FD;

  // this wave's query rows: q0 + 16*wv + r; Q fragment for dim step c: dims 32c + 8g .. +8
  const int64_t qr = q0 + 16 * wv + lr;
  bf16x8 qf[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    if (qr < a.S)
      qf[c] = *reinterpret_cast<const bf16x8*>(Q + qr * a.q_rs + 32 * c + 8 * lg);
    else
      qf[c] = bf16x8{};
  }
  const float scale = 0.08838834764831845f;  // 1/sqrt(128)
  f32x4 o[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m[4], l[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    m[i] = -INFINITY;
    l[i] = 0.f;
  }
  // queries of this workgroup see keys 0 .. pos0 + min(q0 + 63, S - 1)
  const int64_t qlast = (q0 + FQ - 1 < a.S ? q0 + FQ - 1 : a.S - 1);
  const int64_t klast = a.pos0 + qlast;
  // staging assignment: thread t moves keys 4*(t%16)..+3, dims 8*(t/16)..+7
  const int sk = 4 * (tid & 15), sd = 8 * (tid >> 4);
  for (int64_t k0 = 0; k0 <= klast; k0 += FK) {
    __syncthreads();  // previous block's tiles are no longer read
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t key = k0 + sk + j;
      u32x4v kv = u32x4v{0u, 0u, 0u, 0u}, vv = u32x4v{0u, 0u, 0u, 0u};
      if (key <= klast) {
        kv = *reinterpret_cast<const u32x4v*>(Kg + key * a.kv_rs + sd);
        vv = *reinterpret_cast<const u32x4v*>(Vg + key * a.kv_rs + sd);
      }
      *reinterpret_cast<u32x4v*>(Ks + (sk + j) * KP + sd) = kv;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        Vt[(sd + 2 * e) * VP + sk + j] = bf16_t(vv[e] & 0xffffu);
        Vt[(sd + 2 * e + 1) * VP + sk + j] = bf16_t(vv[e] >> 16);
      }
    }
    __syncthreads();
    // S = Q K^T for this wave's 16 queries x 64 keys
    f32x4 sacc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      sacc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const bf16x8 kb = *reinterpret_cast<const bf16x8*>(Ks + (16 * t + lr) * KP + 32 * c + 8 * lg);
        sacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[c], kb, sacc[t], 0, 0, 0);
      }
    }
    // element i of a lane: query row 16*wv + 4*lg + i, key k0 + 16*t + lr
    const bool diag = k0 + FK - 1 > a.pos0 + q0 + 16 * wv;
    float rmax[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t qpos = a.pos0 + q0 + 16 * wv + 4 * lg + i;
      float mx = -INFINITY;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        float v = sacc[t][i] * scale;
        if (diag && k0 + 16 * t + lr > qpos) v = -INFINITY;
        sacc[t][i] = v;
        mx = fmaxf(mx, v);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 1, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 2, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 4, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 8, 64));
      rmax[i] = mx;
    }
    bf16_t* ps = Ps[wv];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float mn = fmaxf(m[i], rmax[i]);
      // rows with no visible key yet keep m = -inf and contribute nothing
      const float corr = mn == -INFINITY ? 1.f : __expf(m[i] - mn);
      float sum = 0.f;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float p = mn == -INFINITY ? 0.f : __expf(sacc[t][i] - mn);
        sum += p;
        ps[(4 * lg + i) * PP + 16 * t + lr] = f2bf(p);
      }
      sum += __shfl_xor(sum, 1, 64);
      sum += __shfl_xor(sum, 2, 64);
      sum += __shfl_xor(sum, 4, 64);
      sum += __shfl_xor(sum, 8, 64);
      l[i] = l[i] * corr + sum;
      m[i] = mn;
#pragma unroll
      for (int t = 0; t < 8; ++t) o[t][i] *= corr;
    }
    // the P tile is private to this wave; its writes precede these reads
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const bf16x8 pa = *reinterpret_cast<const bf16x8*>(ps + lr * PP + 32 * c + 8 * lg);
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const bf16x8 vb = *reinterpret_cast<const bf16x8*>(Vt + (16 * t + lr) * VP + 32 * c + 8 * lg);
        o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, vb, o[t], 0, 0, 0);
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t q = q0 + 16 * wv + 4 * lg + i;
    if (q >= a.S) continue;
    const float inv = 1.f / l[i];
#pragma unroll
    for (int t = 0; t < 8; ++t) O[q * a.o_rs + 16 * t + lr] = f2bf(o[t][i] * inv);
  }
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  const int64_t rows = a.B * a.nH * a.S;
  if (a.bf16 && a.d == 128 && a.S <= 16) {
    hipLaunchKernelGGL(attn_decode_d128, dim3(unsigned(rows)), dim3(256), 0, s, a);
    return hipGetLastError();
  }
  if (a.bf16 && a.d == 128) {
    const int64_t nqb = (a.S + FQ - 1) / FQ;
    hipLaunchKernelGGL(attn_prefill_d128, dim3(unsigned(a.B * a.nH * nqb)), dim3(256), 0, s, a, nqb);
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
