// Training-step kernels: the backward of each forward op, the loss, and the
// optimizer.  fp32 arithmetic throughout; bf16 or fp32 storage as the
// operands say.  Every reduction runs in a fixed order, so a step gives the
// same bits on every run.
//
//  transpose      64x64 tiles through LDS (the backward GEMMs run as
//                 C = A W^T over transposed operands)
//  swiglu         F = silu(G) U and its gradients, elementwise
//  rmsnorm_bwd    one workgroup per row for dx, then per-column sums of
//                 dy x / r over all rows for the gain, sixteen row groups
//                 combined in fixed order
//  attn_bwd       causal attention, head dim 128: D = rowsum(dO o) here,
//                 then the matrix-core dK/dV and dQ passes of attention.hip
//  rope_bwd       rotation by the opposite angle, cache layout to token-major
//  xent           per row: log-sum-exp, loss, (softmax - onehot) / T
//  embed_bwd      one workgroup per 32 vocabulary rows, token order
//  adam           AdamW, elementwise
#include <hip/hip_runtime.h>

#include "common.h"
#include "attention.h"
#include "train.h"

namespace auvm {

using namespace dev;

namespace {

constexpr float kLog2e = 1.4426950408889634f;

// block-wide sum or max of 256 threads, fixed order
template <bool MAX>
__device__ __forceinline__ float block_reduce(float v, float* sh) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  v = MAX ? wave_max(v) : wave_sum(v);
  __syncthreads();
  if (lane == 0) sh[wv] = v;
  __syncthreads();
  float r = sh[0];
#pragma unroll
  for (int w = 1; w < 4; ++w) r = MAX ? fmaxf(r, sh[w]) : r + sh[w];
  return r;
}

template <class T>
__global__ void __launch_bounds__(256) transpose_kernel(const T* __restrict__ a, T* __restrict__ b, int64_t R,
                                                        int64_t C) {
  __shared__ T tile[64][65];
  const int64_t r0 = int64_t(blockIdx.y) * 64, c0 = int64_t(blockIdx.x) * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int64_t r = r0 + i, c = c0 + tx;
    if (r < R && c < C) tile[i][tx] = a[r * C + c];
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int64_t c = c0 + i, r = r0 + tx;
    if (c < C && r < R) b[c * R + r] = tile[tx][i];
  }
}

template <class T>
__global__ void __launch_bounds__(256) swiglu_act_kernel(const T* __restrict__ G, const T* __restrict__ U,
                                                         T* __restrict__ F, int64_t n) {
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256)
    st(F, i, silu(ld(G, i)) * ld(U, i));
}

template <class T>
__global__ void __launch_bounds__(256) swiglu_bwd_kernel(const T* __restrict__ G, const T* __restrict__ U,
                                                         const T* __restrict__ dF, T* __restrict__ dG,
                                                         T* __restrict__ dU, int64_t n) {
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) {
    const float g = ld(G, i), u = ld(U, i), df = ld(dF, i);
    const float sg = 1.f / (1.f + __expf(-g));
    st(dG, i, df * u * sg * (1.f + g * (1.f - sg)));
    st(dU, i, df * g * sg);
  }
}

// y = x / r * g, r = sqrt(mean(x^2) + eps):
// dx = g dy / r - x * sum(g dy x) / (H r^3)
template <class TG>
__global__ void __launch_bounds__(256) rmsnorm_bwd_rows(const float* __restrict__ x, const TG* __restrict__ g,
                                                        const float* __restrict__ dy, float* __restrict__ dx,
                                                        bf16_t* __restrict__ dxb, float* __restrict__ rstd,
                                                        int64_t H, int acc) {
  __shared__ float sh[4];
  const int64_t row = blockIdx.x;
  const float* xr = x + row * H;
  const float* dr = dy + row * H;
  float ss = 0.f, c = 0.f;
  for (int64_t j = threadIdx.x; j < H; j += 256) {
    const float xv = xr[j];
    ss = fmaf(xv, xv, ss);
    c = fmaf(ld(g, j) * dr[j], xv, c);
  }
  ss = block_reduce<false>(ss, sh);
  c = block_reduce<false>(c, sh);
  const float inv = rsqrtf(ss / float(H) + 1e-6f);
  const float k = c * inv * inv * inv / float(H);
  for (int64_t j = threadIdx.x; j < H; j += 256) {
    float v = ld(g, j) * dr[j] * inv - xr[j] * k;
    if (acc) v += dx[row * H + j];
    dx[row * H + j] = v;
    dxb[row * H + j] = f2bf(v);
  }
  if (threadIdx.x == 0) rstd[row] = inv;
}

// dg[j] = sum over rows of dy x / r: 16 columns per workgroup (H / 16
// workgroups fill the chip at model widths), sixteen row groups of 16
// threads, each reading 64-byte row segments; the groups are combined in a
// fixed order
constexpr int kGainCols = 16, kGainGroups = 16;
__global__ void __launch_bounds__(256) rmsnorm_bwd_gain(const float* __restrict__ x, const float* __restrict__ dy,
                                                        const float* __restrict__ rstd, float* __restrict__ dg,
                                                        int64_t T, int64_t H) {
  __shared__ float part[kGainGroups][kGainCols];
  const int c = threadIdx.x % kGainCols, rg = threadIdx.x / kGainCols;
  const int64_t col = int64_t(blockIdx.x) * kGainCols + c;
  float s = 0.f;
  if (col < H)
    for (int64_t r = rg; r < T; r += kGainGroups) s = fmaf(dy[r * H + col] * x[r * H + col], rstd[r], s);
  part[rg][c] = s;
  __syncthreads();
  if (rg == 0 && col < H) {
    float t = part[0][c];
#pragma unroll
    for (int g2 = 1; g2 < kGainGroups; ++g2) t += part[g2][c];
    dg[col] = t;
  }
}

// ---------------------------------------------------------------- attention backward
constexpr int kD = 128;

// D[b,h,i] = sum_d dO[i,d] o[i,d]: one wave per (token, head)
__global__ void __launch_bounds__(256) attn_bwd_rowsum(const bf16_t* __restrict__ o, const bf16_t* __restrict__ dO,
                                                       float* __restrict__ D, int64_t BS, int64_t S, int64_t nH) {
  const int lane = threadIdx.x & 63;
  const int64_t r = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);   // (b*S + i)*nH + h
  if (r >= BS * nH) return;
  const int64_t tok = r / nH, h = r % nH, b = tok / S, i = tok % S;
  const int64_t base = r * kD;
  const float s = wave_sum(bf2f(o[base + lane]) * bf2f(dO[base + lane]) +
                           bf2f(o[base + lane + 64]) * bf2f(dO[base + lane + 64]));
  if (lane == 0) D[(b * nH + h) * S + i] = s;
}

// RoPE is a rotation per pair; its transpose rotates by the opposite angle.
template <class T>
__global__ void rope_bwd_kernel(T* dq, const T* dK, const T* dV, T* dk, T* dv, int64_t S, int64_t nH, int64_t d) {
  const int64_t row = blockIdx.x / nH, h = blockIdx.x % nH;   // row = b*S + s
  const int64_t b = row / S, s = row % S;
  const int64_t half = d / 2;
  const int64_t base = row * nH * d + h * d;
  const int64_t cbase = ((b * nH + h) * S + s) * d;
  for (int64_t i = threadIdx.x; i < half; i += blockDim.x) {
    float sn, c;
    sincosf(rope_angle(s, i, d), &sn, &c);
    const float a1 = ld(dq, base + i), a2 = ld(dq, base + i + half);
    st(dq, base + i, a1 * c + a2 * sn);
    st(dq, base + i + half, a2 * c - a1 * sn);
    const float k1 = ld(dK, cbase + i), k2 = ld(dK, cbase + i + half);
    st(dk, base + i, k1 * c + k2 * sn);
    st(dk, base + i + half, k2 * c - k1 * sn);
    dv[base + i] = dV[cbase + i];
    dv[base + i + half] = dV[cbase + i + half];
  }
}

template <class TD>
__global__ void __launch_bounds__(256) xent_kernel(const float* __restrict__ logits, const int32_t* __restrict__ labels,
                                                   float* __restrict__ losses, TD* __restrict__ dlog, int64_t V,
                                                   float invT) {
  __shared__ float sh[4];
  const int64_t row = blockIdx.x;
  const float* l = logits + row * V;
  float mx = -INFINITY;
  for (int64_t j = threadIdx.x; j < V; j += 256) mx = fmaxf(mx, l[j]);
  mx = block_reduce<true>(mx, sh);
  float s = 0.f;
  for (int64_t j = threadIdx.x; j < V; j += 256) s += __builtin_amdgcn_exp2f((l[j] - mx) * kLog2e);
  s = block_reduce<false>(s, sh);
  const float lse = mx + logf(s);
  int64_t lbl = labels[row];
  lbl = lbl < 0 ? 0 : (lbl < V ? lbl : V - 1);
  if (threadIdx.x == 0) losses[row] = lse - l[lbl];
  for (int64_t j = threadIdx.x; j < V; j += 256) {
    const float pj = __builtin_amdgcn_exp2f((l[j] - lse) * kLog2e);
    st(dlog, row * V + j, (pj - (j == lbl ? 1.f : 0.f)) * invT);
  }
}

// dE rows v0 .. v0+31: each thread owns a set of columns, so the zeroing and
// the accumulation (in token order) need no synchronisation between threads
__global__ void __launch_bounds__(256) embed_bwd_kernel(const int32_t* __restrict__ ids, const float* __restrict__ dx,
                                                        float* __restrict__ dE, int64_t T, int64_t H, int64_t V) {
  __shared__ int32_t sid[256];
  const int64_t v0 = int64_t(blockIdx.x) * 32;
  const int64_t nv = V - v0 < 32 ? V - v0 : 32;
  for (int64_t r = 0; r < nv; ++r)
    for (int64_t c = threadIdx.x; c < H; c += 256) dE[(v0 + r) * H + c] = 0.f;
  for (int64_t t0 = 0; t0 < T; t0 += 256) {
    __syncthreads();
    sid[threadIdx.x] = t0 + threadIdx.x < T ? ids[t0 + threadIdx.x] : -1;
    __syncthreads();
    const int n = int(T - t0 < 256 ? T - t0 : 256);
    for (int k = 0; k < n; ++k) {
      const int64_t id = sid[k];
      if (id < v0 || id >= v0 + nv) continue;
      for (int64_t c = threadIdx.x; c < H; c += 256) dE[id * H + c] += dx[(t0 + k) * H + c];
    }
  }
}

template <class TP>
__global__ void __launch_bounds__(256) adam_kernel(const float* __restrict__ g, float* __restrict__ p32,
                                                   float* __restrict__ m, float* __restrict__ v, TP* __restrict__ p,
                                                   int64_t n, AdamArgs a) {
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) {
    const float gi = g[i];
    const float mi = a.b1 * m[i] + (1.f - a.b1) * gi;
    const float vi = a.b2 * v[i] + (1.f - a.b2) * gi * gi;
    float pi = p32[i] * a.decay;
    pi -= a.step_size * mi / (sqrtf(vi * a.inv_bc2) + a.eps);
    m[i] = mi;
    v[i] = vi;
    p32[i] = pi;
    st(p, i, pi);
  }
}

unsigned grid_for(int64_t n) {
  const int64_t g = (n + 255) / 256;
  return unsigned(g < 65536 ? g : 65536);
}

}  // namespace

hipError_t launch_transpose(const void* a, void* b, int64_t R, int64_t C, bool bf16, hipStream_t s) {
  dim3 grid(unsigned((C + 63) / 64), unsigned((R + 63) / 64));
  if (bf16)
    hipLaunchKernelGGL(transpose_kernel<bf16_t>, grid, dim3(256), 0, s, static_cast<const bf16_t*>(a),
                       static_cast<bf16_t*>(b), R, C);
  else
    hipLaunchKernelGGL(transpose_kernel<float>, grid, dim3(256), 0, s, static_cast<const float*>(a),
                       static_cast<float*>(b), R, C);
  return hipGetLastError();
}

hipError_t launch_swiglu(bool bwd, uint8_t* const* p, int64_t n, bool bf16, hipStream_t s) {
  const unsigned grid = grid_for(n);
  if (bf16) {
    if (bwd)
      hipLaunchKernelGGL(swiglu_bwd_kernel<bf16_t>, dim3(grid), dim3(256), 0, s, (const bf16_t*)p[0],
                         (const bf16_t*)p[1], (const bf16_t*)p[2], (bf16_t*)p[3], (bf16_t*)p[4], n);
    else
      hipLaunchKernelGGL(swiglu_act_kernel<bf16_t>, dim3(grid), dim3(256), 0, s, (const bf16_t*)p[0],
                         (const bf16_t*)p[1], (bf16_t*)p[2], n);
  } else {
    if (bwd)
      hipLaunchKernelGGL(swiglu_bwd_kernel<float>, dim3(grid), dim3(256), 0, s, (const float*)p[0],
                         (const float*)p[1], (const float*)p[2], (float*)p[3], (float*)p[4], n);
    else
      hipLaunchKernelGGL(swiglu_act_kernel<float>, dim3(grid), dim3(256), 0, s, (const float*)p[0],
                         (const float*)p[1], (float*)p[2], n);
  }
  return hipGetLastError();
}

hipError_t launch_rmsnorm_bwd(uint8_t* const* p, int64_t T, int64_t H, int acc, bool g_bf16, hipStream_t s) {
  const float* x = (const float*)p[0];
  const float* dy = (const float*)p[2];
  float* dx = (float*)p[3];
  float* rstd = (float*)p[6];
  if (g_bf16)
    hipLaunchKernelGGL(rmsnorm_bwd_rows<bf16_t>, dim3(unsigned(T)), dim3(256), 0, s, x, (const bf16_t*)p[1], dy, dx,
                       (bf16_t*)p[4], rstd, H, acc);
  else
    hipLaunchKernelGGL(rmsnorm_bwd_rows<float>, dim3(unsigned(T)), dim3(256), 0, s, x, (const float*)p[1], dy, dx,
                       (bf16_t*)p[4], rstd, H, acc);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(rmsnorm_bwd_gain, dim3(unsigned((H + kGainCols - 1) / kGainCols)), dim3(256), 0, s, x, dy, rstd,
                     (float*)p[5], T, H);
  return hipGetLastError();
}

hipError_t launch_attn_bwd(uint8_t* const* p, int64_t B, int64_t S, int64_t nH, hipStream_t s) {
  const int64_t rows = B * S * nH;
  hipLaunchKernelGGL(attn_bwd_rowsum, dim3(unsigned((rows + 3) / 4)), dim3(256), 0, s, (const bf16_t*)p[3],
                     (const bf16_t*)p[5], (float*)p[9], B * S, S, nH);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  AttnBwdArgs a;
  a.q = p[0];
  a.k = p[1];
  a.v = p[2];
  a.dO = p[5];
  a.lse = (const float*)p[4];
  a.D = (const float*)p[9];
  a.dq = p[6];
  a.dk = p[7];
  a.dv = p[8];
  a.B = B;
  a.S = S;
  a.nH = nH;
  a.q_rs = nH * kD;
  return launch_attention_bwd_d128(a, s);
}

hipError_t launch_rope_bwd(uint8_t* const* p, int64_t B, int64_t S, int64_t nH, int64_t d, bool bf16, hipStream_t s) {
  const int threads = d / 2 >= 64 ? 64 : int(d / 2);
  if (bf16)
    hipLaunchKernelGGL(rope_bwd_kernel<bf16_t>, dim3(unsigned(B * S * nH)), dim3(threads), 0, s, (bf16_t*)p[0],
                       (const bf16_t*)p[1], (const bf16_t*)p[2], (bf16_t*)p[3], (bf16_t*)p[4], S, nH, d);
  else
    hipLaunchKernelGGL(rope_bwd_kernel<float>, dim3(unsigned(B * S * nH)), dim3(threads), 0, s, (float*)p[0],
                       (const float*)p[1], (const float*)p[2], (float*)p[3], (float*)p[4], S, nH, d);
  return hipGetLastError();
}

hipError_t launch_xent(uint8_t* const* p, int64_t T, int64_t V, bool bf16, hipStream_t s) {
  if (bf16)
    hipLaunchKernelGGL(xent_kernel<bf16_t>, dim3(unsigned(T)), dim3(256), 0, s, (const float*)p[0],
                       (const int32_t*)p[1], (float*)p[2], (bf16_t*)p[3], V, 1.f / float(T));
  else
    hipLaunchKernelGGL(xent_kernel<float>, dim3(unsigned(T)), dim3(256), 0, s, (const float*)p[0],
                       (const int32_t*)p[1], (float*)p[2], (float*)p[3], V, 1.f / float(T));
  return hipGetLastError();
}

hipError_t launch_embed_bwd(uint8_t* const* p, int64_t T, int64_t H, int64_t V, hipStream_t s) {
  hipLaunchKernelGGL(embed_bwd_kernel, dim3(unsigned((V + 31) / 32)), dim3(256), 0, s, (const int32_t*)p[0],
                     (const float*)p[1], (float*)p[2], T, H, V);
  return hipGetLastError();
}

hipError_t launch_adam(uint8_t* const* p, int64_t n, const AdamArgs& a, bool bf16, hipStream_t s) {
  if (bf16)
    hipLaunchKernelGGL(adam_kernel<bf16_t>, dim3(grid_for(n)), dim3(256), 0, s, (const float*)p[0], (float*)p[1],
                       (float*)p[2], (float*)p[3], (bf16_t*)p[4], n, a);
  else
    hipLaunchKernelGGL(adam_kernel<float>, dim3(grid_for(n)), dim3(256), 0, s, (const float*)p[0], (float*)p[1],
                       (float*)p[2], (float*)p[3], (float*)p[4], n, a);
  return hipGetLastError();
}

}  // namespace auvm
