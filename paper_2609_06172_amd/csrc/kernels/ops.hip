// Memory-bound and small kernels: touch, embedding gather, LayerNorm,
// RMSNorm, RoPE + KV-cache append, argmax, and the op dispatch.
#include <hip/hip_runtime.h>

#include <cmath>

#include "../kernels.h"
#include "common.h"
#include "gemm.h"
#include "moe.h"
#include "train.h"
#include "attention.h"

namespace auvm {

using namespace dev;

namespace {

// ---------------------------------------------------------------- touch
struct TouchArgs {
  uint32_t* data[7];
  uint64_t words[7];
  uint32_t mode[7];
  int n;
  uint32_t* log;
  int64_t slot;
};

// One block per data operand: log the min and max word read, then fill
// written operands with slot+1 (the version this kernel produces).
__global__ void __launch_bounds__(256) touch_kernel(TouchArgs a) {
  __shared__ uint32_t smin[256], smax[256];
  const int i = blockIdx.x;
  if (i >= a.n) return;
  uint32_t* p = a.data[i];
  const uint64_t n = a.words[i];
  const int tid = threadIdx.x;
  if (a.mode[i] & 1u) {
    uint32_t mn = 0xffffffffu, mx = 0u;
    for (uint64_t w = tid; w < n; w += blockDim.x) {
      uint32_t v = p[w];
      mn = min(mn, v);
      mx = max(mx, v);
    }
    smin[tid] = mn;
    smax[tid] = mx;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
      if (tid < s) {
        smin[tid] = min(smin[tid], smin[tid + s]);
        smax[tid] = max(smax[tid], smax[tid + s]);
      }
      __syncthreads();
    }
    if (tid == 0) {
      a.log[16 * a.slot + 2 * (i + 1)] = smin[0];
      a.log[16 * a.slot + 2 * (i + 1) + 1] = smax[0];
    }
    __syncthreads();
  }
  if (a.mode[i] & 2u)
    for (uint64_t w = tid; w < n; w += blockDim.x) p[w] = uint32_t(a.slot + 1);
}

// ---------------------------------------------------------------- embedding
template <class TE>
__global__ void __launch_bounds__(256) embed_kernel(const int32_t* ids, const TE* E, float* x,
                                                    int64_t H, int64_t V) {
  const int64_t t = blockIdx.x;
  int64_t id = ids[t];
  id = id < 0 ? 0 : (id >= V ? V - 1 : id);
  const TE* row = E + id * H;
  for (int64_t j = threadIdx.x; j < H; j += blockDim.x) x[t * H + j] = ld(row, j);
}

// ---------------------------------------------------------------- norms
// Output row i normalises input row i*stride + offset (fp32 statistics).
template <class TO, bool LN>
__global__ void __launch_bounds__(256) norm_kernel(const float* x, const TO* g, const TO* b, TO* h,
                                                   int64_t H, int64_t stride, int64_t offset,
                                                   float eps) {
  __shared__ float red[16];
  const int64_t r = blockIdx.x;
  const float* xr = x + (r * stride + offset) * H;
  float s = 0.f;
  for (int64_t j = threadIdx.x; j < H; j += blockDim.x) s += LN ? xr[j] : xr[j] * xr[j];
  s = block_sum(s, red);
  float mean = LN ? s / float(H) : 0.f;
  float var;
  if (LN) {
    float q = 0.f;
    for (int64_t j = threadIdx.x; j < H; j += blockDim.x) {
      float d = xr[j] - mean;
      q += d * d;
    }
    var = block_sum(q, red) / float(H);
  } else {
    var = s / float(H);
  }
  const float rs = rsqrtf(var + eps);
  for (int64_t j = threadIdx.x; j < H; j += blockDim.x) {
    float y = (xr[j] - mean) * rs * ld(g, j);
    if (LN) y += ld(b, j);
    st(h, r * H + j, y);
  }
}

// Four consecutive elements (index a multiple of 4) in one load or store.
__device__ __forceinline__ void ld4(const float* p, int64_t i, float* o) {
  const float4 v = *reinterpret_cast<const float4*>(p + i);
  o[0] = v.x; o[1] = v.y; o[2] = v.z; o[3] = v.w;
}
__device__ __forceinline__ void ld4(const bf16_t* p, int64_t i, float* o) {
  const uint2 v = *reinterpret_cast<const uint2*>(p + i);
  o[0] = bf2f(bf16_t(v.x & 0xffffu)); o[1] = bf2f(bf16_t(v.x >> 16));
  o[2] = bf2f(bf16_t(v.y & 0xffffu)); o[3] = bf2f(bf16_t(v.y >> 16));
}
__device__ __forceinline__ void st4(float* p, int64_t i, const float* y) {
  *reinterpret_cast<float4*>(p + i) = float4{y[0], y[1], y[2], y[3]};
}
__device__ __forceinline__ void st4(bf16_t* p, int64_t i, const float* y) {
  const uint2 v = {uint32_t(f2bf(y[0])) | (uint32_t(f2bf(y[1])) << 16), uint32_t(f2bf(y[2])) | (uint32_t(f2bf(y[3])) << 16)};
  *reinterpret_cast<uint2*>(p + i) = v;
}

// Row in registers: H % 4 == 0 and H <= 4 * 256 * NV; float4 loads, one read;
// gains, biases and outputs four elements at a time.
template <class TO, bool LN, int NV>
__global__ void __launch_bounds__(256) norm_vec_kernel(const float* x, const TO* g, const TO* b, TO* h,
                                                       int64_t H, int64_t stride, int64_t offset,
                                                       float eps) {
  __shared__ float red[16];
  const int64_t r = blockIdx.x;
  const float4* xr = reinterpret_cast<const float4*>(x + (r * stride + offset) * H);
  const int n4 = int(H / 4);
  float4 v[NV];
  float s = 0.f;
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int j = threadIdx.x + 256 * u;
    v[u] = j < n4 ? xr[j] : float4{0.f, 0.f, 0.f, 0.f};
    s += LN ? (v[u].x + v[u].y + v[u].z + v[u].w)
            : (v[u].x * v[u].x + v[u].y * v[u].y + v[u].z * v[u].z + v[u].w * v[u].w);
  }
  s = block_sum(s, red);
  float mean = 0.f, var;
  if (LN) {
    mean = s / float(H);
    float q = 0.f;
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      if (threadIdx.x + 256 * u < n4) {
        const float a0 = v[u].x - mean, a1 = v[u].y - mean, a2 = v[u].z - mean, a3 = v[u].w - mean;
        q += a0 * a0 + a1 * a1 + a2 * a2 + a3 * a3;
      }
    }
    var = block_sum(q, red) / float(H);
  } else {
    var = s / float(H);
  }
  const float rs = rsqrtf(var + eps);
#pragma unroll
  for (int u = 0; u < NV; ++u) {
    const int j = threadIdx.x + 256 * u;
    if (j >= n4) continue;
    const float e[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
    const int64_t col = 4 * int64_t(j);
    float gv[4], bv[4] = {0.f, 0.f, 0.f, 0.f}, y[4];
    ld4(g, col, gv);
    if (LN) ld4(b, col, bv);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      y[c] = (e[c] - mean) * rs * gv[c];
      if (LN) y[c] += bv[c];
    }
    st4(h, r * H + col, y);
  }
}

template <class TO, bool LN>
void launch_norm(const uint8_t* x, const uint8_t* g, const uint8_t* b, uint8_t* h, const int64_t* sh,
                 float eps, hipStream_t s) {
  const int64_t T = sh[0], H = sh[1];
  const float* xf = reinterpret_cast<const float*>(x);
  const TO *gp = reinterpret_cast<const TO*>(g), *bp = reinterpret_cast<const TO*>(b);
  TO* hp = reinterpret_cast<TO*>(h);
  if (H % 4 == 0 && H <= 4 * 256 * 2)
    hipLaunchKernelGGL((norm_vec_kernel<TO, LN, 2>), dim3(unsigned(T)), dim3(256), 0, s, xf, gp, bp, hp, H,
                       sh[2], sh[3], eps);
  else if (H % 4 == 0 && H <= 4 * 256 * 8)
    hipLaunchKernelGGL((norm_vec_kernel<TO, LN, 8>), dim3(unsigned(T)), dim3(256), 0, s, xf, gp, bp, hp, H,
                       sh[2], sh[3], eps);
  else
    hipLaunchKernelGGL((norm_kernel<TO, LN>), dim3(unsigned(T)), dim3(256), 0, s, xf, gp, bp, hp, H, sh[2],
                       sh[3], eps);
}

// ---------------------------------------------------------------- RoPE + KV append
// One block per (token row, head): rotate pairs (i, i+d/2) of q and k by
// pos * 10000^(-2i/d); write rotated k and v into the caches at pos.
template <class T>
__global__ void rope_kv_kernel(T* q, const T* k, const T* v, T* Kc, T* Vc, int64_t S, int64_t nH,
                               int64_t d, int64_t Lmax, int64_t pos0) {
  const int64_t row = blockIdx.x / nH, h = blockIdx.x % nH;  // row = b*S + s
  const int64_t b = row / S, s = row % S, pos = pos0 + s;
  const int64_t half = d / 2;
  const int64_t base = row * nH * d + h * d;
  const int64_t cbase = ((b * nH + h) * Lmax + pos) * d;
  for (int64_t i = threadIdx.x; i < half; i += blockDim.x) {
    const float ang = rope_angle(pos, i, d);
    float sn, c;
    sincosf(ang, &sn, &c);
    float q1 = ld(q, base + i), q2 = ld(q, base + i + half);
    st(q, base + i, q1 * c - q2 * sn);
    st(q, base + i + half, q2 * c + q1 * sn);
    float k1 = ld(k, base + i), k2 = ld(k, base + i + half);
    st(Kc, cbase + i, k1 * c - k2 * sn);
    st(Kc, cbase + i + half, k2 * c + k1 * sn);
    Vc[cbase + i] = v[base + i];
    Vc[cbase + i + half] = v[base + i + half];
  }
}

// ---------------------------------------------------------------- argmax
__global__ void __launch_bounds__(256) argmax_kernel(const float* logits, int32_t* tok, int32_t* gen,
                                                     int64_t V, int64_t B, int64_t row) {
  __shared__ float sv[256];
  __shared__ int64_t si[256];
  const int64_t b = blockIdx.x;
  const float* l = logits + b * V;
  float best = -INFINITY;
  int64_t bi = V;  // sentinel larger than any index
  for (int64_t j = threadIdx.x; j < V; j += blockDim.x) {
    float v = l[j];
    if (v > best || (v == best && j < bi)) {
      best = v;
      bi = j;
    }
  }
  sv[threadIdx.x] = best;
  si[threadIdx.x] = bi;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (threadIdx.x < s) {
      float v2 = sv[threadIdx.x + s];
      int64_t i2 = si[threadIdx.x + s];
      if (v2 > sv[threadIdx.x] || (v2 == sv[threadIdx.x] && i2 < si[threadIdx.x])) {
        sv[threadIdx.x] = v2;
        si[threadIdx.x] = i2;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    int32_t r = int32_t(si[0] >= V ? 0 : si[0]);
    tok[b] = r;
    if (gen) gen[row * B + b] = r;
  }
}

template <class T>
hipError_t rope_kv(uint8_t* const* p, const int64_t* s, hipStream_t st_) {
  const int64_t B = s[0], S = s[1], nH = s[2], d = s[3], Lmax = s[4], pos0 = s[5];
  int threads = int(d / 2 < 64 ? 64 : d / 2);
  hipLaunchKernelGGL(rope_kv_kernel<T>, dim3(unsigned(B * S * nH)), dim3(threads), 0, st_, (T*)p[0],
                     (const T*)p[1], (const T*)p[2], (T*)p[3], (T*)p[4], S, nH, d, Lmax, pos0);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_poison(uint8_t* p, uint64_t bytes, hipStream_t s) {
  return hipMemsetAsync(p, 0xff, bytes, s);
}

hipError_t launch_op(const Kernel& k, const std::vector<Tensor>& T, uint8_t* const* p, hipStream_t s) {
  const int64_t* sh = k.shape;
  auto dt = [&](int i) { return T[k.ids[i]].dtype; };
  switch (k.op) {
    case AUVM_OP_TOUCH: {
      TouchArgs a{};
      a.n = int(k.ids.size()) - 1;
      a.log = (uint32_t*)p[0];
      a.slot = sh[0];
      for (int i = 0; i < a.n; ++i) {
        a.data[i] = (uint32_t*)p[i + 1];
        a.words[i] = T[k.ids[i + 1]].bytes / 4;
        a.mode[i] = k.modes[i + 1];
      }
      hipLaunchKernelGGL(touch_kernel, dim3(a.n), dim3(256), 0, s, a);
      return hipGetLastError();
    }
    case AUVM_OP_EMBED:
      if (dt(1) == AUVM_BF16)
        hipLaunchKernelGGL(embed_kernel<bf16_t>, dim3(unsigned(sh[0])), dim3(256), 0, s,
                           (const int32_t*)p[0], (const bf16_t*)p[1], (float*)p[2], sh[1], sh[2]);
      else
        hipLaunchKernelGGL(embed_kernel<float>, dim3(unsigned(sh[0])), dim3(256), 0, s,
                           (const int32_t*)p[0], (const float*)p[1], (float*)p[2], sh[1], sh[2]);
      return hipGetLastError();
    case AUVM_OP_LAYERNORM:
      if (dt(3) == AUVM_BF16)
        launch_norm<bf16_t, true>(p[0], p[1], p[2], p[3], sh, 1e-5f, s);
      else
        launch_norm<float, true>(p[0], p[1], p[2], p[3], sh, 1e-5f, s);
      return hipGetLastError();
    case AUVM_OP_RMSNORM:
      if (dt(2) == AUVM_BF16)
        launch_norm<bf16_t, false>(p[0], p[1], nullptr, p[2], sh, 1e-6f, s);
      else
        launch_norm<float, false>(p[0], p[1], nullptr, p[2], sh, 1e-6f, s);
      return hipGetLastError();
    case AUVM_OP_LINEAR:
    case AUVM_OP_LINEAR_GELU:
    case AUVM_OP_LINEAR_RESID:
    case AUVM_OP_LINEAR_SWIGLU: {
      GemmArgs g{};
      bool sw = k.op == AUVM_OP_LINEAR_SWIGLU;
      g.M = sh[0];
      g.N = sh[1];
      g.K = sh[2];
      g.a = p[0];
      g.w = p[1];
      g.w2 = sw ? p[2] : nullptr;
      g.c = p[sw ? 3 : 2];
      g.epi = k.op == AUVM_OP_LINEAR ? EPI_STORE
              : k.op == AUVM_OP_LINEAR_GELU ? EPI_GELU
              : k.op == AUVM_OP_LINEAR_RESID ? EPI_RESID : EPI_SWIGLU;
      g.in_bf16 = dt(0) == AUVM_BF16;
      g.out_bf16 = dt(sw ? 3 : 2) == AUVM_BF16;
      return launch_gemm(g, s);
    }
    case AUVM_OP_LINEAR_QKV: {
      GemmArgs g{};
      g.M = sh[0];
      g.N = sh[1];
      g.K = sh[2];
      g.a = p[0];
      g.epi = EPI_STORE;
      g.in_bf16 = dt(0) == AUVM_BF16;
      g.out_bf16 = dt(4) == AUVM_BF16;
      g.groups = 3;
      for (int i = 0; i < 3; ++i) {
        g.gw[i] = p[1 + i];
        g.gc[i] = p[4 + i];
      }
      return launch_gemm(g, s);
    }
    case AUVM_OP_COPY:
      return hipMemcpyAsync(p[1], p[0], size_t(sh[0]), hipMemcpyDeviceToDevice, s);
    case AUVM_OP_TRANSPOSE:
      return launch_transpose(p[0], p[1], sh[0], sh[1], dt(0) == AUVM_BF16, s);
    case AUVM_OP_SWIGLU_ACT:
    case AUVM_OP_SWIGLU_BWD:
      return launch_swiglu(k.op == AUVM_OP_SWIGLU_BWD, p, sh[0] * sh[1], dt(0) == AUVM_BF16, s);
    case AUVM_OP_RMSNORM_BWD:
      return launch_rmsnorm_bwd(p, sh[0], sh[1], int(sh[2]), dt(1) == AUVM_BF16, s);
    case AUVM_OP_ATTN_BWD:
      return launch_attn_bwd(p, sh[0], sh[1], sh[2], s);
    case AUVM_OP_ROPE_BWD:
      return launch_rope_bwd(p, sh[0], sh[1], sh[2], sh[3], dt(0) == AUVM_BF16, s);
    case AUVM_OP_XENT:
      return launch_xent(p, sh[0], sh[1], dt(3) == AUVM_BF16, s);
    case AUVM_OP_EMBED_BWD:
      return launch_embed_bwd(p, sh[0], sh[1], sh[2], s);
    case AUVM_OP_ADAM: {
      // hyperparameters in fixed point; bias corrections in double on the host
      const double lr = sh[2] * 1e-9, b1 = sh[3] * 1e-6, b2 = sh[4] * 1e-6, eps = sh[5] * 1e-12, wd = sh[6] * 1e-6;
      const double t = double(sh[1]);
      AdamArgs a;
      a.b1 = float(b1);
      a.b2 = float(b2);
      a.eps = float(eps);
      a.decay = float(1.0 - lr * wd);
      a.step_size = float(lr / (1.0 - std::pow(b1, t)));
      a.inv_bc2 = float(1.0 / (1.0 - std::pow(b2, t)));
      return launch_adam(p, sh[0], a, dt(4) == AUVM_BF16, s);
    }
    case AUVM_OP_MOE_ROUTE:
      return launch_moe_route(p[0], p[1], reinterpret_cast<int32_t*>(p[2]), reinterpret_cast<float*>(p[3]), sh[0],
                              sh[1], int(sh[2]), int(sh[3]), dt(0) == AUVM_BF16, s);
    case AUVM_OP_MOE_DISPATCH:
      return launch_moe_dispatch(reinterpret_cast<const int32_t*>(p[0]), reinterpret_cast<int32_t*>(p[1]),
                                 reinterpret_cast<int32_t*>(p[2]), sh[0], int(sh[2]), int(sh[1]), sh[3], s);
    case AUVM_OP_MOE_UP:
    case AUVM_OP_MOE_DOWN: {
      // the expert's row list is row e of the [E, M+1] list tensor
      const bool up = k.op == AUVM_OP_MOE_UP;
      GemmArgs g{};
      g.M = sh[0];
      g.N = sh[1];
      g.K = sh[2];
      g.list = reinterpret_cast<const int32_t*>(p[1]) + sh[3] * (sh[0] + 1);
      g.topk = int(sh[5]);
      g.in_bf16 = true;
      g.a = p[0];
      if (up) {
        g.w = p[2];
        g.w2 = p[3];
        g.c = p[4];
        g.epi = EPI_SWIGLU;
        g.out_bf16 = true;
      } else {
        g.rw = reinterpret_cast<const float*>(p[2]);
        g.w = p[3];
        g.c = p[4];
        g.epi = EPI_MOE;
        g.out_bf16 = false;
      }
      return launch_gemm(g, s);
    }
    case AUVM_OP_ATTN_QKV:
    case AUVM_OP_ATTN_CACHE: {
      AttnArgs a{};
      const bool qkv = k.op == AUVM_OP_ATTN_QKV;
      const int64_t B = sh[0], S = sh[1], nH = sh[2], d = sh[3];
      a.B = B;
      a.S = S;
      a.nH = nH;
      a.d = d;
      if (qkv) {
        const int64_t Hd = nH * d;
        a.q = p[0];
        a.k = p[0] + Hd * (dt(0) == AUVM_BF16 ? 2 : 4);
        a.v = p[0] + 2 * Hd * (dt(0) == AUVM_BF16 ? 2 : 4);
        a.o = p[1];
        a.q_rs = 3 * Hd;
        a.kv_rs = 3 * Hd;
        a.kv_bstride = S * 3 * Hd;  // next sequence
        a.kv_hstride = d;           // next head: column block
        a.pos0 = 0;
      } else {
        const int64_t Lmax = sh[4];
        a.q = p[0];
        a.k = p[1];
        a.v = p[2];
        a.o = p[3];
        a.q_rs = nH * d;
        a.kv_rs = d;
        a.kv_bstride = nH * Lmax * d;
        a.kv_hstride = Lmax * d;
        a.pos0 = sh[5];
      }
      a.o_rs = nH * d;
      a.bf16 = dt(0) == AUVM_BF16;
      if (!qkv && k.ids.size() > 4) a.lse = reinterpret_cast<float*>(p[4]);
      return launch_attention(a, s);
    }
    case AUVM_OP_ROPE_KV:
      return dt(0) == AUVM_BF16 ? rope_kv<bf16_t>(p, sh, s) : rope_kv<float>(p, sh, s);
    case AUVM_OP_ARGMAX:
      hipLaunchKernelGGL(argmax_kernel, dim3(unsigned(sh[0])), dim3(256), 0, s, (const float*)p[0],
                         (int32_t*)p[1], k.ids.size() > 2 ? (int32_t*)p[2] : nullptr, sh[1], sh[0],
                         sh[2]);
      return hipGetLastError();
  }
  return hipErrorInvalidValue;
}

}  // namespace auvm
