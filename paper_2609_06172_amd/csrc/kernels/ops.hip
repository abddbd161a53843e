// Memory-bound and small kernels: touch, embedding gather, LayerNorm,
// RMSNorm, RoPE + KV-cache append, argmax, and the op dispatch.
#include <hip/hip_runtime.h>

#include "../kernels.h"
#include "common.h"
#include "gemm.h"
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
    double ang = double(pos) * pow(10000.0, -2.0 * double(i) / double(d));
    float c = float(cos(ang)), sn = float(sin(ang));
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
        hipLaunchKernelGGL((norm_kernel<bf16_t, true>), dim3(unsigned(sh[0])), dim3(256), 0, s,
                           (const float*)p[0], (const bf16_t*)p[1], (const bf16_t*)p[2], (bf16_t*)p[3],
                           sh[1], sh[2], sh[3], 1e-5f);
      else
        hipLaunchKernelGGL((norm_kernel<float, true>), dim3(unsigned(sh[0])), dim3(256), 0, s,
                           (const float*)p[0], (const float*)p[1], (const float*)p[2], (float*)p[3],
                           sh[1], sh[2], sh[3], 1e-5f);
      return hipGetLastError();
    case AUVM_OP_RMSNORM:
      if (dt(2) == AUVM_BF16)
        hipLaunchKernelGGL((norm_kernel<bf16_t, false>), dim3(unsigned(sh[0])), dim3(256), 0, s,
                           (const float*)p[0], (const bf16_t*)p[1], (const bf16_t*)nullptr,
                           (bf16_t*)p[2], sh[1], sh[2], sh[3], 1e-6f);
      else
        hipLaunchKernelGGL((norm_kernel<float, false>), dim3(unsigned(sh[0])), dim3(256), 0, s,
                           (const float*)p[0], (const float*)p[1], (const float*)nullptr, (float*)p[2],
                           sh[1], sh[2], sh[3], 1e-6f);
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
