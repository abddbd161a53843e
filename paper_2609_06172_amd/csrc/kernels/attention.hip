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
  if (a.lse && lane == 0) a.lse[bh * a.S + i] = m + logf(l);   // scores here are already scaled
}

// Decode attention, head dim 128, bf16: one workgroup per query row.
// A key (or value) row is 256 B = 16 lanes x 16 B, so a wave loads four
// consecutive rows per instruction, fully coalesced.  Lane (grp, sub) =
// (l / 16, l % 16) holds dims 8*sub..8*sub+7; a wave takes blocks of 24 keys
// (key 24*blk + 4*u + grp for u = 0..5, six loads of K and six of V in
// flight), the eight waves interleave blocks, each keeps an online softmax and
// the waves are merged through LDS.  Loaded rows stay packed bf16 in
// registers until used (at most 128 VGPRs, no spills: two workgroups per
// compute unit).
constexpr int kDecU = 6;
constexpr int kDecWaves = 8;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// the two bf16 values packed in a word, as floats
__device__ __forceinline__ float bf_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

__device__ __forceinline__ void load8(const bf16_t* p, float* f) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  u32x4 v = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(v[i] << 16);
    f[2 * i + 1] = __uint_as_float(v[i] & 0xffff0000u);
  }
}

__global__ void __launch_bounds__(64 * kDecWaves, 4) attn_decode_d128(AttnArgs a) {
  __shared__ float sm[kDecWaves], sl[kDecWaves], sacc[kDecWaves][128];
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
  for (int64_t j0 = int64_t(wv) * 4 * kDecU; j0 <= last; j0 += kDecWaves * 4 * kDecU) {
    u32x4 kr[kDecU], vr[kDecU];
    float sc[kDecU];
#pragma unroll
    for (int u = 0; u < kDecU; ++u) {
      const int64_t j = j0 + 4 * u + grp;
      if (j <= last) {
        kr[u] = *reinterpret_cast<const u32x4*>(kb + j * a.kv_rs);
        vr[u] = *reinterpret_cast<const u32x4*>(vb + j * a.kv_rs);
      } else {
        kr[u] = vr[u] = u32x4{0u, 0u, 0u, 0u};
      }
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int u = 0; u < kDecU; ++u) {
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s = fmaf(qf[2 * e], bf_lo(kr[u][e]), s);
        s = fmaf(qf[2 * e + 1], bf_hi(kr[u][e]), s);
      }
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
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] = fmaf(p, bf_lo(vr[u][e]), acc[2 * e]);
        acc[2 * e + 1] = fmaf(p, bf_hi(vr[u][e]), acc[2 * e + 1]);
      }
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
    for (int w = 1; w < kDecWaves; ++w) M = fmaxf(M, sm[w]);
    float L = 0.f, r = 0.f;
    for (int w = 0; w < kDecWaves; ++w) {
      const float f = sm[w] == -INFINITY ? 0.f : __expf(sm[w] - M);
      L += sl[w] * f;
      r += sacc[w][dd] * f;
    }
    o[dd] = f2bf(r / L);
  }
}

// Prefill attention, head dim 128, bf16, on matrix cores (flash-style).
// One workgroup of 4 waves per (b, h, block of 128 queries); wave w owns
// queries 32w..32w+31.  Everything is computed transposed, so that a lane owns
// one query: lane l holds query l % 32 and half of the keys or dims.
//   S^T = K Q^T: A = a 32-key x 16-dim K fragment (LDS), B = Q^T (registers),
//     2 key tiles x 8 dim steps of v_mfma_f32_32x32x16_bf16 per 64-key block;
//   online softmax: a query's 64 scores sit in lanes l and l+32 (32 each), so
//     its max and sum are one exchange between the two (v_permlane32_swap,
//     which swaps the upper half of one register with the lower half of
//     another, on the VALU rather than through LDS);
//   O^T += V^T P^T: A = a 32-dim x 16-key fragment of V^T, read from the
//     row-major V tile with the LDS transpose read (ds_read_b64_tr_b16: within
//     each 16-lane group, lane 4a+b receives element b of the 8-byte rows that
//     lanes a, a+4, a+8, a+12 address), B = P^T assembled in registers (each
//     lane trades four values with its partner lane, by the same swap); 4 dim
//     tiles x 4 key steps per block.
// K and V blocks of 64 keys go from global memory straight into one of two
// LDS buffers (16-byte global_load_lds; a 256-byte row's chunks are permuted
// by a row-dependent XOR that keeps fragment and transpose reads free of bank
// conflicts); the next block streams in while this one is consumed, one
// barrier per block.  Rows past the last visible key are clamped to it: those
// keys are masked, so they contribute exactly zero.  A wave skips blocks
// wholly past its queries; only blocks crossing its diagonal are masked.
// Blocks are ordered per XCD, heaviest first (xcd_order).
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

constexpr int FW = 4;          // waves per workgroup
constexpr int FQ = 32 * FW;    // queries per workgroup
constexpr int FK = 64, FD = 128;
constexpr int TS = FK * FD;    // elements per K or V tile (rows of 256 bytes)
constexpr size_t kFlashLds = size_t(4 * TS) * sizeof(bf16_t);   // K and V, two buffers each

// two floats to bf16 (round to nearest even, one conversion instruction)
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  const bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// Slot of a 16-byte chunk in a 256-byte tile row: chunk ^ kv_swz(row).  A K
// fragment read takes one chunk of 16 aligned consecutive rows per pass; a V
// transpose read takes 4 chunks of 4 consecutive rows.  Rotating the row's
// low nibble by two bits gives both patterns 16 distinct slots (no LDS bank
// conflicts; rows 256 bytes apart all start on the same bank).
__device__ __forceinline__ int kv_swz(int row) { return ((row & 3) << 2) | ((row >> 2) & 3); }

// element offset of (row, dim) in a swizzled 64 x 128 tile
__device__ __forceinline__ int tile_at(int row, int dim) {
  return row * FD + (((dim >> 3) ^ kv_swz(row)) << 3) + (dim & 7);
}

// One 64-key block of K or V rows k0.. into an LDS tile: wave wv fills rows
// 16*i + 4*wv .. +3 for i = 0..3 (1 KB per instruction); lane l fills row
// +l/16, slot l % 16 with the row's chunk (l % 16) ^ kv_swz(row).
__device__ __forceinline__ void load_kv(bf16_t* tile, const bf16_t* __restrict__ G, int64_t rs, int64_t k0,
                                        int64_t klast, int wv, int lane) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r0 = 16 * i + 4 * wv;
    const int row = r0 + (lane >> 4);
    const int64_t key = k0 + row <= klast ? k0 + row : klast;
    const int chunk = (lane & 15) ^ kv_swz(row);
    __builtin_amdgcn_global_load_lds(G + key * rs + 8 * chunk, tile + r0 * FD, 16, 0, 0);
  }
}

// The same rows for a block wholly before klast, from per-lane byte offsets
// (row * rs + 8 * chunk elements, computed once) off a uniform base: no
// clamp and no 64-bit address arithmetic per load.
__device__ __forceinline__ void load_kv_rows(bf16_t* tile, const char* base, const uint32_t* boff, int wv) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const bf16_t*>(base + boff[i]), tile + (16 * i + 4 * wv) * FD,
                                     16, 0, 0);
}

// the B-operand fragment (16 rows of k, this lane's column) of k-step u
// (0, 1) from one 32 x 32 C tile t: rows 16u.. of the tile; the lane and its
// partner (lane ^ 32) trade one 4-row group each.  c_to_b: k-step s of a
// pair of tiles t[0..1] (rows 0..31, 32..63).
__device__ __forceinline__ bf16x8 c_to_b1(const f32x16& t, int u) {
  const int g0 = 2 * u;
  const uint32_t a0 = pack_bf16(t[4 * g0 + 0], t[4 * g0 + 1]);
  const uint32_t a1 = pack_bf16(t[4 * g0 + 2], t[4 * g0 + 3]);
  const uint32_t b0 = pack_bf16(t[4 * g0 + 4], t[4 * g0 + 5]);
  const uint32_t b1 = pack_bf16(t[4 * g0 + 6], t[4 * g0 + 7]);
  // v_permlane32_swap(x, y) returns x' = (lanes < 32: x, lanes >= 32: y of
  // lane - 32) and y' = (lanes < 32: x of lane + 32, lanes >= 32: y): lane
  // l < 32 gets {its a, its partner's a}, lane l >= 32 {its partner's b, its b}
  const auto x0 = __builtin_amdgcn_permlane32_swap(a0, b0, false, false);
  const auto x1 = __builtin_amdgcn_permlane32_swap(a1, b1, false, false);
  const u32x4v pf = {x0[0], x1[0], x0[1], x1[1]};
  return __builtin_bit_cast(bf16x8, pf);
}
__device__ __forceinline__ bf16x8 c_to_b(const f32x16* t, int s) { return c_to_b1(t[s >> 1], s & 1); }
__device__ __forceinline__ bf16x8 tile_t_frag(const bf16_t* tile, int s, int dt, int lane) {
  const int tg = lane >> 4, tj = lane & 15;
  const int row = 16 * s + 8 * (tg >> 1) + (tj >> 2);
  const int dim = 32 * dt + 16 * (tg & 1) + 4 * (tj & 3);
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  const i16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(tile + tile_at(row, dim)));
  const i16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(tile + tile_at(row + 4, dim)));
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  const i16x8 vv = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
  return __builtin_bit_cast(bf16x8, vv);
}

// max and sum of a value and its partner lane's (lane ^ 32), the same on both lanes
__device__ __forceinline__ float swap_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float swap_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Workgroup order of the flash kernels (grid = nblk blocks of each of nbh
// (batch, head) pairs).  Workgroup w runs on XCD w % 8 (round-robin
// dispatch), and each XCD has its own L2: all blocks of one (b, h) go to the
// same XCD, so its K and V (or Q and dO) are fetched into one L2 only.  An
// XCD with more than eight heads takes them four at a time, all blocks of a
// group before the next, heaviest blocks (rank 0) of the group first: the
// blocks resident on the XCD together then share few heads, and the K and V
// tiles they walk stay in its L2 (one group otherwise).  Without eight-way
// divisible heads the order is rank-major.
__device__ __forceinline__ void xcd_order(int64_t w, int64_t nbh, int64_t nblk, int64_t* rank, int64_t* bh) {
  if (nbh % 8 == 0) {
    const int64_t x = w % 8, slot = w / 8, hx = nbh / 8;
    const int64_t G = hx <= 8 ? hx : 4;                     // heads per group
    const int64_t g0 = slot / (G * nblk) * G;               // first head of the group
    const int64_t gn = hx - g0 < G ? hx - g0 : G;           // heads in it (the last may hold fewer)
    const int64_t in = slot - g0 * nblk;
    *rank = in / gn;
    *bh = (g0 + in % gn) * 8 + x;
  } else {
    *rank = w / nbh;
    *bh = w % nbh;
  }
}

__global__ void __launch_bounds__(64 * FW, 2) attn_prefill_d128(AttnArgs a, int64_t nqb) {
  extern __shared__ __align__(16) bf16_t fsm[];
  bf16_t* Ks = fsm;                 // [2][FK][FD]
  bf16_t* Vs = fsm + 2 * TS;        // [2][FK][FD]
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int lq = lane & 31, lh = lane >> 5;
  int64_t rank, bh;
  xcd_order(blockIdx.x, int64_t(gridDim.x) / nqb, nqb, &rank, &bh);
  const int64_t qb = nqb - 1 - rank;
  const int64_t h = bh % a.nH, b = bh / a.nH;
  const int64_t q0 = qb * FQ, qw = q0 + 32 * wv;
  const bf16_t* Q = reinterpret_cast<const bf16_t*>(a.q) + (b * a.S) * a.q_rs + h * FD;
  const bf16_t* Kg = reinterpret_cast<const bf16_t*>(a.k) + b * a.kv_bstride + h * a.kv_hstride;
  const bf16_t* Vg = reinterpret_cast<const bf16_t*>(a.v) + b * a.kv_bstride + h * a.kv_hstride;
  bf16_t* O = reinterpret_cast<bf16_t*>(a.o) + (b * a.S) * a.o_rs + h * FD;

  // Q^T fragment for dim step c: dims 16c + 8*lh .. +8 of this lane's query
  const int64_t qr = qw + lq, qpos = a.pos0 + qr;
  bf16x8 qf[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    if (qr < a.S)
      qf[c] = *reinterpret_cast<const bf16x8*>(Q + qr * a.q_rs + 16 * c + 8 * lh);
    else
      qf[c] = bf16x8{};
  }
  // softmax in base 2 on raw scores: p = 2^(c*s - c*max) with c = log2(e)/sqrt(128)
  constexpr float c2 = 0.12751743074565512f;
  // O^T tile dt: element e is dim 32*dt + 8*(e/4) + 4*lh + e%4 of this lane's query
  f32x16 ot[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) ot[t] = f32x16{};
  float m = -INFINITY, l = 0.f;
  // the workgroup's queries see keys 0 .. klast; this wave's, 0 .. wlast
  const int64_t qlast = (q0 + FQ - 1 < a.S ? q0 + FQ - 1 : a.S - 1);
  const int64_t klast = a.pos0 + qlast;
  const int64_t wlast = a.pos0 + qw + 31;

  // byte offsets of the rows this lane stages, within a block
  uint32_t boff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 16 * i + 4 * wv + (lane >> 4);
    boff[i] = uint32_t((row * a.kv_rs + 8 * ((lane & 15) ^ kv_swz(row))) * int64_t(sizeof(bf16_t)));
  }
  const int64_t rsb = a.kv_rs * int64_t(sizeof(bf16_t));
  auto stage = [&](int64_t k1, int b2) {
    if (k1 + FK - 1 <= klast) {
      load_kv_rows(Ks + b2 * TS, reinterpret_cast<const char*>(Kg) + k1 * rsb, boff, wv);
      load_kv_rows(Vs + b2 * TS, reinterpret_cast<const char*>(Vg) + k1 * rsb, boff, wv);
    } else {                         // the last block: rows past klast clamped
      load_kv(Ks + b2 * TS, Kg, a.kv_rs, k1, klast, wv, lane);
      load_kv(Vs + b2 * TS, Vg, a.kv_rs, k1, klast, wv, lane);
    }
  };
  stage(0, 0);
  int buf = 0;
  for (int64_t k0 = 0; k0 <= klast; k0 += FK, buf ^= 1) {
    __builtin_amdgcn_s_waitcnt(0);   // this wave's loads of the block have landed
    __syncthreads();                 // ... and every other wave's; the other buffer is free
    asm volatile("" ::: "memory");   // LDS now holds data written outside the compiler's view
    if (k0 + FK <= klast) stage(k0 + FK, buf ^ 1);
    if (k0 > wlast) continue;
    const bf16_t* ks = Ks + buf * TS;
    const bf16_t* vs = Vs + buf * TS;
    // S^T tile kt: element e is key k0 + 32*kt + 8*(e/4) + 4*lh + e%4 of this
    // lane's query.  Dim steps go in pairs; each pair is one scheduling region
    // whose first MFMA takes fragments read during the previous region, and
    // whose other MFMAs alternate with the reads of the next pair (the
    // compiler waits for every outstanding LDS read before a region's first
    // MFMA).
    f32x16 st[2] = {f32x16{}, f32x16{}};
    bf16x8 kf[2][4];   // [pair parity][2 * (dim step in pair) + kt]
    auto kread = [&](int cp, int set) {
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
          kf[set][2 * u + kt] =
              *reinterpret_cast<const bf16x8*>(ks + tile_at(32 * kt + lq, 16 * (2 * cp + u) + 8 * lh));
    };
    kread(0, 0);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int cp = 0; cp < 4; ++cp) {
      const int set = cp & 1;
      if (cp + 1 < 4) kread(cp + 1, set ^ 1);
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
          st[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[set][2 * u + kt], qf[2 * cp + u], st[kt], 0, 0, 0);
      if (cp + 1 < 4) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // V^T fragments of key steps 0 and 1, read while the softmax runs
    bf16x8 vf[2][4];   // [key step parity][dt]
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) vf[s][dt] = tile_t_frag(vs, s, dt, lane);
    if (k0 + FK - 1 > a.pos0 + qw) {   // the block crosses this wave's diagonal
      const int kq = int(qpos - k0);   // keys of the block past this one are masked
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (32 * kt + 8 * (e >> 2) + 4 * lh + (e & 3) > kq) st[kt][e] = -INFINITY;
    }
    // the block's maximum: a tree over the lane's 32 scores, then the partner lane's
    float t8[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int kt = i >> 2, e = 4 * (i & 3);
      t8[i] = fmaxf(fmaxf(st[kt][e], st[kt][e + 1]), fmaxf(st[kt][e + 2], st[kt][e + 3]));
    }
    float mx = fmaxf(fmaxf(fmaxf(t8[0], t8[1]), fmaxf(t8[2], t8[3])), fmaxf(fmaxf(t8[4], t8[5]), fmaxf(t8[6], t8[7])));
    mx = swap_max(mx);
    // m is the score the exponentials are taken against.  It moves (and the
    // running sum and output are rescaled) only when a block's maximum
    // exceeds it by more than kGrow raw-score units, so p stays below 2^8;
    // the common factor cancels in o and in the log-sum-exp.
    constexpr float kGrow = 8.f / c2;
    if (__any(mx > m + kGrow)) {   // rare after the first blocks
      const bool grow = mx > m + kGrow;
      const float corr = grow ? __builtin_amdgcn_exp2f((m - mx) * c2) : 1.f;   // 0 while m = -inf
      m = grow ? mx : m;
      l *= corr;
#pragma unroll
      for (int t = 0; t < 4; ++t) ot[t] *= corr;
    }
    // a query with no visible key yet keeps m = -inf and contributes nothing
    const float off = m == -INFINITY ? 0.f : m * c2;
    float ps[4] = {0.f, 0.f, 0.f, 0.f};   // four partial sums: short dependency chains
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = __builtin_amdgcn_exp2f(fmaf(st[kt][e], c2, -off));
        st[kt][e] = p;
        ps[e & 3] += p;
      }
    l += swap_sum((ps[0] + ps[1]) + (ps[2] + ps[3]));
    // O^T += V^T P^T over key steps s (keys 16s..16s+15 of the block); the
    // V^T fragments of step s+2 are read into the slots step s frees
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const bf16x8 pb = c_to_b(st, s);
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        ot[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[s & 1][dt], pb, ot[dt], 0, 0, 0);
        if (s + 2 < 4) vf[s & 1][dt] = tile_t_frag(vs, s + 2, dt, lane);
      }
    }
  }
  if (qr < a.S) {
    const float inv = 1.f / l;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int e = 0; e < 16; ++e)
        O[qr * a.o_rs + 32 * dt + 8 * (e >> 2) + 4 * lh + (e & 3)] = f2bf(ot[dt][e] * inv);
    // m is the raw-score maximum and l sums exp((s - m) / sqrt(128))
    if (a.lse && lh == 0) a.lse[bh * a.S + qr] = m * 0.08838834764831845f + logf(l);
  }
}

// ---------------------------------------------------------------- backward (head dim 128)
// Causal attention backward on matrix cores, from the forward's q, K, V, its
// per-query log-sum-exp and D = rowsum(dO o).  Two passes, no atomics:
//   dQ: one workgroup per (b, h, 128 queries), like the forward: S^T = K Q^T
//     and dP^T = V dO^T (K, V tiles in LDS; Q^T, dO^T fragments of the
//     wave's queries in registers), P^T = exp(S^T/sqrt(d) - lse),
//     dS^T = P^T (dP^T - D), then dQ^T += K^T dS^T with K^T fragments by
//     LDS transpose reads and dS^T traded into the B-operand layout;
//   dK, dV: one workgroup per (b, h, 128 keys), the mirror image: S = Q K^T
//     and dP = dO V^T (Q, dO tiles in LDS, the wave's K, V rows in
//     registers), then dV^T += dO^T P and dK^T += Q^T dS.
// A lane owns one query (dQ pass) or one key (dK, dV pass), so the 32 x 32
// accumulator tiles map to one row of the output each.  The dQ pass fits in
// 256 registers a lane (two workgroups per CU); the dK, dV pass, with two
// accumulator sets, takes one workgroup per CU and software-pipelines its
// LDS reads instead.

constexpr float kBwdScale = 0.08838834764831845f;   // 1 / sqrt(128)
constexpr float kLog2eF = 1.4426950408889634f;

__global__ void __launch_bounds__(64 * FW, 2) attn_bwd_dq_d128(AttnBwdArgs a, int64_t nqb) {
  extern __shared__ __align__(16) bf16_t fsm[];
  bf16_t* Ks = fsm;                 // [2][FK][FD]
  bf16_t* Vs = fsm + 2 * TS;        // [2][FK][FD]
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int lq = lane & 31, lh = lane >> 5;
  int64_t rank, bh;
  xcd_order(blockIdx.x, int64_t(gridDim.x) / nqb, nqb, &rank, &bh);
  const int64_t qb = nqb - 1 - rank;
  const int64_t h = bh % a.nH, b = bh / a.nH, S = a.S;
  const int64_t q0 = qb * FQ, qw = q0 + 32 * wv, qr = qw + lq;
  const bf16_t* Q = reinterpret_cast<const bf16_t*>(a.q) + (b * S) * a.q_rs + h * FD;
  const bf16_t* dO = reinterpret_cast<const bf16_t*>(a.dO) + (b * S) * a.q_rs + h * FD;
  const bf16_t* Kg = reinterpret_cast<const bf16_t*>(a.k) + bh * S * FD;
  const bf16_t* Vg = reinterpret_cast<const bf16_t*>(a.v) + bh * S * FD;
  bf16x8 qf[8], df[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    qf[c] = qr < S ? *reinterpret_cast<const bf16x8*>(Q + qr * a.q_rs + 16 * c + 8 * lh) : bf16x8{};
    df[c] = qr < S ? *reinterpret_cast<const bf16x8*>(dO + qr * a.q_rs + 16 * c + 8 * lh) : bf16x8{};
  }
  const float lse2 = qr < S ? a.lse[bh * S + qr] * kLog2eF : 0.f;
  const float Dq = qr < S ? a.D[bh * S + qr] : 0.f;
  const float c2 = kBwdScale * kLog2eF;
  f32x16 dqt[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) dqt[t] = f32x16{};
  const int64_t klast = (q0 + FQ - 1 < S ? q0 + FQ - 1 : S - 1);
  const int64_t wlast = qw + 31;
  load_kv(Ks, Kg, FD, 0, klast, wv, lane);
  load_kv(Vs, Vg, FD, 0, klast, wv, lane);
  int buf = 0;
  for (int64_t k0 = 0; k0 <= klast; k0 += FK, buf ^= 1) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    asm volatile("" ::: "memory");
    if (k0 + FK <= klast) {
      load_kv(Ks + (buf ^ 1) * TS, Kg, FD, k0 + FK, klast, wv, lane);
      load_kv(Vs + (buf ^ 1) * TS, Vg, FD, k0 + FK, klast, wv, lane);
    }
    // A wave whose queries all precede the block still runs it, fully
    // masked: a uniform loop body keeps the dQ accumulators in place.
    const bf16_t* ks = Ks + buf * TS;
    const bf16_t* vs = Vs + buf * TS;
    // S^T and dP^T tiles kt: element e is key k0 + 32 kt + 8 (e/4) + 4 lh + e%4 of query qr
    f32x16 st[2], dpt[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      st[kt] = f32x16{};
      dpt[kt] = f32x16{};
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(ks + tile_at(32 * kt + lq, 16 * c + 8 * lh));
        st[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[c], st[kt], 0, 0, 0);
        const bf16x8 vf = *reinterpret_cast<const bf16x8*>(vs + tile_at(32 * kt + lq, 16 * c + 8 * lh));
        dpt[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, df[c], dpt[kt], 0, 0, 0);
      }
    }
    // P^T, then dS^T.  Only a block that crosses this wave's diagonal or
    // holds queries past S is masked (a select, not a branch): there a key
    // counts when its offset in the block is at most kq.
    const bool edge = k0 + FK - 1 > qw || qw + 31 >= S;
    const int kq = qr < S ? int(qr - k0) - 4 * lh : -1;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float p = __builtin_amdgcn_exp2f(fmaf(st[kt][e], c2, -lse2));
        if (edge) p = 32 * kt + 8 * (e >> 2) + (e & 3) <= kq ? p : 0.f;
        st[kt][e] = p * (dpt[kt][e] - Dq);       // dS^T
      }
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const bf16x8 dsb = c_to_b(st, s);
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
        dqt[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tile_t_frag(ks, s, dt, lane), dsb, dqt[dt], 0, 0, 0);
    }
  }
  if (qr < S) {
    bf16_t* dq = reinterpret_cast<bf16_t*>(a.dq) + (b * S) * a.q_rs + h * FD;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int e = 0; e < 16; ++e)
        dq[qr * a.q_rs + 32 * dt + 8 * (e >> 2) + 4 * lh + (e & 3)] = f2bf(dqt[dt][e] * kBwdScale);
  }
}

__global__ void __launch_bounds__(64 * FW, 1) attn_bwd_dkv_d128(AttnBwdArgs a, int64_t nkb) {
  extern __shared__ __align__(16) bf16_t fsm[];
  bf16_t* Qs = fsm;                 // [2][FK][FD] query rows
  bf16_t* Os = fsm + 2 * TS;        // [2][FK][FD] dO rows
  __shared__ __align__(16) float lsS[2][FK], dsS[2][FK];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int lq = lane & 31, lh = lane >> 5;
  int64_t kb, bh;   // key block 0 sees every query: the heaviest
  xcd_order(blockIdx.x, int64_t(gridDim.x) / nkb, nkb, &kb, &bh);
  const int64_t h = bh % a.nH, b = bh / a.nH, S = a.S;
  const int64_t kbase = kb * FQ, kw = kbase + 32 * wv, kr = kw + lq;
  const int64_t krc = kr < S ? kr : S - 1;
  const bf16_t* Qg = reinterpret_cast<const bf16_t*>(a.q) + (b * S) * a.q_rs + h * FD;
  const bf16_t* Og = reinterpret_cast<const bf16_t*>(a.dO) + (b * S) * a.q_rs + h * FD;
  const bf16_t* K = reinterpret_cast<const bf16_t*>(a.k) + bh * S * FD;
  const bf16_t* V = reinterpret_cast<const bf16_t*>(a.v) + bh * S * FD;
  bf16x8 kf[8], vf[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    kf[c] = *reinterpret_cast<const bf16x8*>(K + krc * FD + 16 * c + 8 * lh);
    vf[c] = *reinterpret_cast<const bf16x8*>(V + krc * FD + 16 * c + 8 * lh);
  }
  const float c2 = kBwdScale * kLog2eF;
  f32x16 dkt[4], dvt[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) dkt[t] = dvt[t] = f32x16{};
  const int64_t qlast = S - 1;
  auto stats = [&](int bb, int64_t q0) {   // per-query lse (base 2) and D of the block
    if (tid < FK) {
      const int64_t q = q0 + tid;
      lsS[bb][tid] = q < S ? a.lse[bh * S + q] * kLog2eF : 0.f;
      dsS[bb][tid] = q < S ? a.D[bh * S + q] : 0.f;
    }
  };
  load_kv(Qs, Qg, a.q_rs, kbase, qlast, wv, lane);
  load_kv(Os, Og, a.q_rs, kbase, qlast, wv, lane);
  stats(0, kbase);
  int buf = 0;
  for (int64_t q0 = kbase; q0 <= qlast; q0 += FK, buf ^= 1) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    asm volatile("" ::: "memory");
    if (q0 + FK <= qlast) {
      load_kv(Qs + (buf ^ 1) * TS, Qg, a.q_rs, q0 + FK, qlast, wv, lane);
      load_kv(Os + (buf ^ 1) * TS, Og, a.q_rs, q0 + FK, qlast, wv, lane);
      stats(buf ^ 1, q0 + FK);
    }
    // A wave whose keys all follow the block's queries (the first block, for
    // waves 2 and 3) still runs it, fully masked: a uniform loop body keeps
    // the dK and dV accumulators in place across iterations.
    const bf16_t* qs = Qs + buf * TS;
    const bf16_t* os = Os + buf * TS;
    // Only a block that crosses this wave's diagonal or holds queries past S
    // is masked (a select, not a branch): there a query counts when its
    // offset in the block, less 4 lh, lies in [lo, hi).
    const bool edge = q0 < kw + 31 || q0 + FK > S;
    const int lo = int(kr - q0) - 4 * lh, hi = int(S - q0) - 4 * lh;
    // The block's 64 queries in two halves of 32 (qt), each: S and dP tiles
    // (element e is query q0 + 32 qt + 8 (e/4) + 4 lh + e%4 against key kr),
    // P and dS, then their share of dV^T and dK^T.  LDS fragments are read
    // two steps ahead; each step is one scheduling region whose MFMAs take
    // fragments read two regions earlier.
#pragma unroll
    for (int qt = 0; qt < 2; ++qt) {
      f32x16 sc = f32x16{}, dp = f32x16{};
      bf16x8 fa[3][2];   // [step % 3][Q, dO] for dim step c
      auto rda = [&](int c) {
        fa[c % 3][0] = *reinterpret_cast<const bf16x8*>(qs + tile_at(32 * qt + lq, 16 * c + 8 * lh));
        fa[c % 3][1] = *reinterpret_cast<const bf16x8*>(os + tile_at(32 * qt + lq, 16 * c + 8 * lh));
      };
      f32x4 ls[4], ds[4];   // log-sum-exp (base 2) and D of the lane's 16 queries
      rda(0);
      rda(1);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        ls[j] = *reinterpret_cast<const f32x4*>(&lsS[buf][32 * qt + 8 * j + 4 * lh]);
        ds[j] = *reinterpret_cast<const f32x4*>(&dsS[buf][32 * qt + 8 * j + 4 * lh]);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        if (c + 2 < 8) rda(c + 2);
        sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[c % 3][0], kf[c], sc, 0, 0, 0);
        dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[c % 3][1], vf[c], dp, 0, 0, 0);
        if (c + 2 < 8) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      // dV and dK: step t takes query step u = t / 4 of the half and dim
      // tile dt = t % 4; its dO^T and Q^T fragments are read ahead
      bf16x8 fc[3][2];   // [step % 3][dO^T, Q^T]
      auto rdc = [&](int t) {
        const int sq = 2 * qt + (t >> 2), dt = t & 3;
        fc[t % 3][0] = tile_t_frag(os, sq, dt, lane);
        fc[t % 3][1] = tile_t_frag(qs, sq, dt, lane);
      };
      rdc(0);
      rdc(1);
      // P and dS
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int e = 4 * j + i, cq = 32 * qt + 8 * j + i;
          float pv = __builtin_amdgcn_exp2f(fmaf(sc[e], c2, -ls[j][i]));
          if (edge) pv = cq >= lo && cq < hi ? pv : 0.f;
          sc[e] = pv;                            // P
          dp[e] = pv * (dp[e] - ds[j][i]);       // dS
        }
      const bf16x8 pb[2] = {c_to_b1(sc, 0), c_to_b1(sc, 1)};
      const bf16x8 dsb[2] = {c_to_b1(dp, 0), c_to_b1(dp, 1)};
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        if (t + 2 < 8) rdc(t + 2);
        const int u = t >> 2, dt = t & 3;
        dvt[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fc[t % 3][0], pb[u], dvt[dt], 0, 0, 0);
        dkt[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fc[t % 3][1], dsb[u], dkt[dt], 0, 0, 0);
        if (t + 2 < 8) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  if (kr < S) {
    bf16_t* dK = reinterpret_cast<bf16_t*>(a.dk) + bh * S * FD;
    bf16_t* dV = reinterpret_cast<bf16_t*>(a.dv) + bh * S * FD;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int dim = 32 * dt + 8 * (e >> 2) + 4 * lh + (e & 3);
        dK[kr * FD + dim] = f2bf(dkt[dt][e] * kBwdScale);
        dV[kr * FD + dim] = f2bf(dvt[dt][e]);
      }
  }
}

}  // namespace

hipError_t launch_attention_bwd_d128(const AttnBwdArgs& a, hipStream_t s) {
  const int64_t nb = (a.S + FQ - 1) / FQ;
  hipLaunchKernelGGL(attn_bwd_dkv_d128, dim3(unsigned(a.B * a.nH * nb)), dim3(64 * FW), kFlashLds, s, a, nb);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attn_bwd_dq_d128, dim3(unsigned(a.B * a.nH * nb)), dim3(64 * FW), kFlashLds, s, a, nb);
  return hipGetLastError();
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  const int64_t rows = a.B * a.nH * a.S;
  if (a.bf16 && a.d == 128 && a.S <= 16 && !a.lse) {
    hipLaunchKernelGGL(attn_decode_d128, dim3(unsigned(rows)), dim3(64 * kDecWaves), 0, s, a);
    return hipGetLastError();
  }
  if (a.bf16 && a.d == 128) {
    const int64_t nqb = (a.S + FQ - 1) / FQ;
    hipLaunchKernelGGL(attn_prefill_d128, dim3(unsigned(a.B * a.nH * nqb)), dim3(64 * FW), kFlashLds, s, a, nqb);
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
