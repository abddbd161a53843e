// Decode-shaped GEMM (M <= 16 token rows) on bf16 matrix cores.
//
// Y[m, n] = sum_k A[m, k] W[n, k] is HBM-bound on W (16 flop per weight
// byte).  The 16 token rows fill the M side of v_mfma_f32_16x16x32_bf16 and
// 16 weight rows its N side, so every weight byte is read once from HBM.
//
// Routed rows (MoE experts): the same kernel over the rows of a routed-row
// list, gathered by token on input or scattered by token on output.
//
// Grouped products (the query, key and value projections): up to three
// weights of the same shape against one A in one grid, group-major, so the
// launch and its ramp are paid once for all three.
//
// Work split: one 1024-thread workgroup per 16 output features; its sixteen
// waves take interleaved 64-wide K chunks (adjacent waves read adjacent 128 B
// of every row), two chunks in flight per wave, keep fp32 partial tiles in
// registers and reduce them through LDS in a fixed order (deterministic);
// four waves then write one output each per lane.
//
// Loads: the MFMA operand layout gives each row only four lanes (64 B) per
// load instruction, which spends a cache-line request on half a line.  Each
// load instead covers 8 rows x 128 B (lane L: row L / 8, 16-B piece L % 8),
// and the chunk passes through a wave-private LDS tile (16 rows x 128 B) to
// reach the operand layout: lane (r, g) = (l % 16, l / 16) then takes
// A[r, 64c + 32h + 8g .. +8] and W[n0 + r, same k] for half h of chunk c.
// Piece q of row r sits at slot q ^ (r >> 1) of the row, so the 16-lane
// groups of both the stores and the fragment reads hit 16 distinct banks.
#include <hip/hip_runtime.h>

#include "common.h"
#include "gemm.h"

namespace auvm {

using namespace dev;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kUnroll = 2;  // 64-k chunks in flight per wave
constexpr int kWaves = 16;  // waves per workgroup, splitting K

// 16-B slot of piece q (0..7) of row r (0..15) in a chunk tile
__device__ __forceinline__ int tslot(int r, int q) { return 8 * r + (q ^ (r >> 1)); }

// weights and outputs of up to three grouped products (one when ungrouped)
struct Group {
  const bf16_t* w0;
  const bf16_t* w1;
  const bf16_t* w2;
  void* c0;
  void* c1;
  void* c2;
};

// LIST: rows come from a routed-row list (GemmArgs::list): the row count is
// read from the list, and A rows are gathered by token (EPI_SWIGLU) or the
// results scattered into token rows with the routing weight (EPI_MOE).
template <int EPI, class TC, bool LIST>
__global__ void __launch_bounds__(64 * kWaves) gemv_mfma(const bf16_t* __restrict__ A, Group grp,
                                                 const bf16_t* __restrict__ W2, int M, int64_t N, int64_t K,
                                                 const int32_t* __restrict__ list, const float* __restrict__ rw,
                                                 int topk) {
  constexpr bool DUAL = EPI == EPI_SWIGLU;
  constexpr int kParts = DUAL ? 3 : 2;   // A, W (, W2) tiles of a chunk
  __shared__ bf16x8 tile[kWaves][kParts][128];
  __shared__ f32x4 part[kWaves][DUAL ? 2 : 1][64];
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // uniform: scalar chunk loop
  const int r = lane & 15, g = lane >> 4;      // fragment row, k group
  const int fr = lane >> 3, fp = lane & 7;     // load row (within 8), piece
  // group of this workgroup (uniform; selects, so the choice stays scalar)
  const int64_t nb = (N + 15) / 16, bx = blockIdx.x;
  const int gi = bx >= 2 * nb ? 2 : bx >= nb ? 1 : 0;
  const bf16_t* __restrict__ W = gi == 0 ? grp.w0 : gi == 1 ? grp.w1 : grp.w2;
  TC* __restrict__ C = static_cast<TC*>(gi == 0 ? grp.c0 : gi == 1 ? grp.c1 : grp.c2);
  const int64_t n0 = (bx - gi * nb) * 16;
  int rows = M;
  if constexpr (LIST) rows = list[0] < M ? list[0] : M;
  // source rows of this lane's two loads: rows fr and 8 + fr of the tile;
  // rows past the end are clamped, their results dropped
  const bf16_t* ap[2];
  const bf16_t* wp[2];
  const bf16_t* w2p[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int rr = 8 * h + fr;
    int64_t ar = rr < rows ? rr : 0;
    if constexpr (LIST && EPI != EPI_MOE) {
      if (rr < rows) {
        const int64_t t = list[1 + rr] / topk;
        ar = t < 0 ? 0 : (t < M ? t : M - 1);
      }
    }
    ap[h] = A + ar * K;
    const int64_t wn = n0 + rr < N ? n0 + rr : N - 1;
    wp[h] = W + wn * K;
    w2p[h] = DUAL ? W2 + wn * K : nullptr;
  }
  const int64_t nch = (K + 63) / 64;   // K % 32 == 0: the last chunk may hold one half
  bf16x8* my = &tile[wv][0][0];
  f32x4 acc = {0.f, 0.f, 0.f, 0.f}, acc2 = {0.f, 0.f, 0.f, 0.f};
  for (int64_t c0 = wv; c0 < nch; c0 += kWaves * kUnroll) {
    bf16x8 av[kUnroll][2], wt[kUnroll][2], w2t[DUAL ? kUnroll : 1][2];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t c = c0 + kWaves * u < nch ? c0 + kWaves * u : nch - 1;   // loads stay in bounds
      const int pc = 64 * c + 64 > K ? (fp & 3) : fp;                         // half chunk: first half only
      const int64_t off = 64 * c + 8 * pc;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        av[u][h] = *reinterpret_cast<const bf16x8*>(ap[h] + off);
        // weights are read once: non-temporal, so they do not displace the activations in L2
        wt[u][h] = __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(wp[h] + off));
        if constexpr (DUAL) w2t[u][h] = __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(w2p[h] + off));
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t c = c0 + kWaves * u;
      if (c >= nch) break;   // uniform over the wave
      // the wave's own tile: stores, then reads, in order on the LDS queue
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int sl = tslot(8 * h + fr, fp);
        my[sl] = av[u][h];
        my[128 + sl] = wt[u][h];
        if constexpr (DUAL) my[256 + sl] = w2t[u][h];
      }
      const int halves = 64 * c + 64 > K ? 1 : 2;
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        if (hh >= halves) break;
        const int sl = tslot(r, 4 * hh + g);
        const bf16x8 a = my[sl];
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, my[128 + sl], acc, 0, 0, 0);
        if constexpr (DUAL) acc2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, my[256 + sl], acc2, 0, 0, 0);
      }
    }
  }
  part[wv][0][lane] = acc;
  if constexpr (DUAL) part[wv][1][lane] = acc2;
  __syncthreads();
  // Waves 0..3 finish element i = wv of every lane's tile, the partials summed
  // in wave order: one output per lane, so a read-modify-write epilogue waits
  // for memory once.  Accumulator layout: element i of lane l is row
  // 4*(l/16)+i, column l%16.
  if (wv >= 4) return;
  const int i = wv;
  float v = part[0][0][lane][i], v2 = 0.f;
  if constexpr (DUAL) v2 = part[0][1][lane][i];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) {
    v += part[w][0][lane][i];
    if constexpr (DUAL) v2 += part[w][1][lane][i];
  }
  const int64_t col = n0 + (lane & 15);
  const int row = 4 * (lane >> 4) + i;
  if (col >= N || row >= rows) return;
  if constexpr (EPI == EPI_GELU) v = gelu_erf(v);
  if constexpr (EPI == EPI_SWIGLU) v = silu(v) * v2;
  if constexpr (EPI == EPI_MOE) {
    const int64_t j = list[1 + row], lim = int64_t(M) * topk;
    const int64_t jc = j < 0 ? 0 : (j < lim ? j : lim - 1);
    float* x = reinterpret_cast<float*>(C);
    x[(jc / topk) * N + col] += rw[jc] * v;
  } else if constexpr (EPI == EPI_RESID) {
    float* x = reinterpret_cast<float*>(C);
    x[int64_t(row) * N + col] += v;
  } else {
    st(C, int64_t(row) * N + col, v);
  }
}

template <int EPI, class TC, bool LIST = false>
hipError_t go(const GemmArgs& g, hipStream_t s) {
  const bool grouped = g.groups > 1;
  if (grouped && (EPI != EPI_STORE || LIST || g.groups > 3)) return hipErrorInvalidValue;
  const int ng = grouped ? g.groups : 1;
  Group grp;
  const uint8_t* w[3] = {g.w, g.w, g.w};
  uint8_t* c[3] = {g.c, g.c, g.c};
  for (int i = 0; grouped && i < 3; ++i) {   // unused groups repeat the last one; no block reaches them
    w[i] = g.gw[i < ng ? i : ng - 1];
    c[i] = g.gc[i < ng ? i : ng - 1];
  }
  grp.w0 = reinterpret_cast<const bf16_t*>(w[0]);
  grp.w1 = reinterpret_cast<const bf16_t*>(w[1]);
  grp.w2 = reinterpret_cast<const bf16_t*>(w[2]);
  grp.c0 = c[0];
  grp.c1 = c[1];
  grp.c2 = c[2];
  dim3 grid(unsigned(ng * ((g.N + 15) / 16)));
  hipLaunchKernelGGL((gemv_mfma<EPI, TC, LIST>), grid, dim3(64 * kWaves), 0, s, reinterpret_cast<const bf16_t*>(g.a),
                     grp, reinterpret_cast<const bf16_t*>(g.w2), int(g.M), g.N, g.K, g.list, g.rw, g.topk);
  return hipGetLastError();
}

template <class TC>
hipError_t by_epi(const GemmArgs& g, hipStream_t s) {
  if (g.list) {
    if (g.epi == EPI_SWIGLU) return go<EPI_SWIGLU, TC, true>(g, s);
    if (g.epi == EPI_MOE) return go<EPI_MOE, float, true>(g, s);
    return hipErrorInvalidValue;
  }
  switch (g.epi) {
    case EPI_STORE: return go<EPI_STORE, TC>(g, s);
    case EPI_GELU: return go<EPI_GELU, TC>(g, s);
    case EPI_RESID: return go<EPI_RESID, float>(g, s);
    case EPI_SWIGLU: return go<EPI_SWIGLU, TC>(g, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

// bf16 operands, M <= 16, K % 32 == 0 (checked when the kernel was added).
hipError_t launch_gemv_bf16(const GemmArgs& g, hipStream_t s) {
  return g.out_bf16 ? by_epi<bf16_t>(g, s) : by_epi<float>(g, s);
}

}  // namespace auvm
