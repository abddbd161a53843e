// Large prefill GEMM on bf16 matrix cores: C[M,N] (epilogue) = A[M,K] W[N,K]^T.
//
// Workgroup tile 256 x 256 (256 x 128 per weight for the two-weight SwiGLU
// epilogue), K step 64, eight waves in a 2 x 4 grid (two per SIMD, which hide
// each other's LDS and barrier waits); each wave owns 4 x 2 (4 x 1 per weight)
// tiles of v_mfma_f32_32x32x16_bf16.  Within a K step the fragments of the
// next 16-wide sub-step are read from LDS while the current sub-step's MFMAs
// run, interleaved by scheduling barriers.
//
// Operand tiles go from global memory straight into LDS (16-byte
// global_load_lds, no register staging), two stages deep: the next K step
// streams in while the current one feeds the matrix cores.  One wave
// instruction fills 8 rows x 128 bytes of a stage; within a row the eight
// 16-byte chunks are stored at slot chunk ^ ((row >> 1) & 7), which keeps a
// fragment read (32 rows, one chunk) free of LDS bank conflicts.  Rows past M or N are
// clamped to the last row (every load stays in bounds) and their results are
// dropped by the epilogue; K must be a multiple of 64.  The same kernel runs
// the routed rows of an MoE expert from a routed-row list.
#include <hip/hip_runtime.h>

#include "common.h"
#include "gemm.h"

namespace auvm {

using namespace dev;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kBK = 64;      // K elements per stage row (128 bytes)
constexpr int kXcd = 8;
constexpr int kGroupM = 8;

// LDS slot of a 16-byte chunk: chunk ^ swz(row).  A fragment read takes one
// chunk of 32 consecutive rows, served 16 rows at a time over 256 bytes of
// banks (two 128-byte rows); (row >> 1) & 7 gives 16 consecutive rows 16
// distinct (row parity, slot) pairs, so the read is free of bank conflicts.
__device__ __forceinline__ int swz(int row) { return (row >> 1) & 7; }

constexpr int kWaves = 8, kWN = 4;   // 2 x 4 waves

template <int EPI>
struct Shape {
  static constexpr bool kDual = EPI == EPI_SWIGLU;
  static constexpr int kTM = 4, kTN = kDual ? 1 : 2;          // 32x32 tiles per wave (per weight)
  static constexpr int kBM = 2 * 32 * kTM, kBN = kWN * 32 * kTN;
  static constexpr int kRows = kBM + (kDual ? 2 : 1) * kBN;   // rows staged per K step
  static constexpr int kStage = kRows * kBK;                   // bf16 elements per stage
};

// One K step of operand rows into LDS stage buf.  Wave wv fills the 8-row
// blocks wv, wv + 8, ...; lane l fills row 8 * block + l / 8 at slot l % 8
// with the row's chunk (l % 8) ^ swz(row).  The lane's A rows (blocks t <
// kARowsPerLane) come precomputed in arow.  A device function, not a lambda:
// the LDS-load builtin exists only in the device pass.
constexpr int kARowsPerLane = 256 / (8 * kWaves);

template <int EPI>
__device__ __forceinline__ void load_stage(bf16_t* smem, const bf16_t* const* arow, const bf16_t* __restrict__ W,
                                           const bf16_t* __restrict__ W2, int64_t N, int64_t K, int64_t n0,
                                           int wv, int lane, int buf, int64_t k0) {
  using S = Shape<EPI>;
  constexpr bool DUAL = S::kDual;
  constexpr int BM = S::kBM, BN = S::kBN;
  static_assert(S::kRows % (8 * kWaves) == 0, "stage rows split evenly over the waves");
  static_assert(BM == 8 * kWaves * kARowsPerLane, "A rows are the first blocks of a stage");
  bf16_t* base = smem + buf * S::kStage;
  const int rin = lane >> 3, slot = lane & 7;
#pragma unroll
  for (int t = 0; t < S::kRows / (8 * kWaves); ++t) {
    const int b = wv + kWaves * t;
    const int row = 8 * b + rin;
    const bf16_t* src;
    if (t < kARowsPerLane) {
      src = arow[t];
    } else {
      const int wrow = row - BM;
      const bool second = DUAL && wrow >= BN;
      const int64_t r = n0 + (second ? wrow - BN : wrow);
      src = (second ? W2 : W) + (r < N ? r : N - 1) * K;
    }
    const int chunk = slot ^ swz(row);
    __builtin_amdgcn_global_load_lds(src + k0 + 8 * chunk, base + 8 * b * kBK, 16, 0, 0);
  }
}

// LIST: rows come from a routed-row list (GemmArgs::list): tiles past the
// list's count exit at once, A rows are gathered by token (EPI_SWIGLU) or the
// results scattered into token rows with the routing weight (EPI_MOE).
template <int EPI, class TC, bool LIST>
__global__ void __launch_bounds__(64 * kWaves) gemm_big(const bf16_t* __restrict__ A, const bf16_t* __restrict__ W,
                                                const bf16_t* __restrict__ W2, TC* __restrict__ C,
                                                int64_t M, int64_t N, int64_t K, int tilesN,
                                                const int32_t* __restrict__ list, const float* __restrict__ rw,
                                                int topk) {
  using S = Shape<EPI>;
  constexpr bool DUAL = S::kDual;
  constexpr int TM = S::kTM, TN = S::kTN, BM = S::kBM, BN = S::kBN;
  extern __shared__ __align__(16) bf16_t smem[];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int wm = wv / kWN, wn = wv % kWN;

  // Tile order: XCD round-robin remap, then groups of kGroupM row-blocks.
  // Under a routed-row list only the first ceil(count / BM) row-blocks hold
  // rows: the blocks past them exit, and the live ones are remapped among
  // themselves, so that they still spread over all XCDs.
  int nwg = gridDim.x;
  int64_t rows = M;
  if constexpr (LIST) {
    rows = list[0] < M ? list[0] : M;
    const int live = rows > 0 ? int((rows + BM - 1) / BM) * tilesN : 0;
    if (int(blockIdx.x) >= live) return;   // uniform over the workgroup
    nwg = live;
  }
  const int per = nwg / kXcd;
  int id = blockIdx.x;
  if (per > 0 && id < per * kXcd) id = (id % kXcd) * per + id / kXcd;
  const int tilesM = nwg / tilesN;
  const int gsize = kGroupM * tilesN, grp = id / gsize, first = grp * kGroupM;
  const int gm = (tilesM - first) < kGroupM ? (tilesM - first) : kGroupM;
  const int in = id - grp * gsize;
  const int64_t m0 = int64_t(first + in % gm) * BM, n0 = int64_t(in / gm) * BN;
  const bf16_t* arow[kARowsPerLane];
#pragma unroll
  for (int t = 0; t < kARowsPerLane; ++t) {
    const int64_t r = m0 + 8 * (wv + kWaves * t) + (lane >> 3);
    int64_t src = r < rows ? r : rows - 1;   // rows past the end are clamped, their results dropped
    if constexpr (LIST && EPI != EPI_MOE) {
      const int64_t tok = list[1 + src] / topk;
      src = tok < 0 ? 0 : (tok < M ? tok : M - 1);
    }
    arow[t] = A + src * K;
  }

  f32x16 acc[TM][TN], acc2[DUAL ? TM : 1][DUAL ? TN : 1];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x16{};
  if constexpr (DUAL) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc2[i][j] = f32x16{};
  }

  const int lr = lane & 31, lc = lane >> 5;     // fragment row, chunk half
  const int64_t nk = K / kBK;
  load_stage<EPI>(smem, arow, W, W2, N, K, n0, wv, lane, 0, 0);
  for (int64_t kt = 0; kt < nk; ++kt) {
    __builtin_amdgcn_s_waitcnt(0);   // this wave's loads of stage kt have landed
    __syncthreads();                 // ... and every other wave's; stage kt-1 is free
    asm volatile("" ::: "memory");   // LDS now holds data written outside the compiler's view
    const bf16_t* stg = smem + int(kt & 1) * S::kStage;
    // fragments of sub-step ks into register set q
    bf16x8 a[2][TM], b[2][TN], b2[2][DUAL ? TN : 1];
    auto frag = [&](int ks, int q) {
      const int c = 2 * ks + lc;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int row = wm * 32 * TM + 32 * i + lr;
        a[q][i] = *reinterpret_cast<const bf16x8*>(stg + row * kBK + 8 * (c ^ swz(row)));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int row = BM + wn * 32 * TN + 32 * j + lr;
        b[q][j] = *reinterpret_cast<const bf16x8*>(stg + row * kBK + 8 * (c ^ swz(row)));
        if constexpr (DUAL) {
          const int row2 = row + BN;
          b2[q][j] = *reinterpret_cast<const bf16x8*>(stg + row2 * kBK + 8 * (c ^ swz(row2)));
        }
      }
    };
    // Sub-step ks is one scheduling region (fenced by sched_barrier): its first
    // MFMA, whose fragments were read during sub-step ks-1, then the reads of
    // sub-step ks+1 alternating with its other MFMAs.  The compiler waits for
    // every outstanding LDS read before a region's first MFMA, so reads
    // issued at the top of a region, before that MFMA, would stall it; issued
    // after it, they have the rest of the region to land.  Stage kt+1's
    // global loads go out right after sub-step 0's reads.
    frag(0, 0);
    if (kt + 1 < nk) load_stage<EPI>(smem, arow, W, W2, N, K, n0, wv, lane, int((kt + 1) & 1), (kt + 1) * kBK);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      const int q = ks & 1;
      if (ks + 1 < kBK / 16) frag(ks + 1, q ^ 1);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[q][i], b[q][j], acc[i][j], 0, 0, 0);
          if constexpr (DUAL) acc2[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[q][i], b2[q][j], acc2[i][j], 0, 0, 0);
        }
      if (ks + 1 < kBK / 16) {
        constexpr int kReads = TM + TN * (DUAL ? 2 : 1), kMfma = TM * TN * (DUAL ? 2 : 1);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
#pragma unroll
        for (int t = 0; t < kReads; ++t) {
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, kMfma - 1 - kReads, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // accumulator layout: element e of lane l is row 8*(e/4) + 4*(l/32) + e%4, column l%32.
  // Unrolled in full whatever the epilogue's size: a loop left rolled would
  // index the accumulators at run time and move them to scratch memory.
#pragma clang loop unroll(full)
  for (int i = 0; i < TM; ++i)
#pragma clang loop unroll(full)
    for (int j = 0; j < TN; ++j) {
      const int64_t col = n0 + wn * 32 * TN + 32 * j + lr;
      if (col >= N) continue;
      const int64_t r0 = m0 + wm * 32 * TM + 32 * i;   // first row of the 32-row tile
      if constexpr (EPI == EPI_RESID || EPI == EPI_MOE) {
        // Read-modify-write of fp32 rows.  A tile whose 32 rows all exist
        // takes straight-line code: every load, then every store, so the lane
        // waits for memory once per tile rather than once per element (the
        // compiler does not move a load past a store to the same array).
        float* x = reinterpret_cast<float*>(C);
        if (r0 + 32 <= rows) {
          int64_t at[16];
          float sc[16], xv[16];
#pragma clang loop unroll(full)
          for (int e = 0; e < 16; ++e) {
            const int64_t row = r0 + 8 * (e >> 2) + 4 * lc + (e & 3);
            if constexpr (EPI == EPI_MOE) {
              const int64_t jr = list[1 + row], lim = M * topk;
              const int64_t jc = jr < 0 ? 0 : (jr < lim ? jr : lim - 1);
              at[e] = (jc / topk) * N + col;
              sc[e] = rw[jc];
            } else {
              at[e] = row * N + col;
              sc[e] = 1.f;
            }
          }
#pragma clang loop unroll(full)
          for (int e = 0; e < 16; ++e) xv[e] = x[at[e]];
#pragma clang loop unroll(full)
          for (int e = 0; e < 16; ++e) {
            if constexpr (EPI == EPI_MOE)
              x[at[e]] = xv[e] + sc[e] * acc[i][j][e];
            else
              x[at[e]] = xv[e] + acc[i][j][e];
          }
          continue;
        }
      }
      if constexpr ((EPI == EPI_STORE || EPI == EPI_GELU || EPI == EPI_SWIGLU) && sizeof(TC) == 2) {
        // bf16 outputs of a full tile: each lane trades half of its 16
        // values with its neighbour (lane ^ 1, the next column), so that the
        // even lane of a pair holds column pairs for the rows of elements
        // 0..7 and the odd lane for those of 8..15; with N % 4 == 0 a second
        // trade with lane ^ 2 gives four columns, 8 bytes a store: a quarter
        // of the store instructions.
        const int64_t c0 = n0 + wn * 32 * TN + 32 * j;   // first column of the tile
        if (r0 + 32 <= rows && c0 + 32 <= N && (N & 1) == 0) {
          float v[16];
#pragma clang loop unroll(full)
          for (int e = 0; e < 16; ++e) {
            v[e] = acc[i][j][e];
            if constexpr (EPI == EPI_GELU) v[e] = gelu_erf(v[e]);
            if constexpr (EPI == EPI_SWIGLU) v[e] = silu(v[e]) * acc2[i][j][e];
          }
          const bool odd = lr & 1;
          uint32_t pk[8];   // column pair (2m, 2m+1) of the rows of element e (odd lane: e + 8)
#pragma clang loop unroll(full)
          for (int e = 0; e < 8; ++e) {
            const float send = odd ? v[e] : v[e + 8];
            // quad_perm [1, 0, 3, 2]: the value of lane ^ 1
            const float got = __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(send), 0xB1, 0xF, 0xF, false));
            const float lo = odd ? got : v[e], hi = odd ? v[e + 8] : got;
            pk[e] = uint32_t(f2bf(lo)) | (uint32_t(f2bf(hi)) << 16);
          }
          if ((N & 3) == 0) {
            // a second trade with lane ^ 2 (the next column pair): four
            // columns, 8 bytes a lane; the lower pair's lane keeps elements
            // 0..3 of its eight, the upper pair's lane elements 4..7
            const bool up = (lr >> 1) & 1;
            const int64_t c4 = col - (lr & 3);   // first of the four columns
#pragma clang loop unroll(full)
            for (int r = 0; r < 4; ++r) {
              const uint32_t send = up ? pk[r] : pk[r + 4];
              // quad_perm [2, 3, 0, 1]: the value of lane ^ 2
              const uint32_t got = uint32_t(__builtin_amdgcn_mov_dpp(int(send), 0x4E, 0xF, 0xF, false));
              const int i8 = up ? r + 4 : r, ee = odd ? i8 + 8 : i8;
              const int64_t row = r0 + 8 * (ee >> 2) + 4 * lc + (ee & 3);
              const uint2 w = up ? uint2{got, pk[r + 4]} : uint2{pk[r], got};
              *reinterpret_cast<uint2*>(reinterpret_cast<bf16_t*>(C) + row * N + c4) = w;
            }
          } else {
            const int64_t cp = col - (odd ? 1 : 0);   // the pair's even column
#pragma clang loop unroll(full)
            for (int e = 0; e < 8; ++e) {
              const int ee = odd ? e + 8 : e;
              const int64_t row = r0 + 8 * (ee >> 2) + 4 * lc + (ee & 3);
              *reinterpret_cast<uint32_t*>(reinterpret_cast<bf16_t*>(C) + row * N + cp) = pk[e];
            }
          }
          continue;
        }
      }
#pragma clang loop unroll(full)
      for (int e = 0; e < 16; ++e) {
        const int64_t row = r0 + 8 * (e >> 2) + 4 * lc + (e & 3);
        if (row >= rows) continue;
        float v = acc[i][j][e];
        if constexpr (EPI == EPI_GELU) v = gelu_erf(v);
        if constexpr (EPI == EPI_SWIGLU) v = silu(v) * acc2[i][j][e];
        if constexpr (EPI == EPI_MOE) {
          const int64_t jr = list[1 + row], lim = M * topk;
          const int64_t jc = jr < 0 ? 0 : (jr < lim ? jr : lim - 1);
          float* x = reinterpret_cast<float*>(C);
          x[(jc / topk) * N + col] += rw[jc] * v;
        } else if constexpr (EPI == EPI_RESID) {
          float* x = reinterpret_cast<float*>(C);
          x[row * N + col] += v;
        } else {
          st(C, row * N + col, v);
        }
      }
    }
}

template <int EPI, class TC, bool LIST = false>
hipError_t go(const GemmArgs& g, hipStream_t s) {
  using S = Shape<EPI>;
  const int tilesM = int((g.M + S::kBM - 1) / S::kBM), tilesN = int((g.N + S::kBN - 1) / S::kBN);
  const size_t lds = size_t(2) * S::kStage * sizeof(bf16_t);
  hipLaunchKernelGGL((gemm_big<EPI, TC, LIST>), dim3(unsigned(tilesM * tilesN)), dim3(64 * kWaves), lds, s,
                     reinterpret_cast<const bf16_t*>(g.a), reinterpret_cast<const bf16_t*>(g.w),
                     reinterpret_cast<const bf16_t*>(g.w2), reinterpret_cast<TC*>(g.c), g.M, g.N, g.K,
                     tilesN, g.list, g.rw, g.topk);
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

// bf16 operands, K % 64 == 0, M, N >= 1.
hipError_t launch_gemm_big_bf16(const GemmArgs& g, hipStream_t s) {
  if (g.K % kBK != 0 || g.M < 1 || g.N < 1) return hipErrorInvalidValue;
  return g.out_bf16 ? by_epi<bf16_t>(g, s) : by_epi<float>(g, s);
}

}  // namespace auvm
