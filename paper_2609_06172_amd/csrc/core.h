// Internal data model of the runtime: tensor registry, kernel trace, planner
// result.  Host-only; no HIP types here.
#pragma once

#include <cstdint>
#include <string>
#include <utility>
#include <vector>

#include "autouvm.h"

namespace auvm {

constexpr uint64_t kAlign = 256;
constexpr int64_t kInf = int64_t(1) << 62;

inline uint64_t align_up(uint64_t n) { return (n + kAlign - 1) / kAlign * kAlign; }
inline uint32_t dtype_size(uint32_t dt) {
  return dt == AUVM_F32 ? 4 : dt == AUVM_BF16 ? 2 : dt == AUVM_I32 ? 4 : 1;
}

struct Tensor {
  uint64_t arena_off = 0;
  uint64_t bytes = 0;   // registered size
  uint64_t size = 0;    // 256-aligned size (what occupies the pool)
  uint32_t dtype = 0, kind = 0, flags = 0;
  bool host_valid0() const { return kind == AUVM_PARAM || (flags & AUVM_HOST_INIT); }
};

struct Kernel {
  uint32_t op = 0;
  int64_t shape[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  std::vector<int32_t> ids;                      // positional operands
  std::vector<uint8_t> modes;
  std::vector<std::pair<int32_t, uint8_t>> acc;  // distinct ids, first-occurrence order, OR-ed modes
  uint64_t flops = 0, hbm = 0;                   // resolved costs
  uint64_t time_ns = 0;                          // measured time (0: classify analytically)
  uint32_t layer = 0;
};

struct Roofs {
  uint64_t P = 2500000000000000ull;  // flop/s
  uint64_t Bh = 8000000000000ull;    // HBM byte/s
  uint64_t Bl = 64000000000ull;      // host-link byte/s
};

struct PlanCounters {
  uint64_t h2d_prefetch_n = 0, h2d_prefetch_B = 0, h2d_demand_n = 0, h2d_demand_B = 0;
  uint64_t d2h_wb_n = 0, d2h_wb_B = 0, drop_n = 0, alloc_n = 0;
  uint64_t useless_prefetch_n = 0, useless_prefetch_B = 0;
  uint64_t class_n[3] = {0, 0, 0};
};

struct PlanResult {
  std::vector<auvm_sched_entry> schedule;
  std::vector<auvm_residency> residency;
  std::vector<uint8_t> static_cls, dyn_cls;
  PlanCounters counters;
};

struct PlanError {
  auvm_status code;
  std::string msg;
};

// Analytic flops and algorithmic HBM bytes of a kernel (cost.cpp).
void kernel_cost(const Kernel& k, const std::vector<Tensor>& tensors, uint64_t* F, uint64_t* B);
// Operand count / dtype / size validation of a kernel against its shape
// (cost.cpp).  Returns an empty string when the kernel is well formed.
std::string validate_kernel(const Kernel& k, const std::vector<Tensor>& tensors);
// Roofline class of a kernel with X host-resident read bytes; with a measured
// kernel time t_ns > 0 the CGI test compares the link time X/Bl with it.
uint8_t classify(uint64_t F, uint64_t B, uint64_t X, const Roofs& r, uint64_t t_ns = 0);

// The policy (planner.cpp).  Throws PlanError.
PlanResult plan(const std::vector<Tensor>& tensors, const std::vector<Kernel>& kernels,
                uint64_t M, const Roofs& roofs, const auvm_policy& pol);

}  // namespace auvm
