// The context behind the C interface.
#pragma once

#include <memory>
#include <string>
#include <vector>

#include "core.h"

namespace auvm {

class Executor;  // executor.cpp (HIP runtime)
struct ExecDeleter {
  void operator()(Executor* e) const;  // defined next to the executor
};
using ExecPtr = std::unique_ptr<Executor, ExecDeleter>;

struct Ctx {
  int device = -1;                 // < 0: plan-only
  std::string err;
  // arena and registry.  Arena offsets below pinned_bytes live in pinned
  // memory at host; the rest (a tiered arena) in pageable memory at
  // host_pageable, fetched through a pinned staging ring.
  uint64_t arena_bytes = 0, pinned_bytes = 0;
  uint8_t* host = nullptr;
  uint8_t* host_pageable = nullptr;
  bool host_owned = false;
  bool arena_set = false;
  std::vector<uint8_t*> stage;     // staging ring: kStageSlots pinned buffers of kStageBytes
  uint8_t* host_at(uint64_t off) const { return off < pinned_bytes ? host + off : host_pageable + (off - pinned_bytes); }
  bool pageable(const Tensor& t) const { return t.arena_off >= pinned_bytes; }
  std::vector<Tensor> tensors;
  std::vector<Kernel> kernels;
  // budget and policy
  uint64_t M = 0;
  uint8_t* pool = nullptr;
  bool pool_owned = false;
  bool budget_set = false;
  Roofs roofs;
  auvm_policy pol{AUVM_T_A_P, 0, 1, AUVM_PLACE_POOL, 0, 0, 4, 32, 0};
  // plan and execution
  bool planned = false;
  PlanResult plan;
  uint64_t plan_ns = 0, run_ns = 0;
  ExecPtr exec;

  ~Ctx();
};

// Executor interface used by the C entry points (executor.cpp).
ExecPtr make_executor(Ctx& c);
auvm_status exec_bind_streams(Ctx& c, void* compute, void* h2d, void* d2h);
auvm_status exec_run(Ctx& c, uint32_t first_k, uint32_t n_k);
auvm_status exec_run_noalloc(Ctx& c, uint32_t first_k, uint32_t n_k);
auvm_status exec_reset(Ctx& c);
auvm_status exec_read(Ctx& c, int32_t id, void* dst, uint64_t bytes);
const std::vector<auvm_sched_entry>& exec_log(const Ctx& c);
uint64_t exec_kernels_run(const Ctx& c);
uint64_t exec_stall_ns(const Ctx& c);
auvm_status exec_kernel_times(const Ctx& c, float* dur, float* gap, uint64_t cap, uint64_t* n);
const std::vector<auvm_timeline_entry>& exec_timeline(const Ctx& c);
auvm_status host_alloc_pinned(Ctx& c, uint64_t bytes);
// the pageable tier (arena_bytes - pinned_bytes) and the staging ring
auvm_status host_alloc_pageable(Ctx& c);
constexpr int kStageSlots = 4;
constexpr uint64_t kStageBytes = uint64_t(64) << 20;
auvm_status device_alloc_pool(Ctx& c, uint64_t bytes);
void free_owned(Ctx& c);
void release_pool(Ctx& c);   // frees an owned pool, forgets a borrowed one

}  // namespace auvm
