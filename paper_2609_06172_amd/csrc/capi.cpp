// C entry points: argument checking, registry, trace construction, planning.
#include <chrono>
#include <cstring>
#include <new>

#include "ctx.h"

using namespace auvm;

struct auvm_ctx {
  Ctx c;
};

namespace {

auvm_status fail(auvm_ctx* x, auvm_status s, const std::string& m) {
  x->c.err = m;
  return s;
}

template <class T>
auvm_status copy_out(const std::vector<T>& v, T* buf, uint64_t cap, uint64_t* n, const auvm_ctx* x) {
  if (!n) return AUVM_E_INVAL;
  *n = v.size();
  if (!buf) return AUVM_OK;
  if (cap < v.size()) {
    const_cast<auvm_ctx*>(x)->c.err = "buffer holds fewer entries than available";
    return AUVM_E_RANGE;
  }
  if (!v.empty()) std::memcpy(buf, v.data(), v.size() * sizeof(T));
  return AUVM_OK;
}

}  // namespace

extern "C" {

auvm_status auvm_create(int hip_device, auvm_ctx** out) {
  if (!out) return AUVM_E_INVAL;
  *out = nullptr;
  auvm_ctx* x = new (std::nothrow) auvm_ctx();
  if (!x) return AUVM_E_NOMEM;
  x->c.device = hip_device < 0 ? -1 : hip_device;
  if (x->c.device >= 0) {
    x->c.exec = make_executor(x->c);
    if (!x->c.exec) {
      auvm_status s = AUVM_E_HIP;
      delete x;
      return s;
    }
  }
  *out = x;
  return AUVM_OK;
}

void auvm_destroy(auvm_ctx* x) { delete x; }

const char* auvm_last_error(const auvm_ctx* x) { return x ? x->c.err.c_str() : "null context"; }

auvm_status auvm_arena_init(auvm_ctx* x, uint64_t arena_bytes, void* host_pinned) {
  if (!x) return AUVM_E_INVAL;
  Ctx& c = x->c;
  if (c.arena_set) return fail(x, AUVM_E_STATE, "arena already initialised");
  if (arena_bytes == 0) return fail(x, AUVM_E_INVAL, "empty arena");
  c.arena_bytes = arena_bytes;
  c.pinned_bytes = arena_bytes;
  if (host_pinned) {
    c.host = static_cast<uint8_t*>(host_pinned);
  } else if (c.device >= 0) {
    auvm_status s = host_alloc_pinned(c, arena_bytes);
    if (s != AUVM_OK) return s;
  }
  c.arena_set = true;
  return AUVM_OK;
}

auvm_status auvm_arena_init_tiered(auvm_ctx* x, uint64_t arena_bytes, uint64_t pinned_bytes) {
  if (!x) return AUVM_E_INVAL;
  Ctx& c = x->c;
  if (c.arena_set) return fail(x, AUVM_E_STATE, "arena already initialised");
  if (arena_bytes == 0) return fail(x, AUVM_E_INVAL, "empty arena");
  if (pinned_bytes > arena_bytes || pinned_bytes % kAlign)
    return fail(x, AUVM_E_INVAL, "pinned_bytes must be a multiple of 256 no larger than the arena");
  c.arena_bytes = arena_bytes;
  c.pinned_bytes = pinned_bytes;
  if (c.device >= 0) {
    if (pinned_bytes) {
      auvm_status s = host_alloc_pinned(c, pinned_bytes);
      if (s != AUVM_OK) return s;
    }
    if (pinned_bytes < arena_bytes) {
      auvm_status s = host_alloc_pageable(c);
      if (s != AUVM_OK) return s;
    }
  }
  c.arena_set = true;
  return AUVM_OK;
}

auvm_status auvm_register_tensor(auvm_ctx* x, uint64_t arena_off, uint64_t bytes, uint32_t dtype,
                                 uint32_t kind, uint32_t flags, int32_t* out_id) {
  if (!x || !out_id) return AUVM_E_INVAL;
  Ctx& c = x->c;
  if (!c.arena_set) return fail(x, AUVM_E_STATE, "arena_init must come first");
  if (!c.kernels.empty()) return fail(x, AUVM_E_STATE, "tensors must be registered before kernels");
  if (dtype > AUVM_U8 || kind > AUVM_KV || (flags & ~uint32_t(AUVM_HOST_INIT | AUVM_LIVE_OUT)))
    return fail(x, AUVM_E_INVAL, "bad dtype, kind or flags");
  if (bytes == 0 || arena_off % kAlign) return fail(x, AUVM_E_INVAL, "zero size or unaligned offset");
  uint64_t sz = align_up(bytes);
  if (arena_off > c.arena_bytes || c.arena_bytes - arena_off < sz)
    return fail(x, AUVM_E_INVAL, "tensor window outside the arena");
  if (arena_off < c.pinned_bytes && arena_off + sz > c.pinned_bytes)
    return fail(x, AUVM_E_INVAL, "tensor window straddles the pinned and pageable tiers");
  if (arena_off >= c.pinned_bytes && kind != AUVM_PARAM)
    return fail(x, AUVM_E_INVAL, "only parameter tensors may live in the pageable tier");
  for (const Tensor& t : c.tensors)  // registration-order overlap check
    if (arena_off < t.arena_off + t.size && t.arena_off < arena_off + sz)
      return fail(x, AUVM_E_INVAL, "tensor windows overlap");
  Tensor t;
  t.arena_off = arena_off;
  t.bytes = bytes;
  t.size = sz;
  t.dtype = dtype;
  t.kind = kind;
  t.flags = flags;
  c.tensors.push_back(t);
  *out_id = int32_t(c.tensors.size() - 1);
  return AUVM_OK;
}

auvm_status auvm_tensor_host_ptr(auvm_ctx* x, int32_t id, void** out) {
  if (!x || !out) return AUVM_E_INVAL;
  Ctx& c = x->c;
  if (id < 0 || size_t(id) >= c.tensors.size()) return fail(x, AUVM_E_INVAL, "unknown tensor id");
  const Tensor& t = c.tensors[id];
  if (!(c.pageable(t) ? c.host_pageable : c.host)) return fail(x, AUVM_E_STATE, "no host arena in this context");
  *out = c.host_at(t.arena_off);
  return AUVM_OK;
}

auvm_status auvm_add_kernel(auvm_ctx* x, const auvm_kernel_desc* d, int32_t* out_k) {
  if (!x || !d || !out_k) return AUVM_E_INVAL;
  Ctx& c = x->c;
  if (c.planned) return fail(x, AUVM_E_STATE, "kernels cannot be added after plan");
  if (d->op >= AUVM_OP_COUNT) return fail(x, AUVM_E_INVAL, "unknown op");
  if (d->n == 0 || d->n > 16 || !d->ids || !d->modes) return fail(x, AUVM_E_INVAL, "bad operand list");
  Kernel k;
  k.op = d->op;
  std::memcpy(k.shape, d->shape, sizeof k.shape);
  k.layer = d->layer;
  for (uint32_t i = 0; i < d->n; ++i) {
    int32_t id = d->ids[i];
    if (id < 0 || size_t(id) >= c.tensors.size()) return fail(x, AUVM_E_INVAL, "unknown tensor id in kernel");
    if ((d->modes[i] & AUVM_W) && c.pageable(c.tensors[id]))
      return fail(x, AUVM_E_INVAL, "kernel writes tensor " + std::to_string(id) + ", which lives in the pageable tier");
    k.ids.push_back(id);
    k.modes.push_back(d->modes[i]);
    bool merged = false;
    for (auto& a : k.acc)
      if (a.first == id) {
        a.second |= d->modes[i];
        merged = true;
      }
    if (!merged) k.acc.push_back({id, d->modes[i]});
  }
  std::string v = validate_kernel(k, c.tensors);
  if (!v.empty()) return fail(x, AUVM_E_INVAL, "kernel " + std::to_string(c.kernels.size()) + ": " + v);
  uint64_t F, B;
  kernel_cost(k, c.tensors, &F, &B);
  k.flops = d->flops ? d->flops : F;
  k.hbm = d->hbm_bytes ? d->hbm_bytes : B;
  c.kernels.push_back(std::move(k));
  *out_k = int32_t(c.kernels.size() - 1);
  return AUVM_OK;
}

auvm_status auvm_set_budget(auvm_ctx* x, uint64_t device_bytes, void* device_pool) {
  if (!x) return AUVM_E_INVAL;
  Ctx& c = x->c;
  uint64_t M = device_bytes / kAlign * kAlign;
  if (M == 0) return fail(x, AUVM_E_INVAL, "budget below 256 bytes");
  if (c.budget_set) {
    // a new budget: wait for the old pool's work, forget residency and the plan
    if (c.exec) {
      auvm_status s = exec_reset(c);
      if (s != AUVM_OK) return s;
    }
    release_pool(c);
    c.planned = false;
    c.budget_set = false;
  }
  c.M = M;
  if (device_pool) {
    c.pool = static_cast<uint8_t*>(device_pool);
  } else if (c.device >= 0) {
    auvm_status s = device_alloc_pool(c, M);
    if (s != AUVM_OK) return s;
  }
  c.budget_set = true;
  return AUVM_OK;
}

auvm_status auvm_set_roofs(auvm_ctx* x, uint64_t P, uint64_t Bh, uint64_t Bl) {
  if (!x) return AUVM_E_INVAL;
  if (!P || !Bh || !Bl) return fail(x, AUVM_E_INVAL, "roofs must be positive");
  x->c.roofs = Roofs{P, Bh, Bl};
  return AUVM_OK;
}

auvm_status auvm_clear_kernels(auvm_ctx* x) {
  if (!x) return AUVM_E_INVAL;
  Ctx& c = x->c;
  if (c.exec) {
    auvm_status s = exec_reset(c);
    if (s != AUVM_OK) return s;
  }
  c.kernels.clear();
  c.plan = PlanResult{};
  c.planned = false;
  return AUVM_OK;
}

auvm_status auvm_set_kernel_times(auvm_ctx* x, const uint64_t* t_ns, uint64_t n) {
  if (!x) return AUVM_E_INVAL;
  Ctx& c = x->c;
  if (n != c.kernels.size()) return fail(x, AUVM_E_INVAL, "one time per kernel of the trace");
  if (n > 0 && !t_ns) return fail(x, AUVM_E_INVAL, "null times");
  for (uint64_t k = 0; k < n; ++k) c.kernels[k].time_ns = t_ns[k];
  c.planned = false;
  return AUVM_OK;
}

auvm_status auvm_set_policy(auvm_ctx* x, const auvm_policy* p) {
  if (!x || !p) return AUVM_E_INVAL;
  if (p->variant > AUVM_T_A_P || p->placement > AUVM_PLACE_IDEAL)
    return fail(x, AUVM_E_INVAL, "bad policy");
  x->c.pol = *p;
  const bool full = p->variant == AUVM_T_A_P;
  if (p->guard == AUVM_POLICY_DEFAULT) x->c.pol.guard = full ? 4 : 0;
  if (p->bucket == AUVM_POLICY_DEFAULT) x->c.pol.bucket = full ? 32 : 1;
  x->c.planned = false;
  return AUVM_OK;
}

auvm_status auvm_plan(auvm_ctx* x) {
  if (!x) return AUVM_E_INVAL;
  Ctx& c = x->c;
  if (!c.budget_set) return fail(x, AUVM_E_STATE, "set_budget must come before plan");
  if (c.kernels.empty()) return fail(x, AUVM_E_STATE, "no kernels");
  auto t0 = std::chrono::steady_clock::now();
  try {
    c.plan = auvm::plan(c.tensors, c.kernels, c.M, c.roofs, c.pol);
  } catch (const PlanError& e) {
    c.planned = false;
    return fail(x, e.code, e.msg);
  } catch (const std::bad_alloc&) {
    c.planned = false;
    return fail(x, AUVM_E_NOMEM, "out of host memory while planning");
  }
  c.plan_ns = uint64_t(std::chrono::duration_cast<std::chrono::nanoseconds>(
                           std::chrono::steady_clock::now() - t0).count());
  c.planned = true;
  if (c.exec) {
    auvm_status s = exec_reset(c);
    if (s != AUVM_OK) return s;
  }
  return AUVM_OK;
}

auvm_status auvm_bind_streams(auvm_ctx* x, void* compute, void* h2d, void* d2h) {
  if (!x) return AUVM_E_INVAL;
  if (!x->c.exec) return fail(x, AUVM_E_STATE, "plan-only context");
  return exec_bind_streams(x->c, compute, h2d, d2h);
}

auvm_status auvm_run(auvm_ctx* x, uint32_t first_k, uint32_t n_k) {
  if (!x) return AUVM_E_INVAL;
  Ctx& c = x->c;
  if (!c.exec) return fail(x, AUVM_E_STATE, "plan-only context");
  if (!c.planned) return fail(x, AUVM_E_STATE, "plan first");
  if (!c.host || !c.pool) return fail(x, AUVM_E_STATE, "no host arena or device pool");
  if (uint64_t(first_k) + n_k > c.kernels.size()) return fail(x, AUVM_E_INVAL, "segment beyond the trace");
  auto t0 = std::chrono::steady_clock::now();
  auvm_status s = exec_run(c, first_k, n_k);
  c.run_ns += uint64_t(std::chrono::duration_cast<std::chrono::nanoseconds>(
                           std::chrono::steady_clock::now() - t0).count());
  return s;
}

auvm_status auvm_run_noalloc(auvm_ctx* x, uint32_t first_k, uint32_t n_k) {
  if (!x) return AUVM_E_INVAL;
  Ctx& c = x->c;
  if (!c.exec) return fail(x, AUVM_E_STATE, "plan-only context");
  if (!c.planned) return fail(x, AUVM_E_STATE, "plan first");
  if (!c.host || !c.pool) return fail(x, AUVM_E_STATE, "no host arena or device pool");
  if (uint64_t(first_k) + n_k > c.kernels.size()) return fail(x, AUVM_E_INVAL, "segment beyond the trace");
  auto t0 = std::chrono::steady_clock::now();
  auvm_status s = exec_run_noalloc(c, first_k, n_k);
  c.run_ns += uint64_t(std::chrono::duration_cast<std::chrono::nanoseconds>(
                           std::chrono::steady_clock::now() - t0).count());
  return s;
}

auvm_status auvm_reset(auvm_ctx* x) {
  if (!x) return AUVM_E_INVAL;
  if (!x->c.exec) return fail(x, AUVM_E_STATE, "plan-only context");
  if (!x->c.planned) return fail(x, AUVM_E_STATE, "plan first");
  x->c.run_ns = 0;
  return exec_reset(x->c);
}

auvm_status auvm_read_tensor(auvm_ctx* x, int32_t id, void* dst, uint64_t dst_bytes) {
  if (!x || !dst) return AUVM_E_INVAL;
  Ctx& c = x->c;
  if (id < 0 || size_t(id) >= c.tensors.size()) return fail(x, AUVM_E_INVAL, "unknown tensor id");
  if (dst_bytes < c.tensors[id].bytes) return fail(x, AUVM_E_RANGE, "destination too small");
  if (!c.exec) return fail(x, AUVM_E_STATE, "plan-only context");
  return exec_read(c, id, dst, dst_bytes);
}

auvm_status auvm_get_counters(const auvm_ctx* x, auvm_counters* o) {
  if (!x || !o) return AUVM_E_INVAL;
  const Ctx& c = x->c;
  std::memset(o, 0, sizeof *o);
  const PlanCounters& p = c.plan.counters;
  o->h2d_prefetch_n = p.h2d_prefetch_n;
  o->h2d_prefetch_B = p.h2d_prefetch_B;
  o->h2d_demand_n = p.h2d_demand_n;
  o->h2d_demand_B = p.h2d_demand_B;
  o->d2h_wb_n = p.d2h_wb_n;
  o->d2h_wb_B = p.d2h_wb_B;
  o->drop_n = p.drop_n;
  o->alloc_n = p.alloc_n;
  o->useless_prefetch_n = p.useless_prefetch_n;
  o->useless_prefetch_B = p.useless_prefetch_B;
  for (int i = 0; i < 3; ++i) o->class_n[i] = p.class_n[i];
  o->plan_ns = c.plan_ns;
  o->run_ns = c.run_ns;
  o->kernels_run = c.exec ? exec_kernels_run(c) : 0;
  o->stall_ns = c.exec ? exec_stall_ns(c) : 0;
  return AUVM_OK;
}

auvm_status auvm_get_schedule(const auvm_ctx* x, auvm_sched_entry* buf, uint64_t cap, uint64_t* n) {
  if (!x) return AUVM_E_INVAL;
  return copy_out(x->c.plan.schedule, buf, cap, n, x);
}

auvm_status auvm_get_executed(const auvm_ctx* x, auvm_sched_entry* buf, uint64_t cap, uint64_t* n) {
  if (!x) return AUVM_E_INVAL;
  static const std::vector<auvm_sched_entry> none;
  return copy_out(x->c.exec ? exec_log(x->c) : none, buf, cap, n, x);
}

auvm_status auvm_get_residency(const auvm_ctx* x, auvm_residency* buf, uint64_t cap, uint64_t* n) {
  if (!x) return AUVM_E_INVAL;
  return copy_out(x->c.plan.residency, buf, cap, n, x);
}

auvm_status auvm_get_classes(const auvm_ctx* x, auvm_kernel_class* buf, uint64_t cap, uint64_t* n) {
  if (!x) return AUVM_E_INVAL;
  const Ctx& c = x->c;
  std::vector<auvm_kernel_class> v;
  if (c.planned) {
    v.resize(c.kernels.size());
    for (size_t k = 0; k < v.size(); ++k) {
      std::memset(&v[k], 0, sizeof v[k]);
      v[k].static_cls = c.plan.static_cls[k];
      v[k].dyn_cls = c.plan.dyn_cls[k];
      v[k].flops = c.kernels[k].flops;
      v[k].hbm_bytes = c.kernels[k].hbm;
    }
  }
  return copy_out(v, buf, cap, n, x);
}

auvm_status auvm_get_kernel_times(const auvm_ctx* x, float* dur, float* gap, uint64_t cap, uint64_t* n) {
  if (!x || !n) return AUVM_E_INVAL;
  if (!x->c.exec) {
    *n = 0;
    return AUVM_OK;
  }
  return exec_kernel_times(x->c, dur, gap, cap, n);
}

auvm_status auvm_get_timeline(const auvm_ctx* x, auvm_timeline_entry* buf, uint64_t cap, uint64_t* n) {
  if (!x || !n) return AUVM_E_INVAL;
  if (!x->c.exec) {
    *n = 0;
    return AUVM_OK;
  }
  return copy_out(exec_timeline(x->c), buf, cap, n, x);
}

}  // extern "C"
