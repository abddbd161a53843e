// Queue simulator behind tests/sim/hip/hip_runtime_api.h, linked with the
// library's planner, cost model, C ABI and executor sources into a host-only
// test library.  Test infrastructure: the GPU build never uses it.
//
// Every asynchronous call appends an operation to its stream.  Nothing runs
// until a synchronising call (stream or event synchronise, a blocking copy);
// then operations run one at a time, each time taking the next operation of a
// stream chosen at random among the streams whose next operation may start
// (an event wait may start once the awaited record has run).  Any ordering
// the engine's event waits permit can therefore happen, and an ordering they
// do not enforce happens in about half the runs.  A synchronising call that
// finds nothing runnable while its condition is unmet reports hipErrorUnknown
// (a wait cycle).
//
// Kernels: the TOUCH op only, with the GPU kernel's semantics (log the min
// and max word of each read operand, then fill each written operand with
// slot + 1); the poison fill writes 0xFF bytes.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <deque>
#include <functional>
#include <random>
#include <vector>

#include "kernels.h"

struct SimEvent {
  int64_t recorded = 0;   // records issued
  int64_t completed = 0;  // records run
  double t = 0;           // simulated time of the last run record
};

namespace {

struct Op {
  enum Kind { RUN, RECORD, WAIT } kind;
  std::function<void()> fn;   // RUN
  SimEvent* ev = nullptr;     // RECORD, WAIT
  int64_t gen = 0;            // RECORD: record number; WAIT: record number awaited
};

std::vector<SimStream*> g_streams;
std::mt19937_64 g_rng(1);
bool g_drop_waits = false;   // control runs only: every event wait is ignored
double g_clock = 0;
uint64_t g_ops = 0;

}  // namespace

struct SimStream {
  std::deque<Op> q;
};

namespace {

bool ready(const Op& o) { return o.kind != Op::WAIT || o.ev->completed >= o.gen; }

void exec(Op& o) {
  g_clock += 1;
  ++g_ops;
  switch (o.kind) {
    case Op::RUN: o.fn(); break;
    case Op::RECORD:
      o.ev->completed = std::max(o.ev->completed, o.gen);
      o.ev->t = g_clock;
      break;
    case Op::WAIT: break;
  }
}

// Run operations until done() holds; false if nothing can run before that.
bool drive(const std::function<bool()>& done) {
  std::vector<SimStream*> r;
  while (!done()) {
    r.clear();
    for (SimStream* s : g_streams)
      if (!s->q.empty() && ready(s->q.front())) r.push_back(s);
    if (r.empty()) return false;
    SimStream* s = r[g_rng() % r.size()];
    Op o = std::move(s->q.front());
    s->q.pop_front();
    exec(o);
  }
  return true;
}

bool all_idle() {
  for (SimStream* s : g_streams)
    if (!s->q.empty()) return false;
  return true;
}

void push(hipStream_t s, Op o) { s->q.push_back(std::move(o)); }

}  // namespace

extern "C" {
// Seed of the interleaving choices; returns the operations run so far.
uint64_t auvm_sim_seed(uint64_t seed) {
  g_rng.seed(seed);
  return g_ops;
}
// Control runs: drop every event wait (the engine's ordering disappears).
void auvm_sim_drop_waits(int on) { g_drop_waits = on != 0; }
// A stream for a caller to bind (auvm_bind_streams); never destroyed.
void* auvm_sim_new_stream() {
  hipStream_t s = nullptr;
  hipExtStreamCreateWithCUMask(&s, 0, nullptr);
  return s;
}
}

const char* hipGetErrorString(hipError_t e) {
  switch (e) {
    case hipSuccess: return "hipSuccess";
    case hipErrorInvalidValue: return "hipErrorInvalidValue";
    case hipErrorOutOfMemory: return "hipErrorOutOfMemory";
    default: return "hipErrorUnknown (simulated wait cycle)";
  }
}
hipError_t hipSetDevice(int) { return hipSuccess; }
hipError_t hipDeviceGetAttribute(int* v, hipDeviceAttribute_t, int) {
  *v = 256;
  return hipSuccess;
}
hipError_t hipExtStreamCreateWithCUMask(hipStream_t* s, uint32_t, const uint32_t*) {
  *s = new SimStream();
  g_streams.push_back(*s);
  return hipSuccess;
}
hipError_t hipStreamDestroy(hipStream_t s) {
  if (!drive([&] { return s->q.empty(); })) return hipErrorUnknown;
  g_streams.erase(std::remove(g_streams.begin(), g_streams.end(), s), g_streams.end());
  delete s;
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t s) {
  return drive([&] { return s->q.empty(); }) ? hipSuccess : hipErrorUnknown;
}
hipError_t hipStreamWaitEvent(hipStream_t s, hipEvent_t e, unsigned) {
  if (e->recorded == 0 || g_drop_waits) return hipSuccess;   // nothing recorded yet: no wait
  Op o{Op::WAIT};
  o.ev = e;
  o.gen = e->recorded;
  push(s, std::move(o));
  return hipSuccess;
}
hipError_t hipEventCreate(hipEvent_t* e) {
  *e = new SimEvent();
  return hipSuccess;
}
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned) { return hipEventCreate(e); }
hipError_t hipEventDestroy(hipEvent_t e) {
  delete e;
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t e, hipStream_t s) {
  Op o{Op::RECORD};
  o.ev = e;
  o.gen = ++e->recorded;
  push(s, std::move(o));
  return hipSuccess;
}
hipError_t hipEventSynchronize(hipEvent_t e) {
  return drive([&] { return e->completed >= e->recorded; }) ? hipSuccess : hipErrorUnknown;
}
hipError_t hipEventElapsedTime(float* ms, hipEvent_t a, hipEvent_t b) {
  *ms = float((b->t - a->t) * 1e-3);
  return hipSuccess;
}
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t n, hipMemcpyKind, hipStream_t s) {
  Op o{Op::RUN};
  o.fn = [dst, src, n] { std::memcpy(dst, src, n); };
  push(s, std::move(o));
  return hipSuccess;
}
hipError_t hipMemcpy(void* dst, const void* src, size_t n, hipMemcpyKind) {
  if (!drive(all_idle)) return hipErrorUnknown;
  std::memcpy(dst, src, n);
  return hipSuccess;
}
hipError_t hipMalloc(void** p, size_t n) {
  *p = std::aligned_alloc(256, (n + 255) / 256 * 256);
  return *p ? hipSuccess : hipErrorOutOfMemory;
}
hipError_t hipFree(void* p) {
  std::free(p);
  return hipSuccess;
}
hipError_t hipHostMalloc(void** p, size_t n, unsigned) { return hipMalloc(p, n); }
hipError_t hipHostFree(void* p) { return hipFree(p); }

namespace auvm {

hipError_t launch_op(const Kernel& k, const std::vector<Tensor>& T, uint8_t* const* ptrs, hipStream_t s) {
  if (k.op != AUVM_OP_TOUCH) return hipErrorInvalidValue;
  const int n = int(k.ids.size()) - 1;
  std::vector<uint32_t*> data(n);
  std::vector<uint64_t> words(n);
  std::vector<uint8_t> mode(n);
  for (int i = 0; i < n; ++i) {
    data[i] = reinterpret_cast<uint32_t*>(ptrs[i + 1]);
    words[i] = T[k.ids[i + 1]].bytes / 4;
    mode[i] = k.modes[i + 1];
  }
  uint32_t* log = reinterpret_cast<uint32_t*>(ptrs[0]);
  const int64_t slot = k.shape[0];
  Op o{Op::RUN};
  o.fn = [=] {
    for (int i = 0; i < n; ++i) {
      if (mode[i] & 1u) {
        uint32_t mn = 0xffffffffu, mx = 0u;
        for (uint64_t w = 0; w < words[i]; ++w) {
          mn = std::min(mn, data[i][w]);
          mx = std::max(mx, data[i][w]);
        }
        log[16 * slot + 2 * (i + 1)] = mn;
        log[16 * slot + 2 * (i + 1) + 1] = mx;
      }
      if (mode[i] & 2u)
        for (uint64_t w = 0; w < words[i]; ++w) data[i][w] = uint32_t(slot + 1);
    }
  };
  push(s, std::move(o));
  return hipSuccess;
}

// the static device scratch: a host buffer here
uint64_t scratch_capacity() { return uint64_t(8) << 20; }
hipError_t scratch_address(int, void** out) {
  static std::vector<uint8_t> buf(size_t(8) << 20);
  *out = buf.data();
  return hipSuccess;
}

hipError_t launch_poison(uint8_t* p, uint64_t bytes, hipStream_t s) {
  Op o{Op::RUN};
  o.fn = [p, bytes] { std::memset(p, 0xFF, bytes); };
  push(s, std::move(o));
  return hipSuccess;
}

}  // namespace auvm
