// Transfer engine and executor on the HIP runtime.
//
// Replays a plan on four streams: compute (kernels), two h2d streams (pinned
// host arena -> device pool copies, alternating by copy number, so that a copy
// held back by its window's previous readers does not hold back the next one)
// and d2h (write-backs).  A plan with write-backs keeps its copies on one h2d
// stream: both directions share the host link, and a second copy in flight
// halves the rate of the write-back that frees the first copy's window.
// Ordering is event based and never blocks the host inside a run segment:
//  * a copy into a pool window waits for the kernels that last used the
//    tensors previously in that window and for write-backs out of it;
//  * a demand fetch for kernel k additionally waits for kernel k-1, so it
//    starts when execution reaches k (the fault-driven baseline of the paper,
//    Sec. II-A and V-A); prefetches wait only for their victims;
//  * a refetch of a tensor waits for its own pending write-back;
//  * a kernel waits for the copies that brought its operands and, for
//    first-write allocations, for transfers still touching the window.
// Streams are in-order, so each stream keeps the highest kernel/copy index it
// already waits on and skips older waits; copies of the two h2d streams have
// separate event rings and separate highest-waited indices, and a copy into a
// window last written from the other h2d stream waits for that copy.
//
// Timing policy: kernels, host-to-device and device-to-host copies each get a
// track of start/end events; times are chained from one base event per run
// segment through the short gaps between consecutive items of a track, so
// they keep float precision over long runs.
#include <hip/hip_runtime_api.h>

#include <sys/mman.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <condition_variable>
#include <cstring>
#include <map>
#include <mutex>
#include <thread>
#include <vector>

#include "ctx.h"
#include "kernels.h"

namespace auvm {

namespace {
constexpr int64_t kRing = 8192;    // events per ring
constexpr int64_t kTimeRing = 4096;
constexpr int kCopyThreads = 8;    // host threads of a staging copy

// One host memcpy split over worker threads (pageable tier to a staging slot):
// a single thread copies about 10 GB/s, well below the host link.
class CopyPool {
 public:
  explicit CopyPool(int n) : n_threads_(n) {
    th_.reserve(size_t(n));
    for (int i = 0; i < n; ++i) th_.emplace_back([this, i] { work(i); });
  }
  ~CopyPool() {
    {
      std::lock_guard<std::mutex> g(m_);
      stop_ = true;
    }
    cv_.notify_all();
    for (auto& t : th_) t.join();
  }
  void copy(uint8_t* dst, const uint8_t* src, uint64_t n) {
    std::unique_lock<std::mutex> g(m_);
    dst_ = dst;
    src_ = src;
    n_ = n;
    left_ = n_threads_;
    ++gen_;
    cv_.notify_all();
    done_.wait(g, [this] { return left_ == 0; });
  }

 private:
  void work(int i) {
    uint64_t seen = 0;
    for (;;) {
      uint8_t* d;
      const uint8_t* s;
      uint64_t n;
      {
        std::unique_lock<std::mutex> g(m_);
        cv_.wait(g, [&] { return stop_ || gen_ != seen; });
        if (stop_) return;
        seen = gen_;
        d = dst_;
        s = src_;
        n = n_;
      }
      // thread i copies the i-th of n_threads_ page-aligned parts (at least a page)
      const uint64_t per = ((n + uint64_t(n_threads_) - 1) / uint64_t(n_threads_) + 4095) / 4096 * 4096;
      const uint64_t a = std::min(n, per * uint64_t(i)), b = std::min(n, a + per);
      if (b > a) std::memcpy(d + a, s + a, b - a);
      std::lock_guard<std::mutex> g(m_);
      if (--left_ == 0) done_.notify_one();
    }
  }
  const int n_threads_;
  std::vector<std::thread> th_;
  std::mutex m_;
  std::condition_variable cv_, done_;
  uint8_t* dst_ = nullptr;
  const uint8_t* src_ = nullptr;
  uint64_t n_ = 0, gen_ = 0;
  int left_ = 0;
  bool stop_ = false;
};
}  // namespace

class Executor {
 public:
  explicit Executor(Ctx& c) : c_(c) {}
  ~Executor() { destroy(); }

  auvm_status init() {
    if (!ok(hipSetDevice(c_.device), "hipSetDevice")) return AUVM_E_HIP;
    // HIP spreads streams over a few hardware queues; two streams that share
    // one are serialized (a kernel queued behind a copy's completion marker
    // waits for the copy).  A stream created with a CU mask gets a hardware
    // queue of its own; the mask enables every CU.
    int ncu = 0;
    if (!ok(hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, c_.device), "hipDeviceGetAttribute"))
      return AUVM_E_HIP;
    std::vector<uint32_t> mask(size_t((ncu + 31) / 32), 0xffffffffu);
    if (ncu % 32) mask.back() = (1u << (ncu % 32)) - 1u;
    hipStream_t* ss[4] = {&comp_, &h2d_[0], &h2d_[1], &d2h_};
    for (int i = 0; i < 4; ++i) {
      if (!ok(hipExtStreamCreateWithCUMask(ss[i], uint32_t(mask.size()), mask.data()), "hipExtStreamCreateWithCUMask"))
        return AUVM_E_HIP;
      own_[i] = true;
    }
    for (auto* ring : {&kev_, &hev_[0], &hev_[1], &dev_}) {
      ring->assign(kRing, nullptr);
      for (auto& e : *ring)
        if (!ok(hipEventCreateWithFlags(&e, hipEventDisableTiming), "hipEventCreate")) return AUVM_E_HIP;
    }
    kown_.assign(kRing, -1);
    hown_[0].assign(kRing, -1);
    hown_[1].assign(kRing, -1);
    down_.assign(kRing, -1);
    // the static scratch of this device, for run_noalloc; a failure here only
    // disables that entry point
    scratch_status_ = scratch_address(c_.device, &scratch_);
    return AUVM_OK;
  }

  void destroy() {
    if (c_.device < 0) return;
    (void)hipSetDevice(c_.device);
    hipStream_t ss[4] = {comp_, h2d_[0], h2d_[1], d2h_};
    for (int i = 0; i < 4; ++i)
      if (ss[i]) (void)hipStreamSynchronize(ss[i]);
    for (auto* ring : {&kev_, &hev_[0], &hev_[1], &dev_, &bases_})
      for (auto& e : *ring)
        if (e) (void)hipEventDestroy(e);
    for (auto& e : stage_ev_)
      if (e) (void)hipEventDestroy(e);
    copy_pool_.reset();
    for (Track* tr : {&ktr_, &htr_[0], &htr_[1], &dtr_})
      for (auto* ring : {&tr->s, &tr->e})
        for (auto& e : *ring)
          if (e) (void)hipEventDestroy(e);
    for (int i = 0; i < 4; ++i)
      if (own_[i] && ss[i]) (void)hipStreamDestroy(ss[i]);
    comp_ = h2d_[0] = h2d_[1] = d2h_ = nullptr;
  }

  auvm_status bind(void* comp, void* h2d, void* d2h) {
    // a caller's h2d stream carries both copy sequences (in order: still correct)
    hipStream_t* ss[4] = {&comp_, &h2d_[0], &h2d_[1], &d2h_};
    void* in[4] = {comp, h2d, h2d, d2h};
    for (int i = 0; i < 4; ++i) {
      if (!in[i]) continue;
      if (*ss[i]) (void)hipStreamSynchronize(*ss[i]);
      if (own_[i] && *ss[i]) (void)hipStreamDestroy(*ss[i]);
      *ss[i] = static_cast<hipStream_t>(in[i]);
      own_[i] = false;
    }
    return AUVM_OK;
  }

  auvm_status reset() {
    if (!ok(hipSetDevice(c_.device), "hipSetDevice")) return AUVM_E_HIP;
    if (!sync_all()) return AUVM_E_HIP;
    // a tiered arena's staging events and copy threads (the arena comes after
    // the executor; every plan resets it before a run)
    if (!c_.stage.empty() && !copy_pool_) {
      for (auto& e : stage_ev_)
        if (!ok(hipEventCreateWithFlags(&e, hipEventDisableTiming), "hipEventCreate")) return AUVM_E_HIP;
      copy_pool_.reset(new CopyPool(kCopyThreads));
    }
    const size_t nT = c_.tensors.size(), K = c_.kernels.size();
    cursor_ = 0;
    next_k_ = 0;
    where_.assign(nT, -1);
    last_use_.assign(nT, -1);
    copy_seq_.assign(nT, 0);
    wb_seq_.assign(nT, 0);
    h2d_seq_ = d2h_seq_ = 0;
    d2h_waited_k_ = -1;
    comp_waited_d2h_ = pend_d2h_ = 0;
    for (int p = 0; p < 2; ++p) {
      h2d_waited_k_[p] = -1;
      h2d_waited_d2h_[p] = h2d_waited_h2d_[p] = comp_waited_h2d_[p] = pend_h2d_[p] = 0;
      std::fill(hown_[p].begin(), hown_[p].end(), -1);
    }
    std::fill(kown_.begin(), kown_.end(), -1);
    std::fill(down_.begin(), down_.end(), -1);
    hazards_.clear();
    log_.clear();
    log_.reserve(c_.plan.schedule.size());   // a run never grows it
    kernels_run_ = 0;
    stall_ms_ = 0;
    dur_.assign(K, 0.f);
    gap_.assign(K, 0.f);
    for (Track* tr : {&ktr_, &htr_[0], &htr_[1], &dtr_}) tr->restart();
    tl_.clear();
    seg_ = -1;
    two_h2d_ = std::none_of(c_.plan.schedule.begin(), c_.plan.schedule.end(),
                            [](const auvm_sched_entry& e) { return e.op == AUVM_D2H_WRITEBACK; });
    // kernels whose completion some transfer waits on
    need_ev_.assign(K, 0);
    std::vector<int64_t> last(nT, -1);
    for (const auto& e : c_.plan.schedule) {
      if (e.op == AUVM_LAUNCH) {
        for (auto& a : c_.kernels[e.issue_k].acc) last[a.first] = e.issue_k;
      } else if (e.op == AUVM_D2H_WRITEBACK || e.op == AUVM_DROP) {
        if (last[e.tensor] >= 0) need_ev_[last[e.tensor]] = 1;
      } else if (e.op == AUVM_H2D_DEMAND && e.issue_k > 0) {
        need_ev_[e.issue_k - 1] = 1;
      }
    }
    return AUVM_OK;
  }

  auvm_status run(uint32_t first_k, uint32_t n_k) {
    if (int64_t(first_k) != next_k_) {
      c_.err = "run segments must be contiguous: next kernel is " + std::to_string(next_k_);
      return AUVM_E_STATE;
    }
    if (!ok(hipSetDevice(c_.device), "hipSetDevice")) return AUVM_E_HIP;
    if (c_.pol.timing && !begin_segment()) return AUVM_E_HIP;
    const int64_t end_k = int64_t(first_k) + n_k;
    const auto& S = c_.plan.schedule;
    while (cursor_ < S.size() && S[cursor_].issue_k < end_k) {
      auvm_status s = step(S[cursor_]);
      if (s != AUVM_OK) return s;
      log_.push_back(S[cursor_]);
      ++cursor_;
    }
    if (!sync_all()) return AUVM_E_HIP;
    if (c_.pol.timing) harvest_all();
    return AUVM_OK;
  }

  // auvm_run with the kernels' workspace operands (ATTN_BWD's D, RMSNORM_BWD's
  // rstd) in the static scratch instead of their pool windows; no event,
  // stream or memory is created.
  auvm_status run_noalloc(uint32_t first_k, uint32_t n_k) {
    if (c_.pol.timing) {
      c_.err = "run_noalloc: the timing policy creates events; plan with timing off";
      return AUVM_E_STATE;
    }
    if (scratch_status_ != hipSuccess || !scratch_) {
      c_.err = std::string("run_noalloc: no static scratch on this device: ") + hipGetErrorString(scratch_status_);
      return AUVM_E_HIP;
    }
    const int64_t end_k = int64_t(first_k) + n_k;
    for (int64_t k = first_k; k < end_k; ++k) {
      const int w = workspace_operand(c_.kernels[k]);
      if (w < 0) continue;
      const uint64_t need = c_.tensors[c_.kernels[k].ids[w]].bytes;
      if (need > scratch_capacity()) {
        c_.err = "run_noalloc: kernel " + std::to_string(k) + " needs a " + std::to_string(need) +
                 "-byte workspace, above the static scratch's " + std::to_string(scratch_capacity());
        return AUVM_E_RANGE;
      }
    }
    noalloc_ = true;
    auvm_status s = run(first_k, n_k);
    noalloc_ = false;
    return s;
  }

  // positional index of an op's workspace operand, or -1
  static int workspace_operand(const Kernel& k) {
    if (k.op == AUVM_OP_RMSNORM_BWD) return 6;
    if (k.op == AUVM_OP_ATTN_BWD) return 9;
    return -1;
  }

  auvm_status read(int32_t id, void* dst) {
    if (!ok(hipSetDevice(c_.device), "hipSetDevice")) return AUVM_E_HIP;
    if (!sync_all()) return AUVM_E_HIP;
    const Tensor& t = c_.tensors[id];
    if (where_.size() == c_.tensors.size() && where_[id] >= 0) {
      if (!ok(hipMemcpy(dst, c_.pool + where_[id], t.bytes, hipMemcpyDeviceToHost), "hipMemcpy D2H"))
        return AUVM_E_HIP;
    } else {
      std::memcpy(dst, c_.host_at(t.arena_off), t.bytes);
    }
    return AUVM_OK;
  }

  const std::vector<auvm_sched_entry>& log() const { return log_; }
  uint64_t kernels_run() const { return kernels_run_; }
  uint64_t stall_ns() const { return uint64_t(std::llround(stall_ms_ * 1e6)); }

  auvm_status times(float* dur, float* gap, uint64_t cap, uint64_t* n) const {
    const uint64_t m = uint64_t(ktr_.n);
    *n = m;
    if (!dur && !gap) return AUVM_OK;
    if (cap < m) return AUVM_E_RANGE;
    if (dur) std::memcpy(dur, dur_.data(), m * sizeof(float));
    if (gap) std::memcpy(gap, gap_.data(), m * sizeof(float));
    return AUVM_OK;
  }
  const std::vector<auvm_timeline_entry>& timeline() const { return tl_; }

 private:
  struct Hazard {
    uint64_t end;
    int64_t last_k, d2h, h2d;   // h2d: the last copy (or poison fill) into the window
  };
  static int par(int64_t seq) { return int(seq & 1); }   // event ring of copy number seq
  // h2d stream of copy number seq (the rings and waits stay per parity: with
  // one stream for both they are only stronger than needed)
  int lane(int64_t seq) const { return two_h2d_ ? par(seq) : 1; }

  // A copy from the pageable tier: pieces of at most kStageBytes go through
  // the pinned staging ring.  A slot is refilled once the device copy that
  // read it last has completed (its previous copies were issued earlier, so
  // the wait ends); the host copy of a piece overlaps the device copies of
  // the pieces before it.
  bool staged_copy(uint8_t* dst, const uint8_t* src, uint64_t bytes, hipStream_t st) {
    if (c_.stage.size() != size_t(kStageSlots) || !copy_pool_) return ok(hipErrorInvalidValue, "staging ring");
    for (uint64_t done = 0; done < bytes;) {
      const uint64_t n = std::min(kStageBytes, bytes - done);
      const int s = int(stage_next_++ % kStageSlots);
      if (stage_used_[s] && !ok(hipEventSynchronize(stage_ev_[s]), "hipEventSynchronize")) return false;
      copy_pool_->copy(c_.stage[s], src + done, n);
      if (!ok(hipMemcpyAsync(dst + done, c_.stage[s], n, hipMemcpyHostToDevice, st), "hipMemcpyAsync H2D"))
        return false;
      if (!ok(hipEventRecord(stage_ev_[s], st), "hipEventRecord")) return false;
      stage_used_[s] = true;
      done += n;
    }
    return true;
  }

  bool ok(hipError_t e, const char* what) {
    if (e == hipSuccess) return true;
    c_.err = std::string(what) + ": " + hipGetErrorString(e);
    return false;
  }

  bool sync_all() {
    hipStream_t ss[4] = {comp_, h2d_[0], h2d_[1], d2h_};
    for (auto s : ss)
      if (s && !ok(hipStreamSynchronize(s), "hipStreamSynchronize")) return false;
    return true;
  }

  // -- event rings ------------------------------------------------------------
  bool record(std::vector<hipEvent_t>& ring, std::vector<int64_t>& own, int64_t idx, hipStream_t s) {
    int64_t slot = idx % kRing;
    if (!ok(hipEventRecord(ring[slot], s), "hipEventRecord")) return false;
    own[slot] = idx;
    return true;
  }
  // Make stream s wait until item idx of a ring is complete.  A slot reused by
  // a later item of the same in-order stream implies idx is complete too.
  bool wait(hipStream_t s, std::vector<hipEvent_t>& ring, std::vector<int64_t>& own, int64_t idx,
            int64_t& waited) {
    if (idx <= waited) return true;
    int64_t slot = idx % kRing;
    if (own[slot] < idx) {
      c_.err = "internal: wait on an event that was never recorded";
      return false;
    }
    if (!ok(hipStreamWaitEvent(s, ring[slot], 0), "hipStreamWaitEvent")) return false;
    waited = own[slot];
    return true;
  }

  // -- pool-window hazards left behind by evicted tensors ----------------------
  void add_hazard(uint64_t off, uint64_t end, int64_t last_k, int64_t d2h, int64_t h2d) {
    hazards_[off] = Hazard{end, last_k, d2h, h2d};
  }
  // Collect and remove the hazards overlapping [a, b), keeping uncovered parts;
  // h2d[p] is the latest copy into the range made on h2d stream p.
  void take_hazards(uint64_t a, uint64_t b, int64_t* last_k, int64_t* d2h, int64_t h2d[2]) {
    *last_k = -1;
    *d2h = 0;
    h2d[0] = h2d[1] = 0;
    auto it = hazards_.lower_bound(a);
    if (it != hazards_.begin()) {
      auto p = std::prev(it);
      if (p->second.end > a) it = p;
    }
    std::vector<std::pair<uint64_t, Hazard>> keep;
    while (it != hazards_.end() && it->first < b) {
      const Hazard& h = it->second;
      *last_k = std::max(*last_k, h.last_k);
      *d2h = std::max(*d2h, h.d2h);
      if (h.h2d) h2d[par(h.h2d)] = std::max(h2d[par(h.h2d)], h.h2d);
      if (it->first < a) keep.push_back({it->first, Hazard{a, h.last_k, h.d2h, h.h2d}});
      if (h.end > b) keep.push_back({b, Hazard{h.end, h.last_k, h.d2h, h.h2d}});
      it = hazards_.erase(it);
    }
    for (auto& kv : keep) hazards_[kv.first] = kv.second;
  }

  // -- one schedule entry -------------------------------------------------------
  auvm_status step(const auvm_sched_entry& e) {
    const int32_t t = e.tensor;
    if (e.op != AUVM_LAUNCH) {
      if (t < 0 || size_t(t) >= c_.tensors.size()) return internal("schedule names an unknown tensor");
      if (e.dev_off > c_.M || c_.M - e.dev_off < e.bytes || e.bytes < c_.tensors[t].bytes)
        return internal("schedule window outside the device pool");
    }
    switch (e.op) {
      case AUVM_D2H_WRITEBACK:
      case AUVM_DROP: {
        if (where_[t] != int64_t(e.dev_off)) return internal("eviction of a tensor not at its window");
        int64_t wb = 0;
        if (e.op == AUVM_D2H_WRITEBACK) {
          if (last_use_[t] >= 0 && !wait(d2h_, kev_, kown_, last_use_[t], d2h_waited_k_)) return AUVM_E_HIP;
          const Tensor& x = c_.tensors[t];
          if (c_.pol.timing && !begin_item(dtr_, d2h_, AUVM_TL_D2H, int64_t(cursor_), x.bytes))
            return AUVM_E_HIP;
          if (!ok(hipMemcpyAsync(c_.host_at(x.arena_off), c_.pool + e.dev_off, x.bytes,
                                 hipMemcpyDeviceToHost, d2h_), "hipMemcpyAsync D2H"))
            return AUVM_E_HIP;
          if (c_.pol.timing && !end_item(dtr_, d2h_)) return AUVM_E_HIP;
          wb = ++d2h_seq_;
          if (!record(dev_, down_, wb, d2h_)) return AUVM_E_HIP;
          wb_seq_[t] = wb;
        }
        int64_t h2d = copy_seq_[t];
        if (c_.pol.validate) {
          // poison the vacated window once its readers, its fill and its write-back are done
          const int64_t q = h2d_seq_ + 1;
          const int sp = par(q);
          hipStream_t st = h2d_[lane(q)];
          if (last_use_[t] >= 0 && !wait(st, kev_, kown_, last_use_[t], h2d_waited_k_[sp])) return AUVM_E_HIP;
          if (wb && !wait(st, dev_, down_, wb, h2d_waited_d2h_[sp])) return AUVM_E_HIP;
          if (h2d && par(h2d) != sp && !wait(st, hev_[1 - sp], hown_[1 - sp], h2d, h2d_waited_h2d_[sp]))
            return AUVM_E_HIP;
          if (!ok(launch_poison(c_.pool + e.dev_off, e.bytes, st), "poison")) return AUVM_E_HIP;
          h2d = h2d_seq_ = q;
          if (!record(hev_[sp], hown_[sp], h2d, st)) return AUVM_E_HIP;
        }
        add_hazard(e.dev_off, e.dev_off + e.bytes, last_use_[t], wb, h2d);
        where_[t] = -1;
        return AUVM_OK;
      }
      case AUVM_H2D_DEMAND:
      case AUVM_H2D_PREFETCH: {
        if (where_[t] >= 0) return internal("fetch of a resident tensor");
        int64_t lk, d2h, h2d[2];
        take_hazards(e.dev_off, e.dev_off + e.bytes, &lk, &d2h, h2d);
        const int64_t seq = h2d_seq_ + 1;
        const int sp = par(seq), ln = lane(seq);
        hipStream_t st = h2d_[ln];
        if (lk >= 0 && !wait(st, kev_, kown_, lk, h2d_waited_k_[sp])) return AUVM_E_HIP;
        if (e.op == AUVM_H2D_DEMAND && e.issue_k > 0 &&
            !wait(st, kev_, kown_, e.issue_k - 1, h2d_waited_k_[sp]))
          return AUVM_E_HIP;
        int64_t dw = std::max(d2h, wb_seq_[t]);
        if (dw && !wait(st, dev_, down_, dw, h2d_waited_d2h_[sp])) return AUVM_E_HIP;
        // an earlier fill of the window from the other stream lands first
        if (h2d[1 - sp] && !wait(st, hev_[1 - sp], hown_[1 - sp], h2d[1 - sp], h2d_waited_h2d_[sp]))
          return AUVM_E_HIP;
        const Tensor& x = c_.tensors[t];
        const int32_t kind = ln == 1 ? AUVM_TL_H2D : AUVM_TL_H2D_B;   // odd copy numbers: the first stream
        if (c_.pol.timing && !begin_item(htr_[ln], st, kind, int64_t(cursor_), x.bytes)) return AUVM_E_HIP;
        if (c_.pageable(x)) {
          if (!staged_copy(c_.pool + e.dev_off, c_.host_at(x.arena_off), x.bytes, st)) return AUVM_E_HIP;
        } else if (!ok(hipMemcpyAsync(c_.pool + e.dev_off, c_.host + x.arena_off, x.bytes,
                                      hipMemcpyHostToDevice, st), "hipMemcpyAsync H2D")) {
          return AUVM_E_HIP;
        }
        if (c_.pol.timing && !end_item(htr_[ln], st)) return AUVM_E_HIP;
        h2d_seq_ = seq;
        if (!record(hev_[sp], hown_[sp], seq, st)) return AUVM_E_HIP;
        copy_seq_[t] = seq;
        where_[t] = int64_t(e.dev_off);
        return AUVM_OK;
      }
      case AUVM_ALLOC: {
        if (where_[t] >= 0) return internal("allocation of a resident tensor");
        int64_t lk, d2h, h2d[2];
        take_hazards(e.dev_off, e.dev_off + e.bytes, &lk, &d2h, h2d);
        // previous readers ran earlier on the compute stream; transfers did not
        pend_d2h_ = std::max(pend_d2h_, d2h);
        pend_h2d_[0] = std::max(pend_h2d_[0], h2d[0]);
        pend_h2d_[1] = std::max(pend_h2d_[1], h2d[1]);
        copy_seq_[t] = 0;
        where_[t] = int64_t(e.dev_off);
        return AUVM_OK;
      }
      case AUVM_LAUNCH:
        return launch(e.issue_k);
    }
    return internal("unknown schedule op");
  }

  auvm_status launch(int64_t k) {
    const Kernel& kd = c_.kernels[k];
    int64_t need_h2d[2] = {pend_h2d_[0], pend_h2d_[1]};
    for (auto& a : kd.acc) {
      if (where_[a.first] < 0) return internal("operand not resident at launch");
      const int64_t q = copy_seq_[a.first];
      if (q) need_h2d[par(q)] = std::max(need_h2d[par(q)], q);
    }
    for (int p = 0; p < 2; ++p)
      if (need_h2d[p] && !wait(comp_, hev_[p], hown_[p], need_h2d[p], comp_waited_h2d_[p])) return AUVM_E_HIP;
    if (pend_d2h_ && !wait(comp_, dev_, down_, pend_d2h_, comp_waited_d2h_)) return AUVM_E_HIP;
    pend_h2d_[0] = pend_h2d_[1] = pend_d2h_ = 0;
    uint8_t* ptrs[16];
    for (size_t i = 0; i < kd.ids.size(); ++i) ptrs[i] = c_.pool + where_[kd.ids[i]];
    if (noalloc_) {
      const int w = workspace_operand(kd);
      if (w >= 0) ptrs[w] = static_cast<uint8_t*>(scratch_);
    }
    const bool timing = c_.pol.timing != 0;
    if (timing) {
      if (ktr_.n != k) return internal("timed kernels must run from kernel 0 in order");
      if (!begin_item(ktr_, comp_, AUVM_TL_KERNEL, k, 0)) return AUVM_E_HIP;
    }
    if (!ok(launch_op(kd, c_.tensors, ptrs, comp_), "kernel launch")) return AUVM_E_HIP;
    if (timing && !end_item(ktr_, comp_)) return AUVM_E_HIP;
    if (need_ev_[k] && !record(kev_, kown_, k, comp_)) return AUVM_E_HIP;
    for (auto& a : kd.acc) last_use_[a.first] = k;
    next_k_ = k + 1;
    ++kernels_run_;
    return AUVM_OK;
  }

  auvm_status internal(const char* m) {
    c_.err = std::string("internal: ") + m;
    return AUVM_E_STATE;
  }

  // -- timing tracks ---------------------------------------------------------------
  struct Track {
    std::vector<hipEvent_t> s, e;  // start/end events, ring of kTimeRing
    std::vector<int64_t> tl;       // timeline entry of each item
    int64_t n = 0, harvested = 0;
    double next = 0;               // chained start time of item `harvested`
    void restart() {
      tl.clear();
      n = harvested = 0;
      next = 0;
    }
  };

  bool begin_segment() {
    for (Track* tr : {&ktr_, &htr_[0], &htr_[1], &dtr_}) {
      if (!tr->s.empty()) continue;
      tr->s.assign(kTimeRing, nullptr);
      tr->e.assign(kTimeRing, nullptr);
      // timestamps only (ordering uses the sync events and every segment ends
      // with a full wait), so no system-scope fence per event
      for (auto* ring : {&tr->s, &tr->e})
        for (auto& e : *ring)
          if (!ok(hipEventCreateWithFlags(&e, hipEventDisableSystemFence), "hipEventCreate")) return false;
    }
    ++seg_;
    if (size_t(seg_) >= bases_.size()) {
      hipEvent_t b = nullptr;
      if (!ok(hipEventCreateWithFlags(&b, hipEventDisableSystemFence), "hipEventCreate")) return false;
      bases_.push_back(b);
    }
    // the streams are idle here (every segment ends with a full wait)
    if (!ok(hipEventRecord(bases_[seg_], comp_), "hipEventRecord")) return false;
    host0_ = std::chrono::steady_clock::now();
    return true;
  }

  bool begin_item(Track& tr, hipStream_t st, int32_t kind, int64_t index, uint64_t bytes) {
    while (tr.harvested + kTimeRing <= tr.n)   // free the slot this item reuses
      if (!harvest(tr, tr.harvested++)) return false;
    auvm_timeline_entry x{};
    x.kind = kind;
    x.segment = seg_;
    x.index = index;
    x.bytes = bytes;
    x.host_ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - host0_).count();
    tr.tl.push_back(int64_t(tl_.size()));
    tl_.push_back(x);
    return ok(hipEventRecord(tr.s[tr.n % kTimeRing], st), "hipEventRecord");
  }
  bool end_item(Track& tr, hipStream_t st) {
    if (!ok(hipEventRecord(tr.e[tr.n % kTimeRing], st), "hipEventRecord")) return false;
    ++tr.n;
    return true;
  }

  // Item j's duration; its start is the segment base's elapsed time for the
  // first item of a segment, else the chained value; the gap to item j+1 of
  // the same segment sets the next chained start.
  bool harvest(Track& tr, int64_t j) {
    hipEvent_t s = tr.s[j % kTimeRing], e = tr.e[j % kTimeRing];
    float ms = 0;
    if (!ok(hipEventSynchronize(e), "hipEventSynchronize")) return false;
    if (!ok(hipEventElapsedTime(&ms, s, e), "hipEventElapsedTime")) return false;
    auvm_timeline_entry& x = tl_[tr.tl[j]];
    const bool first = j == 0 || tl_[tr.tl[j - 1]].segment != x.segment;
    if (first) {
      float b = 0;
      if (!ok(hipEventElapsedTime(&b, bases_[x.segment], s), "hipEventElapsedTime")) return false;
      tr.next = b;
    }
    x.start_ms = tr.next;
    x.end_ms = tr.next + ms;
    float g = 0;
    const bool chained = j + 1 < tr.n && tl_[tr.tl[j + 1]].segment == x.segment;
    if (chained) {
      hipEvent_t s2 = tr.s[(j + 1) % kTimeRing];
      if (!ok(hipEventSynchronize(s2), "hipEventSynchronize")) return false;
      if (!ok(hipEventElapsedTime(&g, e, s2), "hipEventElapsedTime")) return false;
      tr.next = x.end_ms + g;
    }
    if (&tr == &ktr_) {
      dur_[j] = ms;
      // the gap before the first kernel of a run segment includes host time: not reported
      if (chained) {
        gap_[j + 1] = g;
        stall_ms_ += g;
      }
    }
    return true;
  }
  void harvest_all() {
    for (Track* tr : {&ktr_, &htr_[0], &htr_[1], &dtr_})
      while (tr->harvested < tr->n)
        if (!harvest(*tr, tr->harvested++)) return;
  }

  Ctx& c_;
  hipEvent_t stage_ev_[kStageSlots] = {};   // last device copy out of each staging slot
  bool stage_used_[kStageSlots] = {};
  uint64_t stage_next_ = 0;
  std::unique_ptr<CopyPool> copy_pool_;
  hipStream_t comp_ = nullptr, h2d_[2] = {nullptr, nullptr}, d2h_ = nullptr;
  bool own_[4] = {false, false, false, false};   // comp_, h2d_[0], h2d_[1], d2h_
  std::vector<hipEvent_t> kev_, hev_[2], dev_, bases_;   // hev_[p]: copies of h2d stream p
  std::vector<int64_t> kown_, hown_[2], down_;
  size_t cursor_ = 0;
  int64_t next_k_ = 0;
  std::vector<int64_t> where_, last_use_, copy_seq_, wb_seq_;
  int64_t h2d_seq_ = 0, d2h_seq_ = 0;
  int64_t h2d_waited_k_[2] = {-1, -1}, d2h_waited_k_ = -1, h2d_waited_d2h_[2] = {0, 0};
  int64_t h2d_waited_h2d_[2] = {0, 0};   // stream p: other stream's copies waited for
  int64_t comp_waited_h2d_[2] = {0, 0}, comp_waited_d2h_ = 0;
  int64_t pend_h2d_[2] = {0, 0}, pend_d2h_ = 0;
  bool two_h2d_ = true;   // the plan has no write-backs
  std::map<uint64_t, Hazard> hazards_;
  std::vector<uint8_t> need_ev_;
  std::vector<auvm_sched_entry> log_;
  uint64_t kernels_run_ = 0;
  double stall_ms_ = 0;   // sum of the reported gaps
  std::vector<float> dur_, gap_;
  Track ktr_, htr_[2], dtr_;
  std::vector<auvm_timeline_entry> tl_;
  int32_t seg_ = -1;
  std::chrono::steady_clock::time_point host0_;
  void* scratch_ = nullptr;                 // this device's static scratch
  hipError_t scratch_status_ = hipErrorNotInitialized;
  bool noalloc_ = false;                    // inside run_noalloc
};

Ctx::~Ctx() {
  exec.reset();
  free_owned(*this);
}

void ExecDeleter::operator()(Executor* e) const { delete e; }

ExecPtr make_executor(Ctx& c) {
  ExecPtr x(new Executor(c));
  if (x->init() != AUVM_OK) return nullptr;
  return x;
}

auvm_status exec_bind_streams(Ctx& c, void* a, void* b, void* d) { return c.exec->bind(a, b, d); }
auvm_status exec_run(Ctx& c, uint32_t f, uint32_t n) { return c.exec->run(f, n); }
auvm_status exec_run_noalloc(Ctx& c, uint32_t f, uint32_t n) { return c.exec->run_noalloc(f, n); }
auvm_status exec_reset(Ctx& c) { return c.exec->reset(); }
auvm_status exec_read(Ctx& c, int32_t id, void* dst, uint64_t) { return c.exec->read(id, dst); }
const std::vector<auvm_sched_entry>& exec_log(const Ctx& c) { return c.exec->log(); }
uint64_t exec_kernels_run(const Ctx& c) { return c.exec->kernels_run(); }
uint64_t exec_stall_ns(const Ctx& c) { return c.exec->stall_ns(); }
auvm_status exec_kernel_times(const Ctx& c, float* d, float* g, uint64_t cap, uint64_t* n) {
  return c.exec->times(d, g, cap, n);
}
const std::vector<auvm_timeline_entry>& exec_timeline(const Ctx& c) { return c.exec->timeline(); }

auvm_status host_alloc_pinned(Ctx& c, uint64_t bytes) {
  void* p = nullptr;
  if (hipHostMalloc(&p, bytes, hipHostMallocDefault) != hipSuccess || !p) {
    c.err = "hipHostMalloc of the host arena failed";
    return AUVM_E_NOMEM;
  }
  c.host = static_cast<uint8_t*>(p);
  c.host_owned = true;
  return AUVM_OK;
}

auvm_status host_alloc_pageable(Ctx& c) {
  const uint64_t n = c.arena_bytes - c.pinned_bytes;
  void* p = mmap(nullptr, n, PROT_READ | PROT_WRITE, MAP_PRIVATE | MAP_ANONYMOUS | MAP_NORESERVE, -1, 0);
  if (p == MAP_FAILED) {
    c.err = "mmap of the pageable host tier failed";
    return AUVM_E_NOMEM;
  }
  c.host_pageable = static_cast<uint8_t*>(p);
  for (int i = 0; i < kStageSlots; ++i) {
    void* s = nullptr;
    if (hipHostMalloc(&s, kStageBytes, hipHostMallocDefault) != hipSuccess || !s) {
      c.err = "hipHostMalloc of the staging ring failed";
      return AUVM_E_NOMEM;
    }
    c.stage.push_back(static_cast<uint8_t*>(s));
  }
  return AUVM_OK;
}

auvm_status device_alloc_pool(Ctx& c, uint64_t bytes) {
  void* p = nullptr;
  if (hipSetDevice(c.device) != hipSuccess || hipMalloc(&p, bytes) != hipSuccess || !p) {
    c.err = "hipMalloc of the device pool failed";
    return AUVM_E_NOMEM;
  }
  c.pool = static_cast<uint8_t*>(p);
  c.pool_owned = true;
  return AUVM_OK;
}

void release_pool(Ctx& c) {
  if (c.pool_owned && c.pool) {
    if (c.device >= 0) (void)hipSetDevice(c.device);
    (void)hipFree(c.pool);
  }
  c.pool = nullptr;
  c.pool_owned = false;
}

void free_owned(Ctx& c) {
  if (c.device >= 0) (void)hipSetDevice(c.device);
  if (c.pool_owned && c.pool) (void)hipFree(c.pool);
  if (c.host_owned && c.host) (void)hipHostFree(c.host);
  if (c.host_pageable) (void)munmap(c.host_pageable, c.arena_bytes - c.pinned_bytes);
  for (uint8_t* s : c.stage) (void)hipHostFree(s);
  c.stage.clear();
  c.host_pageable = nullptr;
  c.pool = nullptr;
  c.host = nullptr;
  c.pool_owned = c.host_owned = false;
}

}  // namespace auvm
