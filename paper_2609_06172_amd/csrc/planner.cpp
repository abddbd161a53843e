// The prefetch/evict planner.
//
// Input: the kernel--tensor access trace (Sec. IV-D), tensor sizes, the device
// budget M and the three roofs.  Output: the ordered schedule of transfers,
// evictions and launches, per-kernel roofline classes and residency.
//
// Paper facts this follows: tensor-granular movement of exactly the tensors a
// kernel accesses (Sec. IV-B, IV-E); a roofline that separates compute-,
// memory- and interconnect(CGI)-bound kernels, with proactive prefetch only
// for CGI-bound ones (Sec. III-C, IV-D, IV-E); look-ahead affinity pinning of
// tensors reused by consecutive kernels (Sec. IV-D, IV-E); re-evaluation of
// classes as residency changes (Sec. IV-E); LRU eviction and fault-driven
// migration for the baseline (Sec. II-A, V-A).  Where the paper gives no rule
// (thresholds, victims, placement, look-ahead) the choices are:
//  * class: CGI iff X>0, X*P > F*Bl and X*Bh > B*Bl (with a measured kernel
//    time t: iff X > 0 and X/Bl > t), else COMPUTE iff F*Bh >= B*P, else
//    MEMORY (exact 128-bit products, ties not CGI);
//  * the full method keeps the replacement decisions of farthest-next-use
//    demand paging (the profile knows the future) and moves each fetch of a
//    CGI kernel to the earliest boundary at which its pool window can be
//    vacated, in demand order (integrated prefetching with optimal
//    replacements, issued early); its demand pass prefers victims not used
//    by the previous `guard` kernels, which lets each fetch overlap them;
//  * pool windows are chosen by (-writeback bytes, bucket of the worst
//    victim's next-use distance, -victim bytes, worst next use, -offset)
//    under farthest-next-use victims (the host link carries both directions,
//    so a clean victim is cheaper; next uses within one bucket of kernels
//    count as equally far, so fewer evicted bytes decide among them) and by
//    (worst victim priority, -writeback bytes, -victim bytes, -offset) under
//    LRU; dead values are the best victims and are dropped, not written back.
// Integer arithmetic only, so the schedule is reproducible bit for bit.
#include <algorithm>
#include <cstring>
#include <map>

#include "core.h"

namespace auvm {

namespace {

enum Val : uint8_t { NONE = 0, HOST = 1, DEV_CLEAN = 2, DEV_DIRTY = 3 };

struct Span {
  uint64_t off, end;
  int32_t t;
};

struct Uses {
  std::vector<std::vector<int32_t>> k;     // kernel indices using each tensor
  std::vector<std::vector<uint8_t>> mode;
  std::vector<uint8_t> out;                // live-out: read after the trace ends
  int64_t nu(int32_t t, int64_t kk) const {
    auto& v = k[t];
    auto it = std::lower_bound(v.begin(), v.end(), kk);
    return it == v.end() ? kInf : *it;
  }
  // the value held before kernel kk is read later: by the next use, if it
  // reads, or after the trace for a live-out tensor without further uses
  bool live(int32_t t, int64_t kk) const {
    auto& v = k[t];
    auto it = std::lower_bound(v.begin(), v.end(), kk);
    if (it == v.end()) return out[t] != 0;
    return (mode[t][it - v.begin()] & AUVM_R) != 0;
  }
};

Uses build_uses(const std::vector<Tensor>& T, const std::vector<Kernel>& K) {
  const size_t nT = T.size();
  Uses u;
  u.k.resize(nT);
  u.mode.resize(nT);
  u.out.resize(nT);
  for (size_t t = 0; t < nT; ++t) u.out[t] = (T[t].flags & AUVM_LIVE_OUT) ? 1 : 0;
  for (size_t k = 0; k < K.size(); ++k)
    for (auto& a : K[k].acc) {
      u.k[a.first].push_back(int32_t(k));
      u.mode[a.first].push_back(a.second);
    }
  return u;
}

auvm_sched_entry entry(int op, int32_t t, uint64_t off, uint64_t bytes, int32_t ik, int32_t nk) {
  auvm_sched_entry e;
  std::memset(&e, 0, sizeof e);
  e.op = op;
  e.tensor = t;
  e.dev_off = off;
  e.bytes = bytes;
  e.issue_k = ik;
  e.need_k = nk;
  return e;
}

uint64_t x_missing(const Kernel& k, const std::vector<uint64_t>& size, const std::vector<uint8_t>& val) {
  uint64_t X = 0;
  for (auto& a : k.acc)
    if ((a.second & AUVM_R) && val[a.first] == HOST) X += size[a.first];
  return X;
}

// ------------------------------------------------------------------ pass 1
class Replay {
 public:
  Replay(const std::vector<Tensor>& T, const std::vector<Kernel>& K, uint64_t M, const Roofs& r,
         const auvm_policy& p, bool scan)
      : K_(K), M_(M), roofs_(r), pol_(p), scan_(scan) {
    nT_ = T.size();
    size_.resize(nT_);
    for (size_t t = 0; t < nT_; ++t) size_[t] = T[t].size;
    kinds_.resize(nT_);
    for (size_t t = 0; t < nT_; ++t) kinds_[t] = T[t].kind;
    uses_ = build_uses(T, K);
    belady_ = p.variant == AUVM_T_A_P || p.variant == AUVM_DEMAND_BELADY;
    affinity_ = p.variant == AUVM_T_A || p.variant == AUVM_T_A_P;
    D_ = p.lookahead ? p.lookahead : 1;
    val_.assign(nT_, NONE);
    for (size_t t = 0; t < nT_; ++t) val_[t] = T[t].host_valid0() ? HOST : NONE;
    resident_.assign(nT_, 0);
    off_.assign(nT_, 0);
    lru_.assign(nT_, -1);
    pin_.assign(nT_, -1);
    pf_need_.assign(nT_, -1);
    mark_.assign(nT_, -1);
    last_.assign(nT_, -1);
    guard_ = (p.variant == AUVM_T_A_P && !scan) ? int64_t(p.guard) : 0;
    bucket_ = belady_ ? std::max<int64_t>(1, p.bucket) : 1;
  }

  PlanResult run() {
    PlanResult R;
    const int64_t K = int64_t(K_.size());
    for (int64_t k = 0; k < K; ++k) {
      const Kernel& kd = K_[k];
      R.static_cls.push_back(0);  // filled by the caller
      uint8_t cls = classify(kd.flops, kd.hbm, x_missing(kd, size_, val_), roofs_, kd.time_ns);
      R.dyn_cls.push_back(cls);
      R.counters.class_n[cls]++;
      for (auto& a : kd.acc) mark_[a.first] = k;  // membership in A_k
      // (ii) demand fetch or allocation of every operand that is not resident
      for (auto& a : kd.acc) {
        int32_t t = a.first;
        uint8_t m = a.second;
        if (resident_[t]) continue;
        if ((m & AUVM_R) && val_[t] == NONE)
          throw PlanError{AUVM_E_INVAL, "kernel " + std::to_string(k) + " reads tensor " +
                                            std::to_string(t) + " before any write"};
        auto elig = [&](int32_t u) { return mark_[u] != k && pin_[u] < k; };
        auto guarded = [&](int32_t u) { return elig(u) && last_[u] < k - guard_; };
        uint64_t a_off;
        std::vector<int32_t> victims;
        // a first write of a KV-cache tensor under farthest-next-use victims
        const bool top = belady_ && !(m & AUVM_R) && kinds_[t] == AUVM_KV;
        bool placed = guard_ > 0 && place(t, guarded, k, &a_off, &victims, top);
        if (!placed && !place(t, elig, k, &a_off, &victims, top)) {
          std::fill(pin_.begin(), pin_.end(), -1);
          if (!place(t, elig, k, &a_off, &victims, top)) {
            uint64_t need = 0;
            for (auto& b : kd.acc) need += size_[b.first];
            if (need > M_)
              throw PlanError{AUVM_E_BUDGET, "kernel " + std::to_string(k) + " needs " +
                                                 std::to_string(need) + " B > budget " +
                                                 std::to_string(M_)};
            throw PlanError{AUVM_E_FRAG, "kernel " + std::to_string(k) +
                                             ": no pool window for tensor " + std::to_string(t)};
          }
        }
        for (int32_t u : victims) evict(R, u, k, k);
        insert(t, a_off);
        if (m & AUVM_R) {
          R.schedule.push_back(entry(AUVM_H2D_DEMAND, t, a_off, size_[t], int32_t(k), int32_t(k)));
          R.counters.h2d_demand_n++;
          R.counters.h2d_demand_B += size_[t];
        } else {
          R.schedule.push_back(entry(AUVM_ALLOC, t, a_off, size_[t], int32_t(k), int32_t(k)));
          R.counters.alloc_n++;
        }
        val_[t] = DEV_CLEAN;
        lru_[t] = k;
      }
      // (iii) residency when the kernel launches
      auvm_residency rr;
      rr.k = int32_t(k);
      rr.n_resident = n_res_;
      rr.resident_bytes = used_;
      R.residency.push_back(rr);
      // (iv) launch
      R.schedule.push_back(entry(AUVM_LAUNCH, -1, 0, 0, int32_t(k), int32_t(k)));
      for (auto& a : kd.acc) {
        if (a.second & AUVM_W) val_[a.first] = DEV_DIRTY;
        lru_[a.first] = k;
        last_[a.first] = k;
        pf_need_[a.first] = -1;
      }
      // (v) look-ahead affinity pins
      if (affinity_)
        for (auto& a : kd.acc) {
          int64_t n = uses_.nu(a.first, k + 1);
          if (n != kInf && n - k <= int64_t(pol_.affinity_w)) pin_[a.first] = std::max(pin_[a.first], n);
        }
      // (vi) next-kernel prefetch of the T and T+A steps
      if (scan_) prefetch_scan(R, k);
    }
    return R;
  }

 private:
  int64_t prio(int32_t u, int64_t kp) const {
    if (belady_) return uses_.live(u, kp) ? uses_.nu(u, kp) : kInf;
    return -lru_[u];
  }
  // next-use distance class: uses within the same bucket count as equally far
  int64_t near(int64_t p, int64_t kp) const { return p == kInf ? kInf : (p - kp) / bucket_; }
  bool writes_back(int32_t u, int64_t kp) const {
    return val_[u] == DEV_DIRTY && (pol_.variant == AUVM_DEMAND_LRU || uses_.live(u, kp));
  }

  template <class Elig>
  bool place(int32_t t, Elig elig, int64_t kp, uint64_t* a_out, std::vector<int32_t>* victims,
             bool top = false) {
    const uint64_t s = size_[t];
    victims->clear();
    if (pol_.placement == AUVM_PLACE_IDEAL) {
      if (M_ - used_ >= s) {
        *a_out = 0;
        return true;
      }
      struct C {
        int64_t pr, nb;
        uint64_t wb, sz;
        int32_t u;
      };
      std::vector<C> c;
      for (auto& sp : spans_)
        if (elig(sp.t)) {
          int64_t pr = prio(sp.t, kp);
          c.push_back({pr, near(pr, kp), writes_back(sp.t, kp) ? size_[sp.t] : 0, size_[sp.t], sp.t});
        }
      const bool belady = belady_;
      std::sort(c.begin(), c.end(), [belady](const C& x, const C& y) {
        if (belady) {  // (write-back asc, bucket desc, size desc, next use desc, id)
          if (x.wb != y.wb) return x.wb < y.wb;
          if (x.nb != y.nb) return x.nb > y.nb;
          if (x.sz != y.sz) return x.sz > y.sz;
          if (x.pr != y.pr) return x.pr > y.pr;
          return x.u < y.u;
        }
        if (x.pr != y.pr) return x.pr > y.pr;
        if (x.wb != y.wb) return x.wb < y.wb;
        if (x.sz != y.sz) return x.sz > y.sz;
        return x.u < y.u;
      });
      uint64_t freed = M_ - used_;
      for (auto& x : c) {
        if (freed >= s) break;
        victims->push_back(x.u);
        freed += x.sz;
      }
      if (freed < s) {
        victims->clear();
        return false;
      }
      *a_out = 0;
      return true;
    }
    // pool windows: candidate starts are 0 and the end of every resident
    // span; a first write of a KV-cache tensor (top) also tries the windows
    // flush against the pool's end and against the start of every resident
    // span, and prefers a free window at the highest address, so the
    // long-lived cache packs at the top of the pool and leaves no holes
    // between its tensors for the streamed weights to fragment
    bool found = false;
    int64_t b_pr = 0;
    uint64_t b_wb = 0, b_vb = 0, b_a = 0;
    size_t b_lo = 0, b_hi = 0;
    const size_t n = spans_.size();
    // a: window start; i: the first span ending after a
    auto consider = [&](uint64_t a, size_t i) {
      if (a + s > M_) return;
      int64_t pr = kInf;
      uint64_t wb = 0, vb = 0;
      size_t j = i;
      for (; j < n && spans_[j].off < a + s; ++j) {
        int32_t u = spans_[j].t;
        if (!elig(u)) return;
        pr = std::min(pr, prio(u, kp));
        if (writes_back(u, kp)) wb += size_[u];
        vb += size_[u];
      }
      bool better;
      if (!found) {
        better = true;
      } else if (top) {      // (-writeback bytes, free, bucket of worst next use, -victim bytes, worst next use, offset)
        const int64_t nb = near(pr, kp), bnb = near(b_pr, kp);
        const bool fr = vb == 0, bfr = b_vb == 0;
        better = wb < b_wb ||
                 (wb == b_wb &&
                  (fr > bfr ||
                   (fr == bfr &&
                    (nb > bnb ||
                     (nb == bnb && (vb < b_vb || (vb == b_vb && (pr > b_pr || (pr == b_pr && a > b_a)))))))));
      } else if (belady_) {  // (-writeback bytes, bucket of worst next use, -victim bytes, worst next use)
        const int64_t nb = near(pr, kp), bnb = near(b_pr, kp);
        better = wb < b_wb ||
                 (wb == b_wb && (nb > bnb || (nb == bnb && (vb < b_vb || (vb == b_vb && pr > b_pr)))));
      } else {               // (worst priority, -writeback bytes, -victim bytes)
        better = pr > b_pr || (pr == b_pr && (wb < b_wb || (wb == b_wb && vb < b_vb)));
      }
      if (better) {
        found = true;
        b_pr = pr;
        b_wb = wb;
        b_vb = vb;
        b_a = a;
        b_lo = i;
        b_hi = j;
      }
    };
    for (size_t i = 0; i <= n; ++i) consider(i == 0 ? 0 : spans_[i - 1].end, i);
    if (top) {
      auto first_after = [&](uint64_t a) {
        return size_t(std::upper_bound(spans_.begin(), spans_.end(), a,
                                       [](uint64_t v, const Span& x) { return v < x.end; }) -
                      spans_.begin());
      };
      if (M_ >= s) consider(M_ - s, first_after(M_ - s));
      for (size_t j = 0; j < n; ++j)
        if (spans_[j].off >= s) consider(spans_[j].off - s, first_after(spans_[j].off - s));
    }
    if (!found) return false;
    for (size_t j = b_lo; j < b_hi; ++j) victims->push_back(spans_[j].t);
    *a_out = b_a;
    return true;
  }

  void insert(int32_t t, uint64_t a) {
    resident_[t] = 1;
    off_[t] = a;
    used_ += size_[t];
    n_res_++;
    Span sp{a, a + size_[t], t};
    if (pol_.placement == AUVM_PLACE_IDEAL) {
      spans_.push_back(sp);
      return;
    }
    auto it = std::lower_bound(spans_.begin(), spans_.end(), sp,
                               [](const Span& x, const Span& y) { return x.off < y.off; });
    spans_.insert(it, sp);
  }

  void remove(int32_t t) {
    resident_[t] = 0;
    used_ -= size_[t];
    n_res_--;
    for (size_t i = 0; i < spans_.size(); ++i)
      if (spans_[i].t == t) {
        spans_.erase(spans_.begin() + i);
        return;
      }
  }

  void evict(PlanResult& R, int32_t u, int64_t k, int64_t kp) {
    if (val_[u] == DEV_DIRTY) {
      if (pol_.variant == AUVM_DEMAND_LRU || uses_.live(u, kp)) {
        R.schedule.push_back(entry(AUVM_D2H_WRITEBACK, u, off_[u], size_[u], int32_t(k), -1));
        R.counters.d2h_wb_n++;
        R.counters.d2h_wb_B += size_[u];
        val_[u] = HOST;
      } else {
        R.schedule.push_back(entry(AUVM_DROP, u, off_[u], size_[u], int32_t(k), -1));
        R.counters.drop_n++;
        val_[u] = NONE;
      }
    } else {
      R.schedule.push_back(entry(AUVM_DROP, u, off_[u], size_[u], int32_t(k), -1));
      R.counters.drop_n++;
      val_[u] = HOST;
    }
    if (pf_need_[u] >= 0) {
      R.counters.useless_prefetch_n++;
      R.counters.useless_prefetch_B += size_[u];
      pf_need_[u] = -1;
    }
    remove(u);
  }

  void prefetch_scan(PlanResult& R, int64_t k) {
    const int64_t K = int64_t(K_.size());
    const int64_t jmax = std::min(K - 1, k + int64_t(D_));
    std::vector<int32_t> protected_list;
    ++scan_id_;
    for (int64_t j = k + 1; j <= jmax; ++j) {
      for (auto& a : K_[j].acc) prot_[a.first] = scan_id_;
      std::vector<int32_t> cands;
      for (auto& a : K_[j].acc)
        if ((a.second & AUVM_R) && val_[a.first] == HOST && uses_.live(a.first, k + 1))
          cands.push_back(a.first);
      if (cands.empty()) continue;
      auto elig = [&](int32_t u) { return prot_[u] != scan_id_ && pin_[u] < k + 1; };
      for (int32_t t : cands) {
        uint64_t a_off;
        std::vector<int32_t> victims;
        if (!place(t, elig, k + 1, &a_off, &victims)) return;
        for (int32_t u : victims) evict(R, u, k, k + 1);
        insert(t, a_off);
        R.schedule.push_back(entry(AUVM_H2D_PREFETCH, t, a_off, size_[t], int32_t(k), int32_t(j)));
        R.counters.h2d_prefetch_n++;
        R.counters.h2d_prefetch_B += size_[t];
        val_[t] = DEV_CLEAN;
        lru_[t] = k;
        pf_need_[t] = j;
      }
    }
  }

 public:
  void init_scan_marks() { prot_.assign(nT_, -1); }

 private:
  const std::vector<Kernel>& K_;
  uint64_t M_;
  Roofs roofs_;
  auvm_policy pol_;
  bool scan_;
  size_t nT_ = 0;
  std::vector<uint64_t> size_;
  Uses uses_;
  bool belady_ = false, affinity_ = false;
  uint32_t D_ = 1;
  std::vector<uint8_t> val_, resident_;
  std::vector<uint64_t> off_;
  std::vector<int64_t> lru_, pin_, pf_need_, mark_, prot_, last_;
  int64_t guard_ = 0, bucket_ = 1;
  std::vector<uint32_t> kinds_;
  int64_t scan_id_ = 0;
  std::vector<Span> spans_;  // resident windows sorted by offset (insertion order for IDEAL)
  uint64_t used_ = 0;
  int32_t n_res_ = 0;
};

// ------------------------------------------------------------------ pass 2
struct Interval {
  int32_t t;
  uint64_t off, end;
  int64_t arr, dep, lastacc;
};

struct Unit {
  std::vector<auvm_sched_entry> evictions;
  auvm_sched_entry e;
  int64_t issue;
  int64_t prev_dep;
};

PlanResult retime(const std::vector<Tensor>& T, const std::vector<Kernel>& K, const Roofs& roofs,
                  uint32_t lookahead, const PlanResult& base) {
  const size_t nT = T.size();
  const int64_t nK = int64_t(K.size());
  std::vector<uint64_t> size(nT);
  for (size_t t = 0; t < nT; ++t) size[t] = T[t].size;
  Uses uses = build_uses(T, K);

  // demand timeline: placement units per boundary, residency intervals
  std::vector<std::vector<Unit>> units(nK);
  std::vector<auvm_sched_entry> pending;
  std::vector<Interval> iv;
  std::vector<int64_t> cur(nT, -1), gone(nT, 0);
  for (const auto& e : base.schedule) {
    if (e.op == AUVM_D2H_WRITEBACK || e.op == AUVM_DROP) {
      pending.push_back(e);
      iv[cur[e.tensor]].dep = e.issue_k;
      cur[e.tensor] = -1;
      gone[e.tensor] = e.issue_k;
    } else if (e.op == AUVM_H2D_DEMAND || e.op == AUVM_ALLOC) {
      cur[e.tensor] = int64_t(iv.size());
      iv.push_back({e.tensor, e.dev_off, e.dev_off + e.bytes, e.issue_k, kInf, e.issue_k});
      units[e.issue_k].push_back({pending, e, e.issue_k, gone[e.tensor]});
      pending.clear();
    } else if (e.op == AUVM_LAUNCH) {
      for (auto& a : K[e.issue_k].acc) iv[cur[a.first]].lastacc = e.issue_k;
    }
  }
  std::vector<int64_t> left;  // interval indices that end, by departure
  for (size_t i = 0; i < iv.size(); ++i)
    if (iv[i].dep != kInf) left.push_back(int64_t(i));
  std::stable_sort(left.begin(), left.end(), [&](int64_t a, int64_t b) { return iv[a].dep < iv[b].dep; });
  std::vector<int64_t> deps(left.size());
  for (size_t i = 0; i < left.size(); ++i) deps[i] = iv[left[i]].dep;

  // earliest issue boundary of each CGI fetch, in demand order
  std::vector<std::vector<std::pair<int64_t, size_t>>> early(nK);  // (boundary j, unit index)
  int64_t prev = 0;
  std::vector<int64_t> occ;
  for (int64_t j = 1; j < nK; ++j) {
    if (base.dyn_cls[j] != AUVM_CLS_CGI) continue;
    for (size_t ui = 0; ui < units[j].size(); ++ui) {
      Unit& u = units[j][ui];
      if (u.e.op != AUVM_H2D_DEMAND) continue;
      uint64_t a = u.e.dev_off, end = u.e.dev_off + u.e.bytes;
      int64_t lo = std::max<int64_t>({prev, lookahead ? j - int64_t(lookahead) : 0, u.prev_dep, 0});
      size_t i0 = std::upper_bound(deps.begin(), deps.end(), lo) - deps.begin();
      size_t i1 = std::upper_bound(deps.begin(), deps.end(), j) - deps.begin();
      occ.clear();
      for (size_t i = i0; i < i1; ++i) {
        const Interval& x = iv[left[i]];
        if (x.off < end && a < x.end) occ.push_back(left[i]);
      }
      int64_t k = lo;
      for (;;) {
        int64_t m = -1;
        for (int64_t i : occ)
          if (iv[i].dep > k) m = std::max(m, iv[i].lastacc);
        if (m <= k) break;
        k = m;
      }
      if (k < j) {
        u.issue = k;
        early[k].push_back({j, ui});
        prev = k;
      }
    }
  }

  // the new timeline
  PlanResult R;
  R.static_cls = base.static_cls;
  std::vector<uint8_t> val(nT);
  for (size_t t = 0; t < nT; ++t) val[t] = T[t].host_valid0() ? HOST : NONE;
  std::vector<int64_t> where(nT, -1);
  std::map<uint64_t, int32_t> by_off;  // resident windows
  uint64_t used = 0;
  int32_t n_res = 0;

  auto evict = [&](int32_t t, int64_t k) {
    uint64_t o = uint64_t(where[t]);
    if (val[t] == DEV_DIRTY && uses.live(t, k + 1)) {
      R.schedule.push_back(entry(AUVM_D2H_WRITEBACK, t, o, size[t], int32_t(k), -1));
      R.counters.d2h_wb_n++;
      R.counters.d2h_wb_B += size[t];
      val[t] = HOST;
    } else {
      R.schedule.push_back(entry(AUVM_DROP, t, o, size[t], int32_t(k), -1));
      R.counters.drop_n++;
      val[t] = val[t] == DEV_DIRTY ? NONE : HOST;
    }
    used -= size[t];
    n_res--;
    by_off.erase(o);
    where[t] = -1;
  };
  auto put = [&](const Unit& u, int64_t k, int kind, int32_t need) {
    int32_t t = u.e.tensor;
    uint64_t a = u.e.dev_off, b = u.e.bytes;
    auto it = by_off.lower_bound(a);
    if (it != by_off.begin()) {
      auto p = std::prev(it);
      if (p->first + size[p->second] > a) throw PlanError{AUVM_E_INVAL, "retimed window still occupied"};
    }
    if (it != by_off.end() && it->first < a + b) throw PlanError{AUVM_E_INVAL, "retimed window still occupied"};
    where[t] = int64_t(a);
    by_off[a] = t;
    used += b;
    n_res++;
    R.schedule.push_back(entry(kind, t, a, b, int32_t(k), need));
    if (kind == AUVM_H2D_PREFETCH) {
      R.counters.h2d_prefetch_n++;
      R.counters.h2d_prefetch_B += b;
    } else if (kind == AUVM_H2D_DEMAND) {
      R.counters.h2d_demand_n++;
      R.counters.h2d_demand_B += b;
    } else {
      R.counters.alloc_n++;
    }
    val[t] = DEV_CLEAN;
  };

  for (int64_t k = 0; k < nK; ++k) {
    const Kernel& kd = K[k];
    uint8_t cls = classify(kd.flops, kd.hbm, x_missing(kd, size, val), roofs, kd.time_ns);
    R.dyn_cls.push_back(cls);
    R.counters.class_n[cls]++;
    for (const Unit& u : units[k]) {
      if (u.issue < k) continue;  // fetched ahead
      for (const auto& e : u.evictions)
        if (where[e.tensor] == int64_t(e.dev_off)) evict(e.tensor, k);
      put(u, k, u.e.op, int32_t(k));
    }
    auvm_residency rr;
    rr.k = int32_t(k);
    rr.n_resident = n_res;
    rr.resident_bytes = used;
    R.residency.push_back(rr);
    R.schedule.push_back(entry(AUVM_LAUNCH, -1, 0, 0, int32_t(k), int32_t(k)));
    for (auto& a : kd.acc)
      if (a.second & AUVM_W) val[a.first] = DEV_DIRTY;
    for (auto& ju : early[k]) {
      const Unit& u = units[ju.first][ju.second];
      uint64_t a = u.e.dev_off, end = a + u.e.bytes;
      std::vector<int32_t> over;
      auto it = by_off.lower_bound(a);
      if (it != by_off.begin()) {
        auto p = std::prev(it);
        if (p->first + size[p->second] > a) over.push_back(p->second);
      }
      for (; it != by_off.end() && it->first < end; ++it) over.push_back(it->second);
      for (int32_t t : over) evict(t, k);
      put(u, k, AUVM_H2D_PREFETCH, int32_t(ju.first));
    }
  }
  return R;
}

PlanResult plan_objects(const std::vector<Tensor>& T, const std::vector<Kernel>& K, uint64_t M,
                        const Roofs& roofs, auvm_policy pol);

}  // namespace

PlanResult plan(const std::vector<Tensor>& T, const std::vector<Kernel>& K, uint64_t M,
                const Roofs& roofs, const auvm_policy& pol) {
  if (pol.variant > AUVM_T_A_P) throw PlanError{AUVM_E_INVAL, "unknown policy variant"};
  if (pol.object_bytes) return plan_objects(T, K, M, roofs, pol);
  if (pol.variant == AUVM_T_A_P && pol.placement == AUVM_PLACE_IDEAL)
    throw PlanError{AUVM_E_INVAL, "the full method retimes fetches into physical pool windows"};
  bool scan = pol.variant == AUVM_T || pol.variant == AUVM_T_A;
  Replay r(T, K, M, roofs, pol, scan);
  r.init_scan_marks();
  PlanResult base = r.run();
  for (size_t k = 0; k < K.size(); ++k) {
    uint64_t X = 0;
    for (auto& a : K[k].acc)
      if (a.second & AUVM_R) X += T[a.first].size;
    base.static_cls[k] = classify(K[k].flops, K[k].hbm, X, roofs, K[k].time_ns);
  }
  if (pol.variant != AUVM_T_A_P) return base;
  return retime(T, K, roofs, pol.lookahead, base);
}

namespace {

// Object granularity (the contrast of Sec. III-B, Fig. 3): the policy plans
// the allocator's blocks, then each block move is expanded to its members.
PlanResult plan_objects(const std::vector<Tensor>& T, const std::vector<Kernel>& K, uint64_t M,
                        const Roofs& roofs, auvm_policy pol) {
  const uint64_t ob = pol.object_bytes;
  pol.object_bytes = 0;
  const size_t nT = T.size();
  // blocks: consecutive tensors until the next would pass object_bytes
  std::vector<std::vector<int32_t>> objs;
  {
    std::vector<int32_t> cur;
    uint64_t cb = 0;
    for (size_t t = 0; t < nT; ++t) {
      if (!cur.empty() && cb + T[t].size > ob) {
        objs.push_back(cur);
        cur.clear();
        cb = 0;
      }
      cur.push_back(int32_t(t));
      cb += T[t].size;
    }
    if (!cur.empty()) objs.push_back(cur);
  }
  const size_t nO = objs.size();
  std::vector<int32_t> obj_of(nT);
  std::vector<uint64_t> rel(nT);
  std::vector<Tensor> OT(nO);
  std::vector<uint8_t> valid0(nO, 0);
  for (size_t o = 0; o < nO; ++o) {
    uint64_t r = 0;
    bool out = false;
    for (int32_t t : objs[o]) {
      obj_of[t] = int32_t(o);
      rel[t] = r;
      r += T[t].size;
      if (T[t].host_valid0()) valid0[o] = 1;
      if (T[t].flags & AUVM_LIVE_OUT) out = true;
    }
    Tensor& x = OT[o];
    x.bytes = x.size = r;
    x.dtype = T[objs[o][0]].dtype;
    x.kind = valid0[o] ? uint32_t(AUVM_PARAM) : T[objs[o][0]].kind;
    x.flags = out ? uint32_t(AUVM_LIVE_OUT) : 0u;
  }
  // the coarse trace: a block's first access by a writing kernel needs no
  // fetch; every later access reads the block
  std::vector<Kernel> OK(K.size());
  std::vector<uint8_t> touched(nO, 0);
  for (size_t k = 0; k < K.size(); ++k) {
    Kernel& x = OK[k];
    x.op = K[k].op;
    std::copy(K[k].shape, K[k].shape + 8, x.shape);
    x.flops = K[k].flops;
    x.hbm = K[k].hbm;
    x.time_ns = K[k].time_ns;
    x.layer = K[k].layer;
    for (auto& a : K[k].acc) {
      const int32_t o = obj_of[a.first];
      auto it = std::find_if(x.acc.begin(), x.acc.end(), [&](const std::pair<int32_t, uint8_t>& b) {
        return b.first == o;
      });
      if (it == x.acc.end())
        x.acc.emplace_back(o, a.second);
      else
        it->second |= a.second;
    }
    for (auto& a : x.acc) {
      if (touched[a.first] || valid0[a.first]) a.second = uint8_t(AUVM_R | (a.second & AUVM_W));
      touched[a.first] = 1;
    }
  }
  PlanResult base = plan(OT, OK, M, roofs, pol);

  // expansion to member tensors, in each block's window
  PlanResult R;
  R.static_cls = base.static_cls;
  R.dyn_cls = base.dyn_cls;
  PlanCounters& C = R.counters;
  for (int i = 0; i < 3; ++i) C.class_n[i] = base.counters.class_n[i];
  constexpr uint8_t EMPTY = 4;   // resident, no value yet
  std::vector<uint8_t> val(nT), res(nT, 0);
  for (size_t t = 0; t < nT; ++t) val[t] = T[t].host_valid0() ? HOST : NONE;
  std::vector<uint64_t> pending(nT, 0);   // bytes of a member fetch not yet read
  int32_t n_res = 0;
  uint64_t used = 0;
  auto useless = [&](int32_t t) {
    if (pending[t]) {
      ++C.useless_prefetch_n;
      C.useless_prefetch_B += pending[t];
      pending[t] = 0;
    }
  };
  for (const auvm_sched_entry& e : base.schedule) {
    if (e.op == AUVM_LAUNCH) {
      auvm_residency rr;
      rr.k = e.issue_k;
      rr.n_resident = n_res;
      rr.resident_bytes = used;
      R.residency.push_back(rr);
      R.schedule.push_back(e);
      for (auto& a : K[e.issue_k].acc) {
        const int32_t t = a.first;
        if ((a.second & AUVM_R) && (val[t] == NONE || val[t] == EMPTY))
          throw PlanError{AUVM_E_INVAL, "kernel " + std::to_string(e.issue_k) + " reads tensor " +
                                            std::to_string(t) + " before any write"};
        if (pending[t]) {
          if (a.second & AUVM_R)
            pending[t] = 0;
          else
            useless(t);
        }
        if (a.second & AUVM_W) val[t] = DEV_DIRTY;
      }
      continue;
    }
    for (int32_t t : objs[e.tensor]) {
      const uint64_t a = e.dev_off + rel[t];
      const uint64_t s = T[t].size;
      if (e.op == AUVM_H2D_PREFETCH || e.op == AUVM_H2D_DEMAND || e.op == AUVM_ALLOC) {
        res[t] = 1;
        ++n_res;
        used += s;
        if (e.op != AUVM_ALLOC && val[t] == HOST) {
          R.schedule.push_back(entry(e.op, t, a, s, e.issue_k, e.need_k));
          if (e.op == AUVM_H2D_PREFETCH) {
            ++C.h2d_prefetch_n;
            C.h2d_prefetch_B += s;
          } else {
            ++C.h2d_demand_n;
            C.h2d_demand_B += s;
          }
          pending[t] = s;
          val[t] = DEV_CLEAN;
        } else {
          R.schedule.push_back(entry(AUVM_ALLOC, t, a, s, e.issue_k, e.need_k));
          ++C.alloc_n;
          val[t] = EMPTY;
        }
      } else {
        res[t] = 0;
        --n_res;
        used -= s;
        useless(t);
        if (e.op == AUVM_D2H_WRITEBACK && val[t] == DEV_DIRTY) {
          R.schedule.push_back(entry(AUVM_D2H_WRITEBACK, t, a, s, e.issue_k, -1));
          ++C.d2h_wb_n;
          C.d2h_wb_B += s;
          val[t] = HOST;
        } else {
          R.schedule.push_back(entry(AUVM_DROP, t, a, s, e.issue_k, -1));
          ++C.drop_n;
          val[t] = val[t] == DEV_CLEAN ? HOST : NONE;
        }
      }
    }
  }
  for (size_t t = 0; t < nT; ++t) useless(int32_t(t));
  return R;
}

}  // namespace

}  // namespace auvm
