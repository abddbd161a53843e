"""Reference replay of the tensor-granular, roofline-gated prefetch/evict policy.

What the paper fixes (Sec. IV):
* one profiling pass yields kernel--tensor access pairs, and at run time the
  executor prefetches the tensors the upcoming kernel needs (Sec. IV-D);
* a roofline analysis classifies each kernel as GPU-compute-, GPU-memory- or
  CPU--GPU-interconnect (CGI) bound, and only CGI-bound kernels get proactive
  prefetching; the others are left to on-demand migration (Sec. IV-D, IV-E);
* tensors reused by consecutive kernels are pinned on the device for their
  reuse window (look-ahead affinity, Sec. IV-D, IV-E);
* a runtime monitor re-evaluates classes as evictions change behaviour
  (Sec. IV-E);
* the baseline is demand migration with least-recently-used eviction
  (Sec. II-A, Sec. V-A), and oversubscription factor = allocated bytes over
  device capacity (Sec. II-A).

The paper gives no formulas, thresholds, tie rules, look-ahead depth or victim
rule for its own policy.  The readings used here (each listed in the design
notes) are:

* sizes are rounded up to 256 bytes; the device is one pool of M bytes;
* static class: COMPUTE iff F*Bh >= B*P else MEMORY;  a kernel is CGI iff the
  bytes X of its read operands that are host-resident satisfy X > 0,
  X*P > F*Bl and X*Bh > B*Bl (link time exceeds both device roof times);
  exact integer cross-products, ties not CGI;
* victims for the full method are chosen by farthest next use (Belady/MIN,
  possible because the profile gives the future), dead values first, and a
  window that needs no write-back is preferred over one that does (the host
  link is shared by both directions); LRU for the demand baseline and the
  T / T+A ablation steps;
* placement picks a window of the pool whose resident tensors may all be
  evicted, maximising (-writeback bytes, bucket of the worst victim's
  next-use distance, -victim bytes, worst victim's next use, -offset) under
  farthest-next-use, where uses within the same ``bucket`` kernels count as
  equally far so that, among them, the window evicting fewer bytes wins
  (bucket 1 is exact farthest-next-use), and (worst victim priority,
  -writeback bytes, -victim bytes, -offset) under LRU;
* the ablation steps T and T+A prefetch, after each launch, the missing live
  read operands of the next kernel only (look-ahead 1), with LRU victims, and
  stop at the first operand that cannot be placed; T+A adds the affinity
  pins;
* the full method (T+A+P) is two passes.  The first is the demand timeline
  with farthest-next-use victims, affinity pins and a victim guard (a victim
  preferably unused by the ``guard`` kernels before the demand point).  The
  second (``_retime``) keeps every replacement of the first and moves each
  fetch of a CGI kernel to the earliest boundary at which every tensor that
  held its window has had its last access, in demand order: the
  "conservative" integrated prefetching/caching strategy of Cao, Felten,
  Karlin and Li (optimal replacements, each fetch as early as possible).
  Fetches of kernels that are not CGI stay at their kernel (on-demand).

Integer arithmetic only; no state outside the function.  Slow and plain.
"""
from bisect import bisect_left, bisect_right

from workloads.format import (ALIGN, CLS_CGI, CLS_COMPUTE, CLS_MEMORY,
                              KIND_KV, KIND_PARAM, MODE_R, MODE_W, PLACE_IDEAL,
                              PLACE_POOL, S_ALLOC, S_D2H_WRITEBACK, S_DROP,
                              S_H2D_DEMAND, S_H2D_PREFETCH, S_LAUNCH,
                              VAR_DEMAND_BELADY, VAR_DEMAND_LRU, VAR_T,
                              VAR_T_A, VAR_T_A_P)

from .costs import kernel_cost

INF = 1 << 62
NONE, HOST, DEV_CLEAN, DEV_DIRTY = 0, 1, 2, 3
E_INVAL, E_BUDGET, E_FRAG = -1, -3, -4

DEFAULT_ROOFS = (2_500_000_000_000_000, 8_000_000_000_000, 64_000_000_000)


class PlanError(Exception):
    def __init__(self, code, msg):
        super().__init__(msg)
        self.code = code


def aligned(n):
    return (n + ALIGN - 1) // ALIGN * ALIGN


def merge_operands(operands):
    """Distinct tensor ids in first-occurrence order, modes OR-ed together."""
    order, modes = [], {}
    for t, m in operands:
        if t not in modes:
            order.append(t)
            modes[t] = 0
        modes[t] |= m
    return [(t, modes[t]) for t in order]


def classify(F, B, X, roofs, t_ns=0):
    """Roofline class of a kernel with X host-resident read bytes (Sec. IV-B).

    Analytic (t_ns = 0): CGI iff moving X over the link takes longer than both
    the compute roof F/P and the HBM roof B/Bh.  With a measured kernel time
    t_ns > 0 (the runtime monitor's re-classification, Sec. IV, Online
    Executor): CGI iff the link time X/Bl exceeds it.  Otherwise COMPUTE iff
    F/P >= B/Bh, else MEMORY.  Exact integer products.
    """
    P, Bh, Bl = roofs
    if t_ns > 0:
        if X > 0 and X * 10**9 > t_ns * Bl:
            return CLS_CGI
    elif X > 0 and X * P > F * Bl and X * Bh > B * Bl:
        return CLS_CGI
    return CLS_COMPUTE if F * Bh >= B * P else CLS_MEMORY


class Result:
    def __init__(self):
        self.schedule = []       # (op, tensor, dev_off, bytes, issue_k, need_k)
        self.residency = []      # (k, n_resident, resident_bytes) after demand, before launch
        self.static_cls = []
        self.dyn_cls = []
        self.costs = []          # (F, B)
        self.counters = dict(h2d_prefetch_n=0, h2d_prefetch_B=0, h2d_demand_n=0,
                             h2d_demand_B=0, d2h_wb_n=0, d2h_wb_B=0, drop_n=0,
                             alloc_n=0, useless_prefetch_n=0, useless_prefetch_B=0,
                             class_n=[0, 0, 0])


def plan(tensors, kernels, M, roofs=DEFAULT_ROOFS, variant=VAR_T_A_P, lookahead=0,
         affinity_w=1, placement=PLACE_POOL, guard=None, bucket=None, object_bytes=0):
    """Replay the policy.

    tensors: list of dicts with keys nbytes, dtype, kind, host_init and
             optionally live_out (the final value is read after the trace).
    kernels: list of dicts with keys op, shape, operands [(tid, mode)],
             optional flops / hbm_bytes (0 or missing: analytic cost) and
             time_ns (a measured kernel time; 0 or missing: the analytic
             roofline decides the CGI class, see ``classify``).
    Returns a Result; raises PlanError on E_INVAL / E_BUDGET / E_FRAG.

    The full method (T+A+P) is two passes: the demand timeline with
    farthest-next-use victims and affinity pins, then every fetch of a CGI
    kernel is moved to the earliest boundary at which its window can be
    vacated (``_retime``).  In its demand pass a victim must, if any window
    allows it, not have been used by the ``guard`` kernels before the demand
    point, so that the moved fetch overlaps those kernels (default 4; 0 gives
    plain farthest-next-use).  The other variants are one pass.

    object_bytes > 0 plans at object granularity instead (``plan_objects``).
    """
    if object_bytes:
        return plan_objects(tensors, kernels, M, object_bytes, roofs=roofs, variant=variant,
                            lookahead=lookahead, affinity_w=affinity_w, placement=placement,
                            guard=guard, bucket=bucket)
    if variant == VAR_T_A_P and placement == PLACE_IDEAL:
        raise PlanError(E_INVAL, "the full method retimes fetches into physical pool windows")
    if guard is None:
        guard = 4 if variant == VAR_T_A_P else 0
    if bucket is None:
        bucket = 32 if variant == VAR_T_A_P else 1
    if variant != VAR_T_A_P:
        return _replay(tensors, kernels, M, roofs, variant, lookahead, affinity_w,
                       placement, scan=variant in (VAR_T, VAR_T_A), guard=0,
                       bucket=bucket if variant == VAR_DEMAND_BELADY else 1)
    base = _replay(tensors, kernels, M, roofs, variant, lookahead, affinity_w,
                   placement, scan=False, guard=guard, bucket=bucket)
    return _retime(tensors, kernels, M, roofs, lookahead, base)


def _access(tensors, kernels):
    """Merged access lists, per-tensor uses (ascending) and their modes."""
    A = [merge_operands(k["operands"]) for k in kernels]
    uses = [[] for _ in tensors]
    use_mode = [[] for _ in tensors]
    for k, a in enumerate(A):
        for t, m in a:
            uses[t].append(k)
            use_mode[t].append(m)
    return A, uses, use_mode


def _replay(tensors, kernels, M, roofs, variant, lookahead, affinity_w, placement, scan, guard,
            bucket):
    nT, K = len(tensors), len(kernels)
    size = [aligned(t["nbytes"]) for t in tensors]
    dtypes = [t["dtype"] for t in tensors]
    raw = [t["nbytes"] for t in tensors]
    res = Result()
    belady = variant in (VAR_T_A_P, VAR_DEMAND_BELADY)
    affinity = variant in (VAR_T_A, VAR_T_A_P)
    D = lookahead if lookahead else 1       # T and T+A look at the next kernel

    # ---- access lists, uses and costs
    A, uses, use_mode = _access(tensors, kernels)
    Aset = [set(t for t, _ in a) for a in A]
    FB = []
    for k, kd in enumerate(kernels):
        F, B = kd.get("flops", 0), kd.get("hbm_bytes", 0)
        if (F == 0 or B == 0) and not kd.get("resolved"):
            aF, aB = kernel_cost(kd["op"], kd["shape"], kd["operands"], dtypes, raw)
            F = F or aF
            B = B or aB
        FB.append((F, B))
    res.costs = FB
    tns = [kd.get("time_ns", 0) for kd in kernels]

    def nu(t, k):
        i = bisect_left(uses[t], k)
        return uses[t][i] if i < len(uses[t]) else INF

    def live(t, k):
        """The value held before kernel k is read later: by the next use if it
        reads, or after the trace when the tensor is live-out."""
        i = bisect_left(uses[t], k)
        if i == len(uses[t]):
            return bool(tensors[t].get("live_out", False))
        return bool(use_mode[t][i] & MODE_R)

    for k in range(K):
        F, B = FB[k]
        X = sum(size[t] for t, m in A[k] if m & MODE_R)
        res.static_cls.append(classify(F, B, X, roofs, tns[k]))

    # ---- state
    val = [HOST if (t["kind"] == KIND_PARAM or t["host_init"]) else NONE for t in tensors]
    off = {}                       # resident tensor -> device offset
    last = [-1] * nT
    lru = [-1] * nT
    pin = [-1] * nT
    pf_need = [None] * nT          # pending prefetch (not yet used)
    C = res.counters
    used_bytes = [0]

    def x_missing(j):
        return sum(size[t] for t, m in A[j] if (m & MODE_R) and val[t] == HOST)

    def prio(u, kp):
        if belady:
            return nu(u, kp) if live(u, kp) else INF
        return -lru[u]

    def near(p, kp):
        """Next-use distance class: uses within the same bucket count as equally far."""
        return INF if p == INF else (p - kp) // bucket

    def writes_back(u, kp):
        return val[u] == DEV_DIRTY and (variant == VAR_DEMAND_LRU or live(u, kp))

    def place(t, eligible, kp, top=False):
        """Returns (offset, victims) or None.  top: a first write of a
        KV-cache tensor, which also tries the windows flush against the
        pool's end and against the start of every resident tensor, and takes
        a free window at the highest address (the long-lived cache packs at
        the top of the pool, with no holes between its tensors)."""
        s = size[t]
        if placement == PLACE_IDEAL:
            if M - used_bytes[0] >= s:
                return 0, []
            if belady:
                order = lambda u: (size[u] if writes_back(u, kp) else 0, -near(prio(u, kp), kp),
                                   -size[u], -prio(u, kp), u)
            else:
                order = lambda u: (-prio(u, kp), size[u] if writes_back(u, kp) else 0, -size[u], u)
            cands = sorted((u for u in off if eligible(u)), key=order)
            freed, chosen = M - used_bytes[0], []
            for u in cands:
                if freed >= s:
                    break
                chosen.append(u)
                freed += size[u]
            if freed < s:
                return None
            return 0, chosen
        spans = sorted((o, o + size[u], u) for u, o in off.items())
        starts_ = [sp[0] for sp in spans]
        ends_ = [sp[1] for sp in spans]
        cands = set([0] + ends_)
        if top:
            cands |= set(o - s for o in starts_ if o >= s)
            if M >= s:
                cands.add(M - s)
        cand_starts = sorted(cands)
        best, best_key = None, None
        for a in cand_starts:
            if a + s > M:
                continue
            lo = bisect_right(ends_, a)          # first span ending after a
            hi = bisect_left(starts_, a + s)     # first span starting at or after a+s
            over = [spans[i][2] for i in range(lo, hi)]
            if not all(eligible(u) for u in over):
                continue
            minpr = min((prio(u, kp) for u in over), default=INF)
            wb = sum(size[u] for u in over if writes_back(u, kp))
            vb = sum(size[u] for u in over)
            if top:
                key = (-wb, vb == 0, near(minpr, kp), -vb, minpr, a)
            elif belady:
                key = (-wb, near(minpr, kp), -vb, minpr, -a)
            else:
                key = (minpr, -wb, -vb, -a)
            if best_key is None or key > best_key:
                best, best_key = (a, over), key
        return best

    def evict(u, k, kp):
        if val[u] == DEV_DIRTY:
            if variant == VAR_DEMAND_LRU or live(u, kp):
                res.schedule.append((S_D2H_WRITEBACK, u, off[u], size[u], k, -1))
                C["d2h_wb_n"] += 1
                C["d2h_wb_B"] += size[u]
                val[u] = HOST
            else:
                res.schedule.append((S_DROP, u, off[u], size[u], k, -1))
                C["drop_n"] += 1
                val[u] = NONE
        else:
            res.schedule.append((S_DROP, u, off[u], size[u], k, -1))
            C["drop_n"] += 1
            val[u] = HOST
        if pf_need[u] is not None:
            C["useless_prefetch_n"] += 1
            C["useless_prefetch_B"] += size[u]
            pf_need[u] = None
        del off[u]
        used_bytes[0] -= size[u]

    for k in range(K):
        F, B = FB[k]
        cls = classify(F, B, x_missing(k), roofs, tns[k])
        res.dyn_cls.append(cls)
        C["class_n"][cls] += 1
        # (ii) demand fetch / allocation of the kernel's operands
        for t, m in A[k]:
            if t in off:
                continue
            if (m & MODE_R) and val[t] == NONE:
                raise PlanError(E_INVAL, f"kernel {k} reads tensor {t} before any write")

            def elig(u, k=k):
                return u not in Aset[k] and pin[u] < k

            def elig_guarded(u, k=k):
                return elig(u) and last[u] < k - guard
            top = belady and not (m & MODE_R) and tensors[t]["kind"] == KIND_KV
            r = place(t, elig_guarded, k, top) if guard else None
            if r is None:
                r = place(t, elig, k, top)
            if r is None:
                for u in range(nT):
                    pin[u] = -1
                r = place(t, elig, k, top)
                if r is None:
                    need = sum(size[u] for u, _ in A[k])
                    if need > M:
                        raise PlanError(E_BUDGET, f"kernel {k} needs {need} > budget {M}")
                    raise PlanError(E_FRAG, f"kernel {k}: no window for tensor {t}")
            a, victims = r
            for u in victims:
                evict(u, k, k)
            off[t] = a
            used_bytes[0] += size[t]
            if m & MODE_R:
                res.schedule.append((S_H2D_DEMAND, t, a, size[t], k, k))
                C["h2d_demand_n"] += 1
                C["h2d_demand_B"] += size[t]
            else:
                res.schedule.append((S_ALLOC, t, a, size[t], k, k))
                C["alloc_n"] += 1
            val[t] = DEV_CLEAN
            lru[t] = k
        # (iii) residency at launch
        res.residency.append((k, len(off), used_bytes[0]))
        # (iv) launch
        res.schedule.append((S_LAUNCH, -1, 0, 0, k, k))
        for t, m in A[k]:
            if m & MODE_W:
                val[t] = DEV_DIRTY
            last[t] = k
            lru[t] = k
            pf_need[t] = None
        # (v) look-ahead affinity pins
        if affinity:
            for t, _ in A[k]:
                n = nu(t, k + 1)
                if n != INF and n - k <= affinity_w:
                    pin[t] = max(pin[t], n)
        # (vi) next-kernel prefetch scan of the T and T+A steps
        if not scan:
            continue
        protected = set()
        stop = False
        for j in range(k + 1, min(K - 1, k + D) + 1):
            protected |= Aset[j]
            # host values that an earlier kernel of the window overwrites are
            # dead: only live ones are worth moving
            cands = [t for t, m in A[j] if (m & MODE_R) and val[t] == HOST and live(t, k + 1)]
            if not cands:
                continue

            def pelig(u, k=k, protected=protected):
                return u not in protected and pin[u] < k + 1
            for t in cands:
                r = place(t, pelig, k + 1)
                if r is None:
                    stop = True
                    break
                a, victims = r
                for u in victims:
                    evict(u, k, k + 1)
                off[t] = a
                used_bytes[0] += size[t]
                res.schedule.append((S_H2D_PREFETCH, t, a, size[t], k, j))
                C["h2d_prefetch_n"] += 1
                C["h2d_prefetch_B"] += size[t]
                val[t] = DEV_CLEAN
                lru[t] = k
                pf_need[t] = j
            if stop:
                break
    return res


def _retime(tensors, kernels, M, roofs, lookahead, base):
    """Second pass of the full method: issue each CGI fetch as early as possible.

    ``base`` is the demand timeline (farthest-next-use victims, affinity pins).
    Its replacement decisions are kept; only fetch times change.  A fetch of
    tensor t into window w, demanded at boundary j, may be issued after launch
    k < j when every tensor that occupies any byte of w in the demand timeline
    and leaves it after k is no longer accessed after k (its last access before
    leaving is <= k).  Fetches are issued in their demand order (one link),
    not before an earlier copy of t has left the device (so its write-back, if
    any, precedes the refetch), optionally no more than ``lookahead`` kernels
    ahead, and only for kernels
    the roofline calls CGI-bound in the demand timeline.  Fetches of other
    kernels, and first-write allocations, stay at their kernel.
    """
    nT, K = len(tensors), len(kernels)
    size = [aligned(t["nbytes"]) for t in tensors]
    A, uses, use_mode = _access(tensors, kernels)

    def live(t, k):
        """The value held before kernel k is read later: by the next use if it
        reads, or after the trace when the tensor is live-out."""
        i = bisect_left(uses[t], k)
        if i == len(uses[t]):
            return bool(tensors[t].get("live_out", False))
        return bool(use_mode[t][i] & MODE_R)

    # demand timeline: placement units per boundary and residency intervals
    units = [[] for _ in range(K)]
    pending = []
    intervals, cur, gone = [], {}, {}
    for e in base.schedule:
        op_, t, o, b, ik, nk = e
        if op_ in (S_D2H_WRITEBACK, S_DROP):
            pending.append(e)
            iv = cur.pop(t)
            iv["dep"] = ik
            gone[t] = ik
        elif op_ in (S_H2D_DEMAND, S_ALLOC):
            iv = dict(t=t, off=o, end=o + b, arr=ik, dep=INF, lastacc=ik)
            intervals.append(iv)
            cur[t] = iv
            units[ik].append(dict(evictions=pending, entry=e, iv=iv, issue=ik,
                                  prev_dep=gone.get(t, 0)))
            pending = []
        elif op_ == S_LAUNCH:
            for u, _ in A[ik]:
                cur[u]["lastacc"] = ik
    left = sorted((iv for iv in intervals if iv["dep"] != INF), key=lambda iv: iv["dep"])
    deps = [iv["dep"] for iv in left]

    # earliest issue boundary of each CGI fetch, in demand order
    early = [[] for _ in range(K)]
    prev = 0
    for j in range(1, K):
        if base.dyn_cls[j] != CLS_CGI:
            continue
        for u in units[j]:
            if u["entry"][0] != S_H2D_DEMAND:
                continue
            a, end = u["entry"][2], u["entry"][2] + u["entry"][3]
            # not before the previous copy of the tensor has left the device
            lo = max(prev, j - lookahead if lookahead else 0, u["prev_dep"], 0)
            occ = [iv for iv in left[bisect_right(deps, lo):bisect_right(deps, j)]
                   if iv["off"] < end and a < iv["end"]]
            k = lo
            while True:
                m = max((iv["lastacc"] for iv in occ if iv["dep"] > k), default=-1)
                if m <= k:
                    break
                k = m
            if k < j:
                u["issue"] = k
                early[k].append(u)
                prev = k

    # new timeline
    res = Result()
    res.static_cls = base.static_cls
    res.costs = base.costs
    C = res.counters
    val = [HOST if (t["kind"] == KIND_PARAM or t["host_init"]) else NONE for t in tensors]
    where = {}                      # resident tensor -> offset
    used = [0]

    def evict(t, k):
        if val[t] == DEV_DIRTY and live(t, k + 1):
            res.schedule.append((S_D2H_WRITEBACK, t, where[t], size[t], k, -1))
            C["d2h_wb_n"] += 1
            C["d2h_wb_B"] += size[t]
            val[t] = HOST
        else:
            res.schedule.append((S_DROP, t, where[t], size[t], k, -1))
            C["drop_n"] += 1
            val[t] = NONE if val[t] == DEV_DIRTY else HOST
        used[0] -= size[t]
        del where[t]

    def put(u, k, kind, need):
        op_, t, a, b = u["entry"][:4]
        for v, o in where.items():
            assert not (o < a + b and a < o + size[v]), "retimed window still occupied"
        where[t] = a
        used[0] += b
        res.schedule.append((kind, t, a, b, k, need))
        if kind == S_H2D_PREFETCH:
            C["h2d_prefetch_n"] += 1
            C["h2d_prefetch_B"] += b
        elif kind == S_H2D_DEMAND:
            C["h2d_demand_n"] += 1
            C["h2d_demand_B"] += b
        else:
            C["alloc_n"] += 1
        val[t] = DEV_CLEAN

    for k in range(K):
        F, B = base.costs[k]
        X = sum(size[t] for t, m in A[k] if (m & MODE_R) and val[t] == HOST)
        cls = classify(F, B, X, roofs, kernels[k].get("time_ns", 0))
        res.dyn_cls.append(cls)
        C["class_n"][cls] += 1
        for u in units[k]:
            if u["issue"] < k:
                continue                        # already fetched ahead
            for e in u["evictions"]:
                if where.get(e[1]) == e[2]:
                    evict(e[1], k)
            put(u, k, u["entry"][0], k)
        res.residency.append((k, len(where), used[0]))
        res.schedule.append((S_LAUNCH, -1, 0, 0, k, k))
        for t, m in A[k]:
            if m & MODE_W:
                val[t] = DEV_DIRTY
        for u in early[k]:
            a, b = u["entry"][2], u["entry"][3]
            for t in sorted((v for v, o in where.items() if o < a + b and a < o + size[v]),
                            key=lambda v: where[v]):
                evict(t, k)
            put(u, k, S_H2D_PREFETCH, u["entry"][4])
    return res


def pool_objects(tensors, object_bytes):
    """Tensors grouped into the blocks of a pooling allocator: consecutive
    tensors in registration order share a block until the next one would take
    it past object_bytes (a larger tensor gets a block of its own).  Returns
    the member lists."""
    objs, cur, cur_b = [], [], 0
    for t, td in enumerate(tensors):
        s = aligned(td["nbytes"])
        if cur and cur_b + s > object_bytes:
            objs.append(cur)
            cur, cur_b = [], 0
        cur.append(t)
        cur_b += s
    if cur:
        objs.append(cur)
    return objs


def plan_objects(tensors, kernels, M, object_bytes, **policy):
    """The same policy at object granularity, the contrast of the paper's
    Sec. III-B (Fig. 3): a prefetcher that sees allocator blocks, not tensors,
    moves and evicts whole blocks, and cannot tell which of a block's tensors
    are live.

    The trace is coarsened: each object is one planning unit of its members'
    bytes, valid on the host if any member is; a kernel accesses the objects
    of its operands.  An object's first access by a kernel that only writes
    it needs no fetch (mode W); every later access reads it (liveness is
    unknown per member, so the whole block is live while any access
    remains).  The object plan is then expanded to member tensors in the
    object's window (members contiguous, in registration order): a fetch
    moves every member with a host value (dead or alive) and allocates the
    rest, a write-back copies every member dirty on the device, a drop drops
    them.  A member fetch whose value no kernel reads while it stays
    resident (evicted, overwritten or never accessed first) counts as
    useless (useless_prefetch_n/B); classes and residency are those of the
    object plan."""
    objs = pool_objects(tensors, object_bytes)
    obj_of, rel = {}, {}
    for o, mem in enumerate(objs):
        r = 0
        for t in mem:
            obj_of[t], rel[t] = o, r
            r += aligned(tensors[t]["nbytes"])
    valid0 = [any(tensors[t]["kind"] == KIND_PARAM or tensors[t]["host_init"] for t in mem) for mem in objs]
    otensors = [dict(nbytes=sum(aligned(tensors[t]["nbytes"]) for t in mem), dtype=tensors[mem[0]]["dtype"],
                     kind=KIND_PARAM if valid0[o] else tensors[mem[0]]["kind"], host_init=valid0[o],
                     live_out=any(tensors[t].get("live_out", False) for t in mem))
                for o, mem in enumerate(objs)]
    dtypes = [t["dtype"] for t in tensors]
    raw = [t["nbytes"] for t in tensors]
    touched = [False] * len(objs)
    okernels = []
    for kd in kernels:
        F, B = kd.get("flops", 0), kd.get("hbm_bytes", 0)
        if F == 0 or B == 0:
            aF, aB = kernel_cost(kd["op"], kd["shape"], kd["operands"], dtypes, raw)
            F, B = F or aF, B or aB
        modes, order = {}, []
        for t, m in merge_operands(kd["operands"]):
            o = obj_of[t]
            if o not in modes:
                order.append(o)
                modes[o] = 0
            modes[o] |= m
        ops = []
        for o in order:
            m = modes[o]
            if touched[o] or valid0[o]:
                m = MODE_R | (m & MODE_W)
            ops.append((o, m))
            touched[o] = True
        okernels.append(dict(op=kd["op"], shape=kd["shape"], operands=ops, flops=F, hbm_bytes=B,
                             time_ns=kd.get("time_ns", 0), resolved=True))
    base = plan(otensors, okernels, M, **policy)

    # expansion to member tensors
    res = Result()
    res.static_cls, res.dyn_cls, res.costs = base.static_cls, base.dyn_cls, base.costs
    C = res.counters
    C["class_n"] = list(base.counters["class_n"])
    EMPTY = 4                                   # resident, no value yet
    val = [HOST if (t["kind"] == KIND_PARAM or t["host_init"]) else NONE for t in tensors]
    pending = {}                                # member fetch not yet read: tensor -> bytes
    size = [aligned(t["nbytes"]) for t in tensors]
    resident = set()

    def useless(t):
        if t in pending:
            C["useless_prefetch_n"] += 1
            C["useless_prefetch_B"] += pending.pop(t)

    for op_, o, off, nb, ik, nk in base.schedule:
        if op_ == S_LAUNCH:
            res.residency.append((ik, len(resident), sum(size[t] for t in resident)))
            res.schedule.append((S_LAUNCH, -1, 0, 0, ik, nk))
            for t, m in merge_operands(kernels[ik]["operands"]):
                if (m & MODE_R) and val[t] in (NONE, EMPTY):
                    raise PlanError(E_INVAL, f"kernel {ik} reads tensor {t} before any write")
                if t in pending:
                    if m & MODE_R:
                        del pending[t]
                    else:
                        useless(t)
                if m & MODE_W:
                    val[t] = DEV_DIRTY
            continue
        for t in objs[o]:
            a = off + rel[t]
            if op_ in (S_H2D_PREFETCH, S_H2D_DEMAND, S_ALLOC):
                resident.add(t)
                if op_ != S_ALLOC and val[t] == HOST:
                    res.schedule.append((op_, t, a, size[t], ik, nk))
                    key = "h2d_prefetch" if op_ == S_H2D_PREFETCH else "h2d_demand"
                    C[key + "_n"] += 1
                    C[key + "_B"] += size[t]
                    pending[t] = size[t]
                    val[t] = DEV_CLEAN
                else:
                    res.schedule.append((S_ALLOC, t, a, size[t], ik, nk))
                    C["alloc_n"] += 1
                    val[t] = EMPTY
            else:
                resident.discard(t)
                useless(t)
                if op_ == S_D2H_WRITEBACK and val[t] == DEV_DIRTY:
                    res.schedule.append((S_D2H_WRITEBACK, t, a, size[t], ik, -1))
                    C["d2h_wb_n"] += 1
                    C["d2h_wb_B"] += size[t]
                    val[t] = HOST
                else:
                    res.schedule.append((S_DROP, t, a, size[t], ik, -1))
                    C["drop_n"] += 1
                    val[t] = HOST if val[t] == DEV_CLEAN else NONE
    for t in list(pending):
        useless(t)
    return res


def plan_workload(w, M=None, **kw):
    """Convenience: replay on a workloads.trace.Workload."""
    tensors = [dict(nbytes=t.nbytes, dtype=t.dtype, kind=t.kind, host_init=t.host_init,
                    live_out=t.live_out) for t in w.tensors]
    times = kw.pop("times", None)
    kernels = [dict(op=k.op, shape=k.shape, operands=k.operands) for k in w.kernels]
    if times is not None:
        for kd, t in zip(kernels, times):
            kd["time_ns"] = int(t)
    return plan(tensors, kernels, w.budget() if M is None else M, **kw)
