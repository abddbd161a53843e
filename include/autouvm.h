/*
 * autouvm.h — C interface of the tensor-granular, roofline-gated prefetch
 * runtime for decoder inference under device-memory oversubscription.
 *
 * The paper's problem statement (Sec. I, goals (1)-(3); Sec. IV-A) asks for
 * three things, which this interface exposes directly:
 *   1. tensor-level access information: tensors are registered as
 *      sub-allocations of one pooled arena (Sec. II-B, the pooling allocator
 *      hides them from the driver), and each kernel is registered with the
 *      list of tensors it touches (Sec. IV-D, kernel--tensor access tracing);
 *   2. which migrations are performance-critical: a multi-level roofline
 *      (GPU compute, HBM, CPU--GPU interconnect) classifies kernels and only
 *      interconnect-bound kernels get their tensors fetched ahead
 *      (Sec. III-C, Sec. IV-D "UVM Analyzer", Sec. IV-E "Prefetch Engine");
 *   3. adaptation to memory pressure: the device budget caps a pooled device
 *      arena, and classes are re-evaluated on the residency the plan itself
 *      produces (Sec. IV-E "Runtime Monitor").
 * The oversubscription factor is registered bytes over the device budget
 * (Sec. II-A).
 *
 * Lifecycle: create -> arena_init -> register_tensor* -> (write initial host
 * contents through tensor_host_ptr) -> add_kernel* -> set_budget ->
 * [set_roofs] [set_policy] -> plan -> [bind_streams] -> run* -> read_tensor /
 * get_* -> destroy.  run may be called in contiguous, increasing segments.
 *
 * Threading: a context is not thread-safe; use one context per thread.
 * Errors: every call returns an auvm_status; on failure auvm_last_error()
 * describes it (valid until the next call on the same context).  No call
 * aborts the process.
 */
#ifndef AUTOUVM_H
#define AUTOUVM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct auvm_ctx auvm_ctx;
typedef int32_t auvm_status;

enum {
  AUVM_OK = 0,
  AUVM_E_INVAL = -1,   /* bad argument, unknown id/op, read of a never-written tensor */
  AUVM_E_STATE = -2,   /* call out of lifecycle order */
  AUVM_E_BUDGET = -3,  /* some kernel's operands exceed the device budget */
  AUVM_E_FRAG = -4,    /* no contiguous pool window although bytes would fit */
  AUVM_E_HIP = -5,     /* a HIP runtime call failed (message in last_error) */
  AUVM_E_NOMEM = -6,   /* host or device allocation failed */
  AUVM_E_RANGE = -7    /* caller buffer too small */
};

/* tensor element types */
enum { AUVM_F32 = 0, AUVM_BF16 = 1, AUVM_I32 = 2, AUVM_U8 = 3 };
/* tensor kinds: parameters start valid on the host */
enum { AUVM_PARAM = 0, AUVM_ACT = 1, AUVM_KV = 2 };
/* registration flags: HOST_INIT marks a non-parameter with valid host contents */
/* LIVE_OUT: the tensor's final value is read after the trace (model and
 * optimizer state that the next training step uses): a dirty copy evicted
 * after its last use is written back, not dropped. */
enum { AUVM_HOST_INIT = 1, AUVM_LIVE_OUT = 2 };
/* operand access modes */
enum { AUVM_R = 1, AUVM_W = 2, AUVM_RW = 3 };

/* kernel ops; shape[] integers and positional operands per op:
 *  TOUCH         (log_slot)          log RW (>= 64*(log_slot+1) B), then 1..7 data
 *                                    operands (bytes % 4 == 0): for each data
 *                                    operand i the min and max u32 word read
 *                                    are logged at log[16*slot + 2i], writes
 *                                    fill the operand with slot+1.
 *  EMBED         (T,H,V)             ids R i32[T], E R [V,H], x W f32[T,H]
 *  LAYERNORM     (T,H,stride,offset) x R f32, g R [H], b R [H], h W [T,H];
 *                                    output row i normalises input row i*stride+offset
 *  RMSNORM       (T,H,stride,offset) x R f32, g R [H], h W [T,H]
 *  LINEAR        (M,N,K)             a R [M,K], W R [N,K], c W [M,N]: c = a W^T
 *  LINEAR_GELU   (M,N,K)             as LINEAR, c = gelu_erf(a W^T)
 *  LINEAR_RESID  (M,N,K)             a R, W R, x RW f32[M,N]: x += a W^T
 *  LINEAR_SWIGLU (M,N,K)             a R, Wg R, Wu R, c W: c = silu(a Wg^T) * (a Wu^T)
 *  LINEAR_QKV    (M,N,K)             a R [M,K], Wq R, Wk R, Wv R [N,K], q W, k W, v W [M,N]:
 *                                    three LINEARs of one input in one launch (the
 *                                    attention's query, key and value projections);
 *                                    each output equals its LINEAR bit for bit
 *  ATTN_QKV      (B,S,nH,d)          qkv R [B*S, 3*nH*d] (q|k|v column blocks),
 *                                    o W [B*S, nH*d]; causal within each sequence
 *  ROPE_KV       (B,S,nH,d,Lmax,pos0) q RW, k R, v R [B*S, nH*d], Kc, Vc [B,nH,Lmax,d]:
 *                                    rotate-half RoPE (base 1e4) on q and k at
 *                                    positions pos0.., k and v stored at pos0..
 *  ATTN_CACHE    (B,S,nH,d,Lmax,pos0) q R, Kc R, Vc R, o W [, lse W f32[B,nH,S]]:
 *                                    query i attends to cache positions 0..pos0+i;
 *                                    lse: the natural log-sum-exp of each query's
 *                                    scaled scores (kept for the backward pass)
 *  ARGMAX        (B,V,row)           logits R f32[B,V], tok W i32[B], [gen RW i32[.,B]]:
 *                                    lowest index of the row maximum; also gen[row]
 * Routed-expert (MoE) FFN, top-K of E experts (K <= E <= 16), bf16 weights:
 *  MOE_ROUTE     (M,H,E,K)           h R [M,H], Wr R [E,H], rte W i32[M,K], rtw W f32[M,K]:
 *                                    router logits h Wr^T; the K largest (ties: lower
 *                                    expert index) in descending order, weights the
 *                                    softmax over the selected logits
 *  MOE_DISPATCH  (M,E,K,row)         rte R, lists W i32[E, M+1], log RW i32[(row+1)*E]:
 *                                    lists[e] = count, then the entries j = K*token+slot
 *                                    with rte[j] == e in increasing j; log[row*E+e] = count
 *  MOE_UP        (M,F,H,e,n,K)       h R [M,H], lists R, Wg R [F,H], Wu R [F,H], fe W [M,F]:
 *                                    for i < count(e): fe[i] = silu(h[tok] Wg^T) * (h[tok] Wu^T),
 *                                    tok = lists[e][1+i] / K; n = routed rows expected by
 *                                    the trace (cost model only)
 *  MOE_DOWN      (M,H,F,e,n,K)       fe R, lists R, rtw R, Wd R [H,F], x RW f32[M,H]:
 *                                    for i < count(e): x[tok] += rtw[j] * (fe[i] Wd^T),
 *                                    j = lists[e][1+i], tok = j / K
 * Training step (backward and optimizer), bf16 activations and weights with
 * fp32 residual stream, gradients, master weights and moments:
 *  COPY          (bytes)             a R, b W: device copy of the first bytes
 *  TRANSPOSE     (R,C)               a R [R,C], b W [C,R] (same dtype)
 *  SWIGLU_ACT    (T,F)               G R, U R, F W [T,F]: F = silu(G) * U
 *  SWIGLU_BWD    (T,F)               G R, U R, dF R, dG W, dU W: the gradients of F
 *  RMSNORM_BWD   (T,H,acc)           x R f32[T,H], g R [H], dy R f32[T,H], dx W|RW f32[T,H],
 *                                    dxb W bf16[T,H], dg W f32[H], rstd W f32[T]: the
 *                                    RMSNorm (eps 1e-6) gradients; dx is overwritten
 *                                    (acc 0) or accumulated into (acc 1), dxb is dx in
 *                                    bf16, rstd a workspace
 *  ATTN_BWD      (B,S,nH,d)          q R, K R, V R, o R, lse R, do R, dq W, dK W, dV W, D W:
 *                                    causal attention gradients from the forward's
 *                                    operands (q, o, do, dq [B*S, nH*d]; K, V, dK, dV
 *                                    [B,nH,S,d]; lse, D f32[B,nH,S], D a workspace); d = 128
 *  ROPE_BWD      (B,S,nH,d)          dq RW, dK R, dV R, dk W, dv W: rotates dq and dK back
 *                                    (rotate-half, base 1e4, positions 0..S-1), dk, dv
 *                                    token-major [B*S, nH*d]
 *  XENT          (T,V)               logits R f32[T,V], labels R i32[T], losses W f32[T],
 *                                    dlogits W [T,V]: per-row cross-entropy and the
 *                                    gradient of the mean loss, (softmax - onehot) / T
 *  EMBED_BWD     (T,H,V)             ids R i32[T], dx R f32[T,H], dE W f32[V,H]: rows of dx
 *                                    summed into their token's row, in token order
 *  ADAM          (n,t,lr,b1,b2,eps,wd) g R f32[n], p32 RW f32, m RW f32, v RW f32, p W [n]:
 *                                    AdamW at step t with decoupled weight decay and
 *                                    bias correction; hyperparameters in fixed point
 *                                    (lr*1e9, b1*1e6, b2*1e6, eps*1e12, wd*1e6); p is the
 *                                    updated p32 in p's dtype
 * Activations between kernels use the tensors' own dtypes (f32 or bf16);
 * arithmetic accumulates in fp32. */
enum {
  AUVM_OP_TOUCH = 0, AUVM_OP_EMBED = 1, AUVM_OP_LAYERNORM = 2, AUVM_OP_RMSNORM = 3,
  AUVM_OP_LINEAR = 4, AUVM_OP_LINEAR_GELU = 5, AUVM_OP_LINEAR_RESID = 6,
  AUVM_OP_LINEAR_SWIGLU = 7, AUVM_OP_ATTN_QKV = 8, AUVM_OP_ROPE_KV = 9,
  AUVM_OP_ATTN_CACHE = 10, AUVM_OP_ARGMAX = 11, AUVM_OP_MOE_ROUTE = 12,
  AUVM_OP_MOE_DISPATCH = 13, AUVM_OP_MOE_UP = 14, AUVM_OP_MOE_DOWN = 15, AUVM_OP_COPY = 16,
  AUVM_OP_TRANSPOSE = 17, AUVM_OP_SWIGLU_ACT = 18, AUVM_OP_SWIGLU_BWD = 19, AUVM_OP_RMSNORM_BWD = 20,
  AUVM_OP_ATTN_BWD = 21, AUVM_OP_ROPE_BWD = 22, AUVM_OP_XENT = 23, AUVM_OP_EMBED_BWD = 24,
  AUVM_OP_ADAM = 25, AUVM_OP_LINEAR_QKV = 26, AUVM_OP_COUNT = 27
};

/* policy variants: the paper's ablation ladder (T, T+A, T+A+P; Sec. V-E)
 * and the two demand-migration baselines (Sec. V-A "Baseline") */
enum { AUVM_DEMAND_LRU = 0, AUVM_DEMAND_BELADY = 1, AUVM_T = 2, AUVM_T_A = 3, AUVM_T_A_P = 4 };
enum { AUVM_PLACE_POOL = 0, AUVM_PLACE_IDEAL = 1 };
/* schedule entry ops */
enum { AUVM_H2D_PREFETCH = 0, AUVM_H2D_DEMAND = 1, AUVM_D2H_WRITEBACK = 2,
       AUVM_DROP = 3, AUVM_ALLOC = 4, AUVM_LAUNCH = 5 };
/* roofline classes (Sec. IV-D "UVM Analyzer") */
enum { AUVM_CLS_COMPUTE = 0, AUVM_CLS_MEMORY = 1, AUVM_CLS_CGI = 2 };

typedef struct {
  uint32_t op;            /* AUVM_OP_* */
  int64_t shape[8];       /* op-specific integers, unused trailing entries 0 */
  uint32_t n;             /* operand count */
  const int32_t* ids;     /* n tensor ids in the op's positional order */
  const uint8_t* modes;   /* n access modes (AUVM_R/W/RW) */
  uint64_t flops;         /* 0: analytic count for the op */
  uint64_t hbm_bytes;     /* 0: analytic algorithmic bytes for the op */
  uint32_t layer;         /* reporting only */
} auvm_kernel_desc;

/* guard or bucket value that asks for the library's default for the variant */
#define AUVM_POLICY_DEFAULT 0xFFFFFFFFu

typedef struct {
  uint32_t variant;       /* AUVM_DEMAND_LRU .. AUVM_T_A_P (default T_A_P, guard 4, bucket 32) */
  uint32_t lookahead;     /* max kernels a fetch runs ahead; 0 = T/T+A: 1, T+A+P: unlimited */
  uint32_t affinity_w;    /* pin operands reused within this many kernels (default 1) */
  uint32_t placement;     /* AUVM_PLACE_POOL (default) or AUVM_PLACE_IDEAL (plan-only) */
  uint32_t validate;      /* 1: fill every dropped or written-back window with NaN bytes */
  uint32_t timing;        /* 1: record per-kernel start/end events during run */
  uint32_t guard;         /* T+A+P only: a demand at kernel j prefers victims not used by
                             kernels j-guard..j-1, so their replacement fetch can start
                             that many kernels earlier (0 = plain farthest-next-use;
                             AUVM_POLICY_DEFAULT = 4 for T+A+P, 0 otherwise) */
  uint32_t bucket;        /* T+A+P and DEMAND_BELADY: victims' next uses are compared in
                             buckets of this many kernels, and within a bucket the pool
                             window that evicts fewer bytes wins (1 = exact
                             farthest-next-use; 0 is read as 1; AUVM_POLICY_DEFAULT = 32
                             for T+A+P, 1 otherwise) */
  uint64_t object_bytes;  /* 0 (default): tensor granularity, the method.  > 0: the same variant
                             at the granularity of a pooling allocator's blocks, the contrast
                             of the paper's Sec. III-B (Fig. 3): consecutive tensors in
                             registration order share a block until the next would take it
                             past object_bytes (a larger tensor gets its own); blocks move and
                             are evicted whole, a fetch moves every member with a host value,
                             a write-back every dirty member, and a block's members count as
                             live while any access to the block remains.  The schedule lists
                             member tensors (contiguous in the block's window);
                             useless_prefetch_n/B count member fetches whose value no kernel
                             reads while resident. */
} auvm_policy;

typedef struct {
  int32_t op;             /* AUVM_H2D_PREFETCH .. AUVM_LAUNCH */
  int32_t tensor;         /* -1 for LAUNCH */
  uint64_t dev_off;       /* pool offset of the tensor's window */
  uint64_t bytes;         /* 256-aligned tensor size (0 for LAUNCH) */
  int32_t issue_k;        /* boundary: before launch k (demand/alloc/evict) or after it (prefetch) */
  int32_t need_k;         /* kernel the fetch serves; -1 for evictions */
} auvm_sched_entry;

typedef struct {
  int32_t k;
  int32_t n_resident;
  uint64_t resident_bytes; /* resident bytes when kernel k launches */
} auvm_residency;

typedef struct {
  uint8_t static_cls;     /* class with every read operand host-resident */
  uint8_t dyn_cls;        /* class on the planned residency at the kernel's boundary */
  uint8_t pad[6];
  uint64_t flops;
  uint64_t hbm_bytes;
} auvm_kernel_class;

typedef struct {
  uint64_t h2d_prefetch_n, h2d_prefetch_B;
  uint64_t h2d_demand_n, h2d_demand_B;    /* demand fetches ("faults") */
  uint64_t d2h_wb_n, d2h_wb_B;
  uint64_t drop_n, alloc_n;
  uint64_t useless_prefetch_n, useless_prefetch_B;   /* prefetches dropped before their kernel;
                                             at object granularity: member fetches never read
                                             while resident */
  uint64_t class_n[3];                    /* kernels per dynamic class */
  uint64_t plan_ns;                       /* host time of the last auvm_plan */
  uint64_t run_ns;                        /* host wall time inside auvm_run calls */
  uint64_t kernels_run;                   /* launches executed since plan/reset */
  uint64_t stall_ns;                      /* timing policy: compute-stream idle time between
                                             consecutive kernels of each run segment since
                                             plan/reset (kernels waiting for their operands'
                                             copies, or for the host); 0 without timing */
} auvm_counters;

/* Create a context bound to HIP device `hip_device`; a negative device gives a
 * plan-only context (no HIP call is ever made; run/read_tensor fail with
 * AUVM_E_STATE).  *out receives the context; caller destroys it. */
auvm_status auvm_create(int hip_device, auvm_ctx** out);
/* Free everything the context allocated; borrowed memory and streams are left alone. */
void auvm_destroy(auvm_ctx* ctx);
const char* auvm_last_error(const auvm_ctx* ctx);

/* Host backing store of all tensors.  host_pinned == NULL: the context
 * allocates arena_bytes of pinned host memory (plan-only contexts allocate
 * nothing).  Otherwise the caller lends memory that must be pinned, at least
 * arena_bytes long, and outlive the context.  Once per context. */
auvm_status auvm_arena_init(auvm_ctx* ctx, uint64_t arena_bytes, void* host_pinned);

/* A host backing store larger than the host lets the process pin.  Offsets
 * [0, pinned_bytes) are pinned host memory and [pinned_bytes, arena_bytes)
 * pageable memory, both allocated by the context (plan-only contexts
 * allocate nothing).  Fetches of tensors in the pageable tier pass through a
 * pinned staging ring of 4 x 64 MiB: host threads copy a piece into a free
 * slot, then the slot goes to the device on the copy stream; the tensors and
 * the schedule are the same as in a pinned arena.  A tensor window must lie
 * wholly in one tier, only parameter tensors may lie in the pageable tier,
 * and no kernel may write one (auvm_register_tensor and auvm_add_kernel
 * return AUVM_E_INVAL), so nothing is ever written back there.
 * pinned_bytes: a multiple of 256, at most arena_bytes (equal: as
 * auvm_arena_init with NULL).  Once per context; AUVM_E_NOMEM when either
 * allocation fails.  The pageable tier extends the host side of the pooled
 * arena beyond pinned memory (Sec. II-A: the CPU's memory as the backing
 * store of an oversubscribed device). */
auvm_status auvm_arena_init_tiered(auvm_ctx* ctx, uint64_t arena_bytes, uint64_t pinned_bytes);

/* Register a tensor as the sub-allocation [arena_off, arena_off+bytes) of the
 * arena; ids are dense in registration order.  arena_off must be 256-aligned;
 * windows must not overlap and must lie inside the arena.  PARAM and
 * HOST_INIT tensors start valid on the host; others start with no value. */
auvm_status auvm_register_tensor(auvm_ctx* ctx, uint64_t arena_off, uint64_t bytes,
                                 uint32_t dtype, uint32_t kind, uint32_t flags,
                                 int32_t* out_id);
/* Host address of a tensor's arena window (for writing initial contents). */
auvm_status auvm_tensor_host_ptr(auvm_ctx* ctx, int32_t id, void** out);

/* Append a kernel to the trace.  The op's operand count, dtypes and byte
 * sizes are checked against its shape here (AUVM_E_INVAL on mismatch), so no
 * launch can address outside its operands.  Repeated ids in one kernel are
 * merged for planning with the union of their modes.  *out_k = kernel index. */
auvm_status auvm_add_kernel(auvm_ctx* ctx, const auvm_kernel_desc* desc, int32_t* out_k);

/* Device budget M (rounded down to 256) and the pool it is carved from.
 * device_pool == NULL: the context allocates M bytes (never in plan-only
 * contexts).  Otherwise the caller lends a device buffer of >= M bytes.
 * Called again, it replaces budget and pool (the oversubscription factor of
 * the same tensors and trace): it waits for outstanding work, frees a pool
 * the context allocated, forgets device residency as auvm_reset does and
 * drops the plan, so read outputs first and call auvm_plan before the next
 * run.  A borrowed old pool may be released once this returns. */
auvm_status auvm_set_budget(auvm_ctx* ctx, uint64_t device_bytes, void* device_pool);
/* Roofs in flop/s and byte/s (integers).  Default: 2.5e15, 8e12, 64e9. */
auvm_status auvm_set_roofs(auvm_ctx* ctx, uint64_t peak_flops, uint64_t hbm_Bps, uint64_t link_Bps);
auvm_status auvm_set_policy(auvm_ctx* ctx, const auvm_policy* policy);
/* Drop every kernel and the plan, and reset execution as auvm_reset does;
 * tensors, host arena contents, budget, roofs and policy stay.  Lets a
 * caller replace a profiling trace by the trace it recorded (Sec. IV-D,
 * kernel-tensor access tracing): for routed experts the access lists depend
 * on the router, so the profiling trace holds every expert and the recorded
 * one only the experts that were routed rows (Sec. III-A: move only the
 * tensors a kernel accesses).  Read outputs before calling. */
auvm_status auvm_clear_kernels(auvm_ctx* ctx);

/* Measured execution time of every kernel of the trace, in nanoseconds (the
 * runtime monitor's measurements, Sec. IV, Online Executor, Runtime Monitor:
 * kernel classifications are re-evaluated from measured kernel time).  A
 * kernel with time t > 0 is CGI-bound iff it has host-resident read bytes X
 * and X/Bl > t (exact integer test); t = 0 keeps the analytic roofline test.
 * The static COMPUTE/MEMORY class stays analytic.  n must equal the number of
 * kernels (AUVM_E_INVAL otherwise).  The current plan is dropped: call
 * auvm_plan again (which also resets execution) before the next run. */
auvm_status auvm_set_kernel_times(auvm_ctx* ctx, const uint64_t* t_ns, uint64_t n);

/* Build the transfer schedule for the whole trace (host only, deterministic).
 * AUVM_E_BUDGET / AUVM_E_FRAG / AUVM_E_INVAL as described above.  Then
 * resets execution as auvm_reset does: device-resident values are forgotten,
 * so read the outputs of a run (auvm_read_tensor) before planning again. */
auvm_status auvm_plan(auvm_ctx* ctx);

/* Lend the compute, host-to-device and device-to-host streams (hipStream_t
 * values passed as pointers); NULL entries keep the context's own.  The
 * context creates its streams each on a hardware queue of its own, so copies
 * overlap kernels.  Lent streams must not share a hardware queue with each
 * other (HIP maps ordinary streams onto a few shared queues): on a shared
 * queue a kernel waits for every copy enqueued before it, which serializes
 * transfers with compute. */
auvm_status auvm_bind_streams(auvm_ctx* ctx, void* compute, void* h2d, void* d2h);

/* Execute boundaries first_k .. first_k+n_k-1 of the plan (their transfers
 * and launches, plus fetches issued after the last launch), then wait for
 * all three streams.  Segments must be contiguous and increasing from 0. */
auvm_status auvm_run(auvm_ctx* ctx, uint32_t first_k, uint32_t n_k);
/* auvm_run for callers that cannot allocate (code under HIP graph capture,
 * serving loops, harnesses that forbid allocation): the same transfers and
 * launches, but the kernels' workspace operands (ATTN_BWD's D, RMSNORM_BWD's
 * rstd) live in the library's static device scratch, 8 MiB per GPU (each GPU
 * the library runs on holds it until the process ends), instead of their pool
 * windows, whose contents are undefined afterwards; no memory, stream or
 * event is created (the plan must have timing off: AUVM_E_STATE otherwise).
 * A workspace above 8 MiB gives AUVM_E_RANGE before anything is enqueued.
 * Every call on one GPU shares that GPU's scratch and leaves its contents
 * behind: calls that overlap on one GPU (several contexts or threads) race.
 * The scratch needs no clearing: each workspace is written before it is read. */
auvm_status auvm_run_noalloc(auvm_ctx* ctx, uint32_t first_k, uint32_t n_k);
/* Forget all device residency and rewind to kernel 0.  The caller must
 * restore host contents of tensors the trace reads before writing. */
auvm_status auvm_reset(auvm_ctx* ctx);

/* Copy the current value of a tensor into dst (host memory, >= its bytes):
 * from the device when the newest copy is there, else from the host arena.
 * Does not change residency or the schedule. */
auvm_status auvm_read_tensor(auvm_ctx* ctx, int32_t id, void* dst, uint64_t dst_bytes);

auvm_status auvm_get_counters(const auvm_ctx* ctx, auvm_counters* out);
/* Two-call pattern: buf == NULL stores the count in *n; cap < count gives
 * AUVM_E_RANGE.  get_schedule returns the plan, get_executed the entries
 * executed so far (identical to the plan's prefix). */
auvm_status auvm_get_schedule(const auvm_ctx* ctx, auvm_sched_entry* buf, uint64_t cap, uint64_t* n);
auvm_status auvm_get_executed(const auvm_ctx* ctx, auvm_sched_entry* buf, uint64_t cap, uint64_t* n);
auvm_status auvm_get_residency(const auvm_ctx* ctx, auvm_residency* buf, uint64_t cap, uint64_t* n);
auvm_status auvm_get_classes(const auvm_ctx* ctx, auvm_kernel_class* buf, uint64_t cap, uint64_t* n);
/* Per executed kernel (timing policy): duration and the compute-stream gap
 * before it (time from the previous kernel's end to this kernel's start), in
 * milliseconds, for kernels 0 .. n-1 of the last run segments since reset. */
auvm_status auvm_get_kernel_times(const auvm_ctx* ctx, float* dur_ms, float* gap_ms,
                                  uint64_t cap, uint64_t* n);

/* One executed kernel or copy on the device timeline (timing policy).  Times
 * are milliseconds from the start of the run segment that issued it: host_ms
 * when the host thread issued it, start_ms/end_ms when its stream began and
 * finished it (from an event recorded on the idle streams at the segment's
 * start).  This extends the runtime monitor's kernel timestamps (Sec. IV,
 * Online Executor, Runtime Monitor) to the copies, so that link busy time,
 * compute busy time and the stalls of each on the other can be measured.
 * Host-to-device copies alternate between two streams by copy number (odd
 * numbers, the first copy included, on the first): AUVM_TL_H2D entries come
 * from one, AUVM_TL_H2D_B from the other; each stream's entries are in order,
 * and the two may overlap.  A plan with write-backs keeps all its copies on
 * the first stream. */
enum { AUVM_TL_KERNEL = 0, AUVM_TL_H2D = 1, AUVM_TL_D2H = 2, AUVM_TL_H2D_B = 3 };
typedef struct auvm_timeline_entry {
  int32_t kind;     /* AUVM_TL_* */
  int32_t segment;  /* run call ordinal since the last reset, from 0 */
  int64_t index;    /* kernel index, or index of the copy's schedule entry */
  uint64_t bytes;   /* bytes moved (copies), 0 for kernels */
  double host_ms;
  double start_ms;
  double end_ms;
} auvm_timeline_entry;

/* Entries of the run segments since reset in issue order (kernels and copies
 * interleaved).  Two-call pattern as get_schedule; empty unless the policy's
 * timing flag was set while they ran. */
auvm_status auvm_get_timeline(const auvm_ctx* ctx, auvm_timeline_entry* buf, uint64_t cap, uint64_t* n);

#ifdef __cplusplus
}
#endif
#endif /* AUTOUVM_H */
