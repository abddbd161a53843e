// Kernel cost model and operand validation.
//
// The roofline placement of a kernel (Sec. III-C, Sec. IV-D "UVM Analyzer")
// needs its floating-point work F and its memory traffic B.  The paper counts
// them with binary instrumentation; here they are the algorithmic counts of
// each op from its shape: 2*M*N*K per GEMM, every operand element read or
// written once, read-modify-write counted twice.
#include <sstream>

#include "core.h"

namespace auvm {

namespace {

uint64_t es(const std::vector<Tensor>& T, const Kernel& k, int i) {
  return dtype_size(T[k.ids[i]].dtype);
}

}  // namespace

void kernel_cost(const Kernel& k, const std::vector<Tensor>& T, uint64_t* Fo, uint64_t* Bo) {
  const int64_t* s = k.shape;
  uint64_t F = 0, B = 0;
  switch (k.op) {
    case AUVM_OP_TOUCH:
      for (auto& a : k.acc) B += T[a.first].bytes * (a.second == AUVM_RW ? 2 : 1);
      break;
    case AUVM_OP_EMBED: {
      uint64_t Tn = s[0], H = s[1];
      B = 4 * Tn + Tn * H * es(T, k, 1) + Tn * H * es(T, k, 2);
      break;
    }
    case AUVM_OP_LAYERNORM: {
      uint64_t Tn = s[0], H = s[1];
      F = 8 * Tn * H;
      B = Tn * H * es(T, k, 0) + H * es(T, k, 1) + H * es(T, k, 2) + Tn * H * es(T, k, 3);
      break;
    }
    case AUVM_OP_RMSNORM: {
      uint64_t Tn = s[0], H = s[1];
      F = 4 * Tn * H;
      B = Tn * H * es(T, k, 0) + H * es(T, k, 1) + Tn * H * es(T, k, 2);
      break;
    }
    case AUVM_OP_LINEAR:
    case AUVM_OP_LINEAR_GELU:
    case AUVM_OP_LINEAR_RESID: {
      uint64_t M = s[0], N = s[1], K = s[2];
      F = 2 * M * N * K;
      if (k.op == AUVM_OP_LINEAR_GELU) F += 8 * M * N;
      if (k.op == AUVM_OP_LINEAR_RESID) F += M * N;
      uint64_t out = M * N * es(T, k, 2) * (k.op == AUVM_OP_LINEAR_RESID ? 2 : 1);
      B = M * K * es(T, k, 0) + N * K * es(T, k, 1) + out;
      break;
    }
    case AUVM_OP_LINEAR_QKV: {
      uint64_t M = s[0], N = s[1], K = s[2];
      F = 6 * M * N * K;
      B = M * K * es(T, k, 0) + N * K * (es(T, k, 1) + es(T, k, 2) + es(T, k, 3)) +
          M * N * (es(T, k, 4) + es(T, k, 5) + es(T, k, 6));
      break;
    }
    case AUVM_OP_LINEAR_SWIGLU: {
      uint64_t M = s[0], N = s[1], K = s[2];
      F = 4 * M * N * K + 4 * M * N;
      B = M * K * es(T, k, 0) + N * K * (es(T, k, 1) + es(T, k, 2)) + M * N * es(T, k, 3);
      break;
    }
    case AUVM_OP_ATTN_QKV: {
      uint64_t Bt = s[0], S = s[1], nH = s[2], d = s[3];
      uint64_t pairs = S * (S + 1) / 2;
      F = Bt * nH * pairs * (4 * d + 4);
      B = Bt * S * nH * d * (3 * es(T, k, 0) + es(T, k, 1));
      break;
    }
    case AUVM_OP_ROPE_KV: {
      uint64_t n = uint64_t(s[0]) * s[1] * s[2] * s[3];
      F = 6 * n;
      B = n * (2 * es(T, k, 0) + es(T, k, 1) + es(T, k, 2) + es(T, k, 3) + es(T, k, 4));
      break;
    }
    case AUVM_OP_ATTN_CACHE: {
      uint64_t Bt = s[0], S = s[1], nH = s[2], d = s[3], pos0 = s[5];
      uint64_t pairs = S * pos0 + S * (S + 1) / 2;
      F = Bt * nH * pairs * (4 * d + 4);
      B = Bt * S * nH * d * (es(T, k, 0) + es(T, k, 3)) +
          Bt * nH * (pos0 + S) * d * (es(T, k, 1) + es(T, k, 2));
      if (k.ids.size() > 4) B += 4 * Bt * nH * S;   // row log-sum-exp
      break;
    }
    case AUVM_OP_ARGMAX: {
      uint64_t Bt = s[0], V = s[1];
      F = Bt * V;
      B = Bt * V * es(T, k, 0) + 4 * Bt + (k.ids.size() > 2 ? 4 * Bt : 0);
      break;
    }
    // Routed experts: n (shape[4]) is the row count the trace expects the
    // expert to see, so a decode expert prices as a weight read and a
    // prefill expert as its GEMM.
    case AUVM_OP_MOE_ROUTE: {
      uint64_t M = s[0], H = s[1], E = s[2], K = s[3];
      F = 2 * M * H * E;
      B = M * H * es(T, k, 0) + E * H * es(T, k, 1) + 8 * M * K;
      break;
    }
    case AUVM_OP_MOE_DISPATCH: {
      uint64_t M = s[0], E = s[1], K = s[2];
      B = 4 * M * K + 4 * (M * K + E) + 8 * E;
      break;
    }
    case AUVM_OP_MOE_UP: {
      uint64_t Fw = s[1], H = s[2], n = s[4];
      F = 4 * n * Fw * H + 4 * n * Fw;
      B = n * H * es(T, k, 0) + 4 * (n + 1) + Fw * H * (es(T, k, 2) + es(T, k, 3)) + n * Fw * es(T, k, 4);
      break;
    }
    case AUVM_OP_MOE_DOWN: {
      uint64_t H = s[1], Fw = s[2], n = s[4];
      F = 2 * n * H * Fw + 2 * n * H;
      B = n * Fw * es(T, k, 0) + 4 * (n + 1) + 4 * n + H * Fw * es(T, k, 3) + 8 * n * H;
      break;
    }
    // training step: every operand element read or written once
    case AUVM_OP_COPY: B = 2 * uint64_t(s[0]); break;
    case AUVM_OP_TRANSPOSE: B = 2 * uint64_t(s[0]) * s[1] * es(T, k, 0); break;
    case AUVM_OP_SWIGLU_ACT: {
      uint64_t n = uint64_t(s[0]) * s[1];
      F = 5 * n;
      B = n * (es(T, k, 0) + es(T, k, 1) + es(T, k, 2));
      break;
    }
    case AUVM_OP_SWIGLU_BWD: {
      uint64_t n = uint64_t(s[0]) * s[1];
      F = 10 * n;
      B = n * (es(T, k, 0) + es(T, k, 1) + es(T, k, 2) + es(T, k, 3) + es(T, k, 4));
      break;
    }
    case AUVM_OP_RMSNORM_BWD: {
      uint64_t Tn = s[0], H = s[1], n = Tn * H;
      F = 10 * n;
      B = n * (es(T, k, 0) + es(T, k, 2) + es(T, k, 4)) + n * es(T, k, 3) * (s[2] ? 2 : 1) +
          H * (es(T, k, 1) + es(T, k, 5)) + 4 * Tn;
      break;
    }
    case AUVM_OP_ATTN_BWD: {
      uint64_t Bt = s[0], S = s[1], nH = s[2], d = s[3];
      uint64_t pairs = S * (S + 1) / 2;
      F = Bt * nH * pairs * (10 * d + 8);
      uint64_t e = 0;
      for (int i : {0, 1, 2, 3, 5, 6, 7, 8}) e += es(T, k, i);
      B = Bt * S * nH * d * e + 12 * Bt * nH * S;
      break;
    }
    case AUVM_OP_ROPE_BWD: {
      uint64_t n = uint64_t(s[0]) * s[1] * s[2] * s[3];
      F = 6 * n;
      B = n * (2 * es(T, k, 0) + es(T, k, 1) + es(T, k, 2) + es(T, k, 3) + es(T, k, 4));
      break;
    }
    case AUVM_OP_XENT: {
      uint64_t Tn = s[0], V = s[1];
      F = 4 * Tn * V;
      B = Tn * V * (es(T, k, 0) + es(T, k, 3)) + 8 * Tn;
      break;
    }
    case AUVM_OP_EMBED_BWD: {
      uint64_t Tn = s[0], H = s[1], V = s[2];
      F = Tn * H;
      B = 4 * Tn + Tn * H * es(T, k, 1) + V * H * es(T, k, 2);
      break;
    }
    case AUVM_OP_ADAM: {
      uint64_t n = s[0];
      F = 12 * n;
      B = n * (es(T, k, 0) + 2 * es(T, k, 1) + 2 * es(T, k, 2) + 2 * es(T, k, 3) + es(T, k, 4));
      break;
    }
  }
  *Fo = F;
  *Bo = B;
}

uint8_t classify(uint64_t F, uint64_t B, uint64_t X, const Roofs& r, uint64_t t_ns) {
  using u128 = unsigned __int128;
  if (t_ns > 0) {  // runtime monitor: link time X/Bl against the measured time
    if (X > 0 && u128(X) * 1000000000u > u128(t_ns) * r.Bl) return AUVM_CLS_CGI;
  } else if (X > 0 && u128(X) * r.P > u128(F) * r.Bl && u128(X) * r.Bh > u128(B) * r.Bl) {
    return AUVM_CLS_CGI;
  }
  return u128(F) * r.Bh >= u128(B) * r.P ? AUVM_CLS_COMPUTE : AUVM_CLS_MEMORY;
}

namespace {

struct V {
  const Kernel& k;
  const std::vector<Tensor>& T;
  std::ostringstream err;
  bool ok = true;

  void fail(const std::string& m) {
    if (ok) err << m;
    ok = false;
  }
  const Tensor& t(int i) { return T[k.ids[i]]; }
  // operand i: allowed dtype mask (bit per dtype), minimum elements, mode mask
  void need(int i, unsigned dtmask, uint64_t elems, const char* what) {
    if (!ok) return;
    const Tensor& x = t(i);
    if (!(dtmask & (1u << x.dtype))) {
      fail(std::string("operand ") + what + " has an unsupported dtype");
      return;
    }
    if (x.bytes < elems * dtype_size(x.dtype)) {
      std::ostringstream m;
      m << "operand " << what << " holds " << x.bytes << " B, shape needs "
        << elems * dtype_size(x.dtype);
      fail(m.str());
    }
  }
  void mode(int i, unsigned allowed_mask, const char* what) {
    if (!ok) return;
    if (!(allowed_mask & (1u << k.modes[i]))) fail(std::string("operand ") + what + " has the wrong mode");
  }
  void count(size_t lo, size_t hi) {
    if (k.ids.size() < lo || k.ids.size() > hi) fail("wrong operand count for the op");
  }
  void pos(int i, const char* what) {
    if (k.shape[i] <= 0) fail(std::string("shape ") + what + " must be positive");
  }
};

constexpr unsigned F32 = 1u << AUVM_F32, BF16 = 1u << AUVM_BF16, I32 = 1u << AUVM_I32,
                   U8 = 1u << AUVM_U8, FP = F32 | BF16;
constexpr unsigned MR = 1u << AUVM_R, MW = 1u << AUVM_W, MRW = 1u << AUVM_RW;

}  // namespace

std::string validate_kernel(const Kernel& k, const std::vector<Tensor>& T) {
  V v{k, T, {}};
  const int64_t* s = k.shape;
  for (size_t i = 0; i < k.modes.size(); ++i)
    if (k.modes[i] < 1 || k.modes[i] > 3) v.fail("bad access mode");
  switch (k.op) {
    case AUVM_OP_TOUCH: {
      v.count(2, 8);
      if (!v.ok) break;
      if (s[0] < 0) v.fail("negative log slot");
      v.need(0, F32 | I32 | U8, 0, "log");
      v.mode(0, MRW, "log");
      if (v.ok && T[k.ids[0]].bytes < 64 * uint64_t(s[0] + 1)) v.fail("log too small for slot");
      for (size_t i = 1; i < k.ids.size(); ++i) {
        if (T[k.ids[i]].bytes % 4 || T[k.ids[i]].bytes == 0) v.fail("touch operand bytes % 4 != 0");
        if (k.ids[i] == k.ids[0]) v.fail("touch data operand aliases the log");
        for (size_t j = 1; j < i; ++j)
          if (k.ids[j] == k.ids[i]) v.fail("touch data operands repeat");
      }
      break;
    }
    case AUVM_OP_EMBED:
      v.count(3, 3);
      v.pos(0, "T"); v.pos(1, "H"); v.pos(2, "V");
      if (!v.ok) break;
      v.need(0, I32, s[0], "ids"); v.mode(0, MR, "ids");
      v.need(1, FP, uint64_t(s[2]) * s[1], "E"); v.mode(1, MR, "E");
      v.need(2, F32, uint64_t(s[0]) * s[1], "x"); v.mode(2, MW | MRW, "x");
      break;
    case AUVM_OP_LAYERNORM:
    case AUVM_OP_RMSNORM: {
      bool ln = k.op == AUVM_OP_LAYERNORM;
      v.count(ln ? 4 : 3, ln ? 4 : 3);
      v.pos(0, "T"); v.pos(1, "H"); v.pos(2, "stride");
      if (!v.ok) break;
      if (s[3] < 0) v.fail("negative row offset");
      uint64_t rows = uint64_t(s[0] - 1) * s[2] + s[3] + 1;
      v.need(0, F32, rows * s[1], "x"); v.mode(0, MR, "x");
      v.need(1, FP, s[1], "g"); v.mode(1, MR, "g");
      if (ln) { v.need(2, FP, s[1], "b"); v.mode(2, MR, "b"); }
      int o = ln ? 3 : 2;
      v.need(o, FP, uint64_t(s[0]) * s[1], "h"); v.mode(o, MW | MRW, "h");
      if (v.ok && T[k.ids[1]].dtype != T[k.ids[o]].dtype) v.fail("gain and output dtypes differ");
      break;
    }
    case AUVM_OP_LINEAR:
    case AUVM_OP_LINEAR_GELU:
    case AUVM_OP_LINEAR_RESID:
    case AUVM_OP_LINEAR_SWIGLU: {
      bool sw = k.op == AUVM_OP_LINEAR_SWIGLU;
      v.count(sw ? 4 : 3, sw ? 4 : 3);
      v.pos(0, "M"); v.pos(1, "N"); v.pos(2, "K");
      if (!v.ok) break;
      uint64_t M = s[0], N = s[1], K = s[2];
      v.need(0, FP, M * K, "a"); v.mode(0, MR, "a");
      v.need(1, FP, N * K, "W"); v.mode(1, MR, "W");
      if (sw) { v.need(2, FP, N * K, "Wu"); v.mode(2, MR, "Wu"); }
      int o = sw ? 3 : 2;
      if (k.op == AUVM_OP_LINEAR_RESID) {
        v.need(o, F32, M * N, "x"); v.mode(o, MRW, "x");
      } else {
        v.need(o, FP, M * N, "c"); v.mode(o, MW | MRW, "c");
      }
      if (!v.ok) break;
      uint32_t da = T[k.ids[0]].dtype, dw = T[k.ids[1]].dtype;
      if (da != dw || (sw && T[k.ids[2]].dtype != dw)) v.fail("activation and weight dtypes differ");
      if (da == AUVM_BF16 && K % 32) v.fail("bf16 GEMM needs K % 32 == 0");
      if (da == AUVM_F32 && T[k.ids[o]].dtype != AUVM_F32) v.fail("fp32 GEMM writes fp32");
      break;
    }
    case AUVM_OP_LINEAR_QKV: {
      v.count(7, 7);
      v.pos(0, "M"); v.pos(1, "N"); v.pos(2, "K");
      if (!v.ok) break;
      uint64_t M = s[0], N = s[1], K = s[2];
      static const char* const wn[3] = {"Wq", "Wk", "Wv"};
      static const char* const on[3] = {"q", "k", "v"};
      v.need(0, FP, M * K, "a"); v.mode(0, MR, "a");
      for (int i = 0; i < 3; ++i) {
        v.need(1 + i, FP, N * K, wn[i]); v.mode(1 + i, MR, wn[i]);
        v.need(4 + i, FP, M * N, on[i]); v.mode(4 + i, MW | MRW, on[i]);
      }
      if (!v.ok) break;
      uint32_t da = T[k.ids[0]].dtype;
      for (int i = 1; i < 4; ++i)
        if (T[k.ids[i]].dtype != da) v.fail("activation and weight dtypes differ");
      for (int i = 5; i < 7; ++i)
        if (T[k.ids[i]].dtype != T[k.ids[4]].dtype) v.fail("q, k and v dtypes differ");
      for (int i = 4; i < 7; ++i)
        for (int j = 0; j < i; ++j)
          if (k.ids[i] == k.ids[j]) v.fail("q, k and v must be distinct tensors, none an input");
      if (da == AUVM_BF16 && K % 32) v.fail("bf16 GEMM needs K % 32 == 0");
      if (da == AUVM_F32 && T[k.ids[4]].dtype != AUVM_F32) v.fail("fp32 GEMM writes fp32");
      break;
    }
    case AUVM_OP_ATTN_QKV: {
      v.count(2, 2);
      v.pos(0, "B"); v.pos(1, "S"); v.pos(2, "nH"); v.pos(3, "d");
      if (!v.ok) break;
      uint64_t rows = uint64_t(s[0]) * s[1], hd = uint64_t(s[2]) * s[3];
      v.need(0, FP, rows * 3 * hd, "qkv"); v.mode(0, MR, "qkv");
      v.need(1, FP, rows * hd, "o"); v.mode(1, MW | MRW, "o");
      if (!v.ok) break;
      if (T[k.ids[0]].dtype != T[k.ids[1]].dtype) v.fail("qkv and o dtypes differ");
      if (s[3] != 32 && s[3] != 64 && s[3] != 128) v.fail("head dim must be 32, 64 or 128");
      break;
    }
    case AUVM_OP_ROPE_KV:
    case AUVM_OP_ATTN_CACHE: {
      bool rope = k.op == AUVM_OP_ROPE_KV;
      v.count(rope ? 5 : 4, 5);
      v.pos(0, "B"); v.pos(1, "S"); v.pos(2, "nH"); v.pos(3, "d"); v.pos(4, "Lmax");
      if (!v.ok) break;
      if (s[5] < 0 || s[5] + s[1] > s[4]) v.fail("positions exceed the cache length");
      uint64_t rows = uint64_t(s[0]) * s[1], hd = uint64_t(s[2]) * s[3];
      uint64_t cache = uint64_t(s[0]) * s[2] * s[4] * s[3];
      if (rope) {
        v.need(0, FP, rows * hd, "q"); v.mode(0, MRW, "q");
        v.need(1, FP, rows * hd, "k"); v.mode(1, MR, "k");
        v.need(2, FP, rows * hd, "v"); v.mode(2, MR, "v");
        v.need(3, FP, cache, "Kc"); v.mode(3, MW | MRW, "Kc");
        v.need(4, FP, cache, "Vc"); v.mode(4, MW | MRW, "Vc");
      } else {
        v.need(0, FP, rows * hd, "q"); v.mode(0, MR, "q");
        v.need(1, FP, cache, "Kc"); v.mode(1, MR, "Kc");
        v.need(2, FP, cache, "Vc"); v.mode(2, MR, "Vc");
        v.need(3, FP, rows * hd, "o"); v.mode(3, MW | MRW, "o");
        if (k.ids.size() > 4) {
          v.need(4, F32, uint64_t(s[0]) * s[2] * s[1], "lse"); v.mode(4, MW | MRW, "lse");
        }
      }
      if (!v.ok) break;
      uint32_t dt = T[k.ids[0]].dtype;
      for (size_t i = 1; i < k.ids.size() && i < 4; ++i)
        if (T[k.ids[i]].dtype != dt) v.fail("attention operand dtypes differ");
      if (s[3] != 32 && s[3] != 64 && s[3] != 128) v.fail("head dim must be 32, 64 or 128");
      break;
    }
    case AUVM_OP_ARGMAX: {
      v.count(2, 3);
      v.pos(0, "B"); v.pos(1, "V");
      if (!v.ok) break;
      v.need(0, F32, uint64_t(s[0]) * s[1], "logits"); v.mode(0, MR, "logits");
      v.need(1, I32, s[0], "tok"); v.mode(1, MW | MRW, "tok");
      if (k.ids.size() > 2) {
        if (s[2] < 0) v.fail("negative gen row");
        v.need(2, I32, uint64_t(s[2] + 1) * s[0], "gen"); v.mode(2, MRW, "gen");
      }
      break;
    }
    case AUVM_OP_MOE_ROUTE: {
      v.count(4, 4);
      v.pos(0, "M"); v.pos(1, "H"); v.pos(2, "E"); v.pos(3, "K");
      if (!v.ok) break;
      if (s[2] > 16 || s[3] > s[2]) v.fail("routing needs K <= E <= 16");
      if (s[1] % 8) v.fail("router needs H % 8 == 0");
      uint64_t M = s[0], H = s[1], E = s[2], K = s[3];
      v.need(0, FP, M * H, "h"); v.mode(0, MR, "h");
      v.need(1, FP, E * H, "Wr"); v.mode(1, MR, "Wr");
      v.need(2, I32, M * K, "rte"); v.mode(2, MW | MRW, "rte");
      v.need(3, F32, M * K, "rtw"); v.mode(3, MW | MRW, "rtw");
      if (v.ok && T[k.ids[0]].dtype != T[k.ids[1]].dtype) v.fail("h and router dtypes differ");
      break;
    }
    case AUVM_OP_MOE_DISPATCH: {
      v.count(3, 3);
      v.pos(0, "M"); v.pos(1, "E"); v.pos(2, "K");
      if (!v.ok) break;
      if (s[1] > 16 || s[2] > s[1]) v.fail("routing needs K <= E <= 16");
      if (s[3] < 0) v.fail("negative log row");
      if (s[0] * s[2] >= (int64_t(1) << 31)) v.fail("M * K must fit 31 bits");
      uint64_t M = s[0], E = s[1], K = s[2];
      v.need(0, I32, M * K, "rte"); v.mode(0, MR, "rte");
      v.need(1, I32, E * (M + 1), "lists"); v.mode(1, MW | MRW, "lists");
      v.need(2, I32, uint64_t(s[3] + 1) * E, "log"); v.mode(2, MRW, "log");
      break;
    }
    case AUVM_OP_MOE_UP:
    case AUVM_OP_MOE_DOWN: {
      const bool up = k.op == AUVM_OP_MOE_UP;
      v.count(5, 5);
      v.pos(0, "M"); v.pos(1, "N"); v.pos(2, "K"); v.pos(4, "n"); v.pos(5, "topk");
      if (!v.ok) break;
      if (s[3] < 0) v.fail("negative expert index");
      if (s[4] > s[0]) v.fail("routed rows exceed M");
      if (s[1] % 64 || s[2] % 64) v.fail("expert GEMMs need N % 64 == 0 and K % 64 == 0");
      if (s[5] > 16) v.fail("topk above 16");
      if (!v.ok) break;
      uint64_t M = s[0], N = s[1], Kd = s[2], e = s[3], K = s[5];
      v.need(0, BF16, M * Kd, up ? "h" : "fe"); v.mode(0, MR, up ? "h" : "fe");
      v.need(1, I32, (e + 1) * (M + 1), "lists"); v.mode(1, MR, "lists");
      if (up) {
        v.need(2, BF16, N * Kd, "Wg"); v.mode(2, MR, "Wg");
        v.need(3, BF16, N * Kd, "Wu"); v.mode(3, MR, "Wu");
        v.need(4, BF16, M * N, "fe"); v.mode(4, MW | MRW, "fe");
      } else {
        v.need(2, F32, M * K, "rtw"); v.mode(2, MR, "rtw");
        v.need(3, BF16, N * Kd, "Wd"); v.mode(3, MR, "Wd");
        v.need(4, F32, M * N, "x"); v.mode(4, MRW, "x");
      }
      break;
    }
    case AUVM_OP_COPY:
      v.count(2, 2); v.pos(0, "bytes");
      if (!v.ok) break;
      v.need(0, F32 | BF16 | I32 | U8, 0, "a"); v.mode(0, MR, "a");
      v.mode(1, MW | MRW, "b");
      if (v.ok && (T[k.ids[0]].bytes < uint64_t(s[0]) || T[k.ids[1]].bytes < uint64_t(s[0])))
        v.fail("copy longer than an operand");
      break;
    case AUVM_OP_TRANSPOSE: {
      v.count(2, 2); v.pos(0, "R"); v.pos(1, "C");
      if (!v.ok) break;
      if (s[0] > (int64_t(1) << 22)) v.fail("transpose rows above 2^22");
      uint64_t n = uint64_t(s[0]) * s[1];
      v.need(0, FP, n, "a"); v.mode(0, MR, "a");
      v.need(1, FP, n, "b"); v.mode(1, MW | MRW, "b");
      if (v.ok && T[k.ids[0]].dtype != T[k.ids[1]].dtype) v.fail("transpose dtypes differ");
      break;
    }
    case AUVM_OP_SWIGLU_ACT:
    case AUVM_OP_SWIGLU_BWD: {
      const bool bwd = k.op == AUVM_OP_SWIGLU_BWD;
      v.count(bwd ? 5 : 3, bwd ? 5 : 3); v.pos(0, "T"); v.pos(1, "F");
      if (!v.ok) break;
      uint64_t n = uint64_t(s[0]) * s[1];
      for (size_t i = 0; i < k.ids.size(); ++i) {
        const bool in = i < (bwd ? 3u : 2u);
        v.need(int(i), FP, n, "operand"); v.mode(int(i), in ? MR : (MW | MRW), "operand");
        if (v.ok && T[k.ids[i]].dtype != T[k.ids[0]].dtype) v.fail("SwiGLU operand dtypes differ");
      }
      break;
    }
    case AUVM_OP_RMSNORM_BWD: {
      v.count(7, 7); v.pos(0, "T"); v.pos(1, "H");
      if (!v.ok) break;
      if (s[2] != 0 && s[2] != 1) v.fail("acc must be 0 or 1");
      uint64_t Tn = s[0], H = s[1];
      v.need(0, F32, Tn * H, "x"); v.mode(0, MR, "x");
      v.need(1, FP, H, "g"); v.mode(1, MR, "g");
      v.need(2, F32, Tn * H, "dy"); v.mode(2, MR, "dy");
      v.need(3, F32, Tn * H, "dx"); v.mode(3, s[2] ? MRW : (MW | MRW), "dx");
      v.need(4, BF16, Tn * H, "dxb"); v.mode(4, MW | MRW, "dxb");
      v.need(5, F32, H, "dg"); v.mode(5, MW | MRW, "dg");
      v.need(6, F32, Tn, "rstd"); v.mode(6, MW | MRW, "rstd");
      break;
    }
    case AUVM_OP_ATTN_BWD: {
      v.count(10, 10); v.pos(0, "B"); v.pos(1, "S"); v.pos(2, "nH"); v.pos(3, "d");
      if (!v.ok) break;
      if (s[3] != 128) v.fail("attention backward needs head dim 128");
      uint64_t n = uint64_t(s[0]) * s[1] * s[2] * s[3], rows = uint64_t(s[0]) * s[2] * s[1];
      const char* nm[10] = {"q", "K", "V", "o", "lse", "do", "dq", "dK", "dV", "D"};
      for (int i = 0; i < 10; ++i) {
        const bool f32 = i == 4 || i == 9;
        v.need(i, f32 ? F32 : BF16, f32 ? rows : n, nm[i]);
        v.mode(i, i < 6 ? MR : (MW | MRW), nm[i]);
      }
      break;
    }
    case AUVM_OP_ROPE_BWD: {
      v.count(5, 5); v.pos(0, "B"); v.pos(1, "S"); v.pos(2, "nH"); v.pos(3, "d");
      if (!v.ok) break;
      if (s[3] % 2) v.fail("head dim must be even");
      uint64_t n = uint64_t(s[0]) * s[1] * s[2] * s[3];
      const char* nm[5] = {"dq", "dK", "dV", "dk", "dv"};
      const unsigned md[5] = {MRW, MR, MR, MW | MRW, MW | MRW};
      for (int i = 0; i < 5; ++i) {
        v.need(i, FP, n, nm[i]); v.mode(i, md[i], nm[i]);
        if (v.ok && T[k.ids[i]].dtype != T[k.ids[0]].dtype) v.fail("RoPE backward dtypes differ");
      }
      break;
    }
    case AUVM_OP_XENT: {
      v.count(4, 4); v.pos(0, "T"); v.pos(1, "V");
      if (!v.ok) break;
      uint64_t Tn = s[0], V = s[1];
      v.need(0, F32, Tn * V, "logits"); v.mode(0, MR, "logits");
      v.need(1, I32, Tn, "labels"); v.mode(1, MR, "labels");
      v.need(2, F32, Tn, "losses"); v.mode(2, MW | MRW, "losses");
      v.need(3, FP, Tn * V, "dlogits"); v.mode(3, MW | MRW, "dlogits");
      break;
    }
    case AUVM_OP_EMBED_BWD: {
      v.count(3, 3); v.pos(0, "T"); v.pos(1, "H"); v.pos(2, "V");
      if (!v.ok) break;
      v.need(0, I32, s[0], "ids"); v.mode(0, MR, "ids");
      v.need(1, F32, uint64_t(s[0]) * s[1], "dx"); v.mode(1, MR, "dx");
      v.need(2, F32, uint64_t(s[2]) * s[1], "dE"); v.mode(2, MW | MRW, "dE");
      break;
    }
    case AUVM_OP_ADAM: {
      v.count(5, 5); v.pos(0, "n"); v.pos(1, "step");
      if (!v.ok) break;
      if (s[2] < 0 || s[3] < 0 || s[3] >= 1000000 || s[4] < 0 || s[4] >= 1000000 || s[5] < 0 || s[6] < 0)
        v.fail("AdamW hyperparameters out of range");
      uint64_t n = s[0];
      v.need(0, F32, n, "g"); v.mode(0, MR, "g");
      v.need(1, F32, n, "p32"); v.mode(1, MRW, "p32");
      v.need(2, F32, n, "m"); v.mode(2, MRW, "m");
      v.need(3, F32, n, "v"); v.mode(3, MRW, "v");
      v.need(4, FP, n, "p"); v.mode(4, MW | MRW, "p");
      break;
    }
    default:
      v.fail("unknown op");
  }
  return v.ok ? std::string() : v.err.str();
}

}  // namespace auvm
