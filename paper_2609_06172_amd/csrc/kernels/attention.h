// Causal softmax attention over strided q / k / v views.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace auvm {

// Query i of sequence b, head h sits at position pos0+i and attends to keys
// 0..pos0+i.  Element addresses (in elements of the dtype):
//   q(b,h,i) = q + (b*S + i)*q_rs + h*d
//   k(b,h,j) = k + b*kv_bstride + h*kv_hstride + j*kv_rs   (same for v)
//   o(b,h,i) = o + (b*S + i)*o_rs + h*d
struct AttnArgs {
  const uint8_t *q, *k, *v;
  uint8_t* o;
  int64_t B, S, nH, d, pos0;
  int64_t q_rs, o_rs, kv_rs, kv_bstride, kv_hstride;
  bool bf16;
  // optional [B, nH, S] output: natural log-sum-exp of each query's scaled scores
  float* lse = nullptr;
};

hipError_t launch_attention(const AttnArgs& a, hipStream_t s);

// Causal attention backward, head dim 128, bf16, positions 0..S-1: q, dO, dq
// token-major [B*S, nH*128] (row stride q_rs = nH*128); K, V, dK, dV
// [B, nH, S, 128]; lse (natural) and D = rowsum(dO o) fp32 [B, nH, S].
struct AttnBwdArgs {
  const uint8_t *q, *k, *v, *dO;
  const float *lse, *D;
  uint8_t *dq, *dk, *dv;
  int64_t B, S, nH, q_rs;
};
hipError_t launch_attention_bwd_d128(const AttnBwdArgs& a, hipStream_t s);

}  // namespace auvm
