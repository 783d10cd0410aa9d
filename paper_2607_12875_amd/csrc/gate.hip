// MoE Gate (the first node of the paper's MoE Gate -> Fused MoE -> Weight Sum
// skeleton, Fig. 1): per token, score the E router logits, pick the top-k
// experts and compute their routing weights.  One 64-lane wavefront per
// token; the selection itself (rank or arg-max, chosen by the number of
// experts) is in gate_select.hpp, shared with the router kernel.
#include "gate_select.hpp"
#include "launch.hpp"

namespace moe {

#ifndef MOE_GATE_RANK_MAX_EPL
#define MOE_GATE_RANK_MAX_EPL 1  // rank selection up to 64 experts, arg-max rounds above
#endif

template <int EPL>
__global__ __launch_bounds__(256) void gate_argmax_kernel(
    const float* __restrict__ logits, const float* __restrict__ bias, int T, int E, int k,
    int mode, int renorm, float scale, int32_t* __restrict__ ids, float* __restrict__ w,
    int32_t* __restrict__ ids2, float* __restrict__ w2) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;  // uniform per wave
  const size_t o = static_cast<size_t>(t) * k;
  gate_argmax_row<EPL>(logits + static_cast<size_t>(t) * E, bias, E, k, mode, renorm, scale, ids + o, w + o,
                       ids2 ? ids2 + o : nullptr, w2 ? w2 + o : nullptr);
}

template <int EPL>
__global__ __launch_bounds__(256) void gate_rank_kernel(
    const float* __restrict__ logits, const float* __restrict__ bias, int T, int E, int k,
    int mode, int renorm, float scale, int32_t* __restrict__ ids, float* __restrict__ w,
    int32_t* __restrict__ ids2, float* __restrict__ w2) {
  __shared__ __attribute__((aligned(16))) double skey[4][EPL * 64];
  __shared__ double sval[4][EPL * 64];  // logit (softmax) or sigmoid score, for the weights
  __shared__ double sel[4][MOE_GATE_MAX_K];
  const int wv = threadIdx.x >> 6;
  const int t = blockIdx.x * 4 + wv;
  if (t >= T) return;  // uniform per wave; waves never wait on each other
  const size_t o = static_cast<size_t>(t) * k;
  gate_rank_row<EPL>(logits + static_cast<size_t>(t) * E, bias, E, k, mode, renorm, scale, ids + o, w + o,
                     ids2 ? ids2 + o : nullptr, w2 ? w2 + o : nullptr, skey[wv], sval[wv], sel[wv]);
}

hipError_t launch_gate_topk(const float* logits, const float* bias, int T, int E, int k, int mode,
                            int renorm, float scale, int32_t* ids, float* w, int32_t* ids2,
                            float* w2, hipStream_t s) {
  const dim3 grid((T + 3) / 4), block(256);
  const int epl = (E + 63) / 64;
#define MOE_GATE_CASE(K, N)                                                              \
  hipLaunchKernelGGL(K<N>, grid, block, 0, s, logits, bias, T, E, k, mode, renorm, scale, \
                     ids, w, ids2, w2)
#define MOE_GATE_DISPATCH(K)                 \
  do {                                       \
    if (epl <= 1) MOE_GATE_CASE(K, 1);       \
    else if (epl <= 2) MOE_GATE_CASE(K, 2);  \
    else if (epl <= 4) MOE_GATE_CASE(K, 4);  \
    else if (epl <= 8) MOE_GATE_CASE(K, 8);  \
    else MOE_GATE_CASE(K, 16);               \
  } while (0)
  if (epl <= MOE_GATE_RANK_MAX_EPL) MOE_GATE_DISPATCH(gate_rank_kernel);
  else MOE_GATE_DISPATCH(gate_argmax_kernel);
#undef MOE_GATE_DISPATCH
#undef MOE_GATE_CASE
  return hipGetLastError();
}

}  // namespace moe
