// MoE Gate (the first node of the paper's MoE Gate -> Fused MoE -> Weight Sum
// skeleton, Fig. 1): per token, score the E router logits, pick the top-k
// experts and compute their routing weights.
//
// One 64-lane wavefront per token.  Lane l owns experts l, l+64, ... (up to
// EPL per lane), keeps their selection keys in fp64 registers, and the wave
// runs k rounds of a cross-lane arg-max (larger key wins, equal keys -> lower
// expert index).  Keys and weights are computed in fp64 so the selection is
// decided at a precision where ids are reproducible bit for bit; weights are
// rounded to fp32 once at the end.
#include "common.hpp"
#include "launch.hpp"

namespace moe {

__device__ __forceinline__ void wave_argmax(double& v, int& e) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    double ov = __shfl_xor(v, off);
    int oe = __shfl_xor(e, off);
    if (ov > v || (ov == v && oe < e)) { v = ov; e = oe; }
  }
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

__device__ __forceinline__ double wave_max(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmax(v, __shfl_xor(v, off));
  return v;
}

template <int EPL>
__global__ __launch_bounds__(256) void gate_topk_kernel(
    const float* __restrict__ logits, const float* __restrict__ bias, int T, int E, int k,
    int mode, int renorm, float scale, int32_t* __restrict__ ids, float* __restrict__ w,
    int32_t* __restrict__ ids2, float* __restrict__ w2) {
  const int lane = lane_id();
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;  // uniform per wave
  const float* lg = logits + static_cast<size_t>(t) * E;

  double key[EPL];
  double lv[EPL];  // logit in fp64 (softmax) or sigmoid score (sigmoid)
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = lane + 64 * i;
    if (e < E) {
      const double l = static_cast<double>(lg[e]);
      const double b = bias ? static_cast<double>(bias[e]) : 0.0;
      if (mode == 0) {
        lv[i] = l;
        key[i] = l + b;
      } else {
        const double s = 1.0 / (1.0 + exp(-l));
        lv[i] = s;
        key[i] = s + b;
      }
    } else {
      lv[i] = -INFINITY;
      key[i] = -INFINITY;
    }
  }

  int my_id = 0;
  double my_v = 0.0;
  for (int j = 0; j < k; ++j) {
    double bv = -INFINITY;
    int be = 0x7fffffff;
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (key[i] > bv) { bv = key[i]; be = lane + 64 * i; }  // strict: lower index kept
    wave_argmax(bv, be);
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (lane + 64 * i == be) key[i] = -INFINITY;
    // the owner lane broadcasts the selected expert's logit / score
    double v = 0.0;
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (lane + 64 * i == be) v = lv[i];
    v = wave_sum(v);  // exactly one lane contributed
    if (lane == j) { my_id = be; my_v = v; }
  }

  const bool sel = lane < k;
  double wt;
  if (mode == 0) {
    if (renorm) {
      const double m = wave_max(sel ? my_v : -INFINITY);
      const double z = sel ? exp(my_v - m) : 0.0;
      wt = z / wave_sum(z);
    } else {
      double m = -INFINITY;
#pragma unroll
      for (int i = 0; i < EPL; ++i) m = fmax(m, lv[i]);
      m = wave_max(m);
      double s = 0.0;
#pragma unroll
      for (int i = 0; i < EPL; ++i)
        if (lane + 64 * i < E) s += exp(lv[i] - m);
      wt = exp(my_v - m) / wave_sum(s);
    }
  } else {
    wt = renorm ? my_v / wave_sum(sel ? my_v : 0.0) : my_v;
  }
  wt *= static_cast<double>(scale);
  if (sel) {
    const size_t o = static_cast<size_t>(t) * k + lane;
    ids[o] = my_id;
    w[o] = static_cast<float>(wt);
    if (ids2) ids2[o] = my_id;
    if (w2) w2[o] = static_cast<float>(wt);
  }
}

hipError_t launch_gate_topk(const float* logits, const float* bias, int T, int E, int k, int mode,
                            int renorm, float scale, int32_t* ids, float* w, int32_t* ids2,
                            float* w2, hipStream_t s) {
  const dim3 grid((T + 3) / 4), block(256);
  const int epl = (E + 63) / 64;
#define MOE_GATE_CASE(N)                                                                     \
  hipLaunchKernelGGL(gate_topk_kernel<N>, grid, block, 0, s, logits, bias, T, E, k, mode, \
                     renorm, scale, ids, w, ids2, w2)
  if (epl <= 1) MOE_GATE_CASE(1);
  else if (epl <= 2) MOE_GATE_CASE(2);
  else if (epl <= 4) MOE_GATE_CASE(4);
  else if (epl <= 8) MOE_GATE_CASE(8);
  else MOE_GATE_CASE(16);
#undef MOE_GATE_CASE
  return hipGetLastError();
}

}  // namespace moe
