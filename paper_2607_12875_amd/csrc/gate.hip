// MoE Gate (the first node of the paper's MoE Gate -> Fused MoE -> Weight Sum
// skeleton, Fig. 1): per token, score the E router logits, pick the top-k
// experts and compute their routing weights.
//
// One 64-lane wavefront per token, two selection algorithms (below), chosen
// by the number of experts.  Lane l owns experts l, l+64, ... (up to EPL per
// lane) and computes their selection keys in fp64; the order is
// larger key first, equal keys -> lower expert index.  Keys and weights are
// computed in fp64 so the selection is decided at a precision where ids are
// reproducible bit for bit; weights are rounded to fp32 once at the end.
#include "common.hpp"
#include "launch.hpp"

namespace moe {

constexpr int MOE_GATE_MAX_K = 32;  // the ABI's top_k limit

#ifndef MOE_GATE_RANK_MAX_EPL
#define MOE_GATE_RANK_MAX_EPL 1  // rank selection up to 64 experts, arg-max rounds above
#endif

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

// Arg-max selection: k rounds of a cross-lane arg-max over the keys held in
// registers.  Its work per token grows with k * log2(64), not with E, so it
// wins once there are many experts per lane and enough tokens to hide the
// shuffle latency.
template <int EPL>
__global__ __launch_bounds__(256) void gate_argmax_kernel(
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

// Rank selection: every key goes to LDS; lane l counts, for each key it owns,
// the keys that beat it (larger, or equal at a lower expert index).  That
// rank is the key's slot in descending order, so the k winners write their
// id directly; no sequential arg-max rounds.  Keys stay fp64 throughout.
template <int EPL>
__global__ __launch_bounds__(256) void gate_rank_kernel(
    const float* __restrict__ logits, const float* __restrict__ bias, int T, int E, int k,
    int mode, int renorm, float scale, int32_t* __restrict__ ids, float* __restrict__ w,
    int32_t* __restrict__ ids2, float* __restrict__ w2) {
  __shared__ double skey[4][EPL * 64];
  __shared__ double sval[4][EPL * 64];  // logit (softmax) or sigmoid score, for the weights
  __shared__ double sel[4][MOE_GATE_MAX_K];
  const int lane = lane_id(), wv = threadIdx.x >> 6;
  const int t = blockIdx.x * 4 + wv;
  if (t >= T) return;  // uniform per wave; waves never wait on each other below
  const float* lg = logits + static_cast<size_t>(t) * E;

  double key[EPL], lv[EPL];
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
        const double sg = 1.0 / (1.0 + exp(-l));
        lv[i] = sg;
        key[i] = sg + b;
      }
    } else {
      lv[i] = -INFINITY;
      key[i] = -INFINITY;
    }
    skey[wv][e] = key[i];
    sval[wv][e] = lv[i];
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

  int rank[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) rank[i] = 0;
#pragma unroll 4
  for (int e2 = 0; e2 < E; ++e2) {
    const double k2 = skey[wv][e2];  // same address in every lane: a broadcast read
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = lane + 64 * i;
      rank[i] += (k2 > key[i]) || (k2 == key[i] && e2 < e);
    }
  }
  __builtin_amdgcn_wave_barrier();  // every lane is done reading the keys
  int32_t* slot_id = reinterpret_cast<int32_t*>(&skey[wv][0]);  // reused: id of slot j
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = lane + 64 * i;
    if (e < E && rank[i] < k) {
      slot_id[rank[i]] = e;
      sel[wv][rank[i]] = lv[i];
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  if (lane >= k) return;

  const double my_v = sel[wv][lane];
  double wt;
  if (mode == 0) {
    if (renorm) {
      double m = -INFINITY;
      for (int j = 0; j < k; ++j) m = fmax(m, sel[wv][j]);
      double z = 0.0;
      for (int j = 0; j < k; ++j) z += exp(sel[wv][j] - m);
      wt = exp(my_v - m) / z;
    } else {
      double m = -INFINITY;
      for (int e2 = 0; e2 < E; ++e2) m = fmax(m, sval[wv][e2]);
      double z = 0.0;
      for (int e2 = 0; e2 < E; ++e2) z += exp(sval[wv][e2] - m);
      wt = exp(my_v - m) / z;
    }
  } else if (renorm) {
    double z = 0.0;
    for (int j = 0; j < k; ++j) z += sel[wv][j];
    wt = my_v / z;
  } else {
    wt = my_v;
  }
  wt *= static_cast<double>(scale);
  const size_t o = static_cast<size_t>(t) * k + lane;
  const int my_id = slot_id[lane];
  ids[o] = my_id;
  w[o] = static_cast<float>(wt);
  if (ids2) ids2[o] = my_id;
  if (w2) w2[o] = static_cast<float>(wt);
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
