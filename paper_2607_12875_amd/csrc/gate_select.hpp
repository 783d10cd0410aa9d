// Top-k selection and routing weights of one token on one 64-lane wavefront
// (the MoE Gate node of Fig. 1), shared by the gate kernel (logits read from
// HBM) and the router kernel (logits computed into LDS).
//
// Lane l owns experts l, l+64, ... (up to EPL per lane) and computes their
// selection keys in fp64; the order is larger key first, equal keys -> lower
// expert index.  Keys and weights are computed in fp64 so the selection is
// decided at a precision where ids are reproducible bit for bit; weights are
// rounded to fp32 once at the end.
#pragma once
#include "common.hpp"

namespace moe {

constexpr int MOE_GATE_MAX_K = 32;  // the ABI's top_k limit

// Wave reductions without LDS round trips: four DPP steps (VALU lane
// permutes) inside each row of 16 lanes -- quad_perm [1,0,3,2] (0xB1) and
// [2,3,0,1] (0x4E) pair lanes at distance 1 and 2, row_half_mirror (0x141)
// the two quads of a half row, row_mirror (0x140) the two half rows -- after
// which every lane of a row holds the row's result; the four row results
// are then read as wave-uniform values and combined in row order.  Every
// lane of the wave must take part.
template <int CTRL>
__device__ __forceinline__ int dpp_i32(int v) {
  return __builtin_amdgcn_update_dpp(v, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const unsigned long long b = static_cast<unsigned long long>(__double_as_longlong(v));
  const uint32_t lo = static_cast<uint32_t>(dpp_i32<CTRL>(static_cast<int>(b)));
  const uint32_t hi = static_cast<uint32_t>(dpp_i32<CTRL>(static_cast<int>(b >> 32)));
  return __longlong_as_double(static_cast<long long>(static_cast<unsigned long long>(hi) << 32 | lo));
}
__device__ __forceinline__ double readlane_f64(double v, int l) {
  const unsigned long long b = static_cast<unsigned long long>(__double_as_longlong(v));
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(b), l));
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(b >> 32), l));
  return __longlong_as_double(static_cast<long long>(static_cast<unsigned long long>(hi) << 32 | lo));
}

// (v, e) <- the better of (v, e) and (ov, oe): larger value, equal values ->
// lower index.  A total order, so the reduction's pairing does not matter.
__device__ __forceinline__ void argmax_take(double& v, int& e, double ov, int oe) {
  if (ov > v || (ov == v && oe < e)) { v = ov; e = oe; }
}

__device__ __forceinline__ void wave_argmax(double& v, int& e) {
  argmax_take(v, e, dpp_f64<0xB1>(v), dpp_i32<0xB1>(e));
  argmax_take(v, e, dpp_f64<0x4E>(v), dpp_i32<0x4E>(e));
  argmax_take(v, e, dpp_f64<0x141>(v), dpp_i32<0x141>(e));
  argmax_take(v, e, dpp_f64<0x140>(v), dpp_i32<0x140>(e));
  double bv = readlane_f64(v, 0);
  int be = __builtin_amdgcn_readlane(e, 0);
#pragma unroll
  for (int r = 1; r < 4; ++r) argmax_take(bv, be, readlane_f64(v, 16 * r), __builtin_amdgcn_readlane(e, 16 * r));
  v = bv;
  e = be;
}

__device__ __forceinline__ double wave_sum(double v) {
  v += dpp_f64<0xB1>(v);
  v += dpp_f64<0x4E>(v);
  v += dpp_f64<0x141>(v);
  v += dpp_f64<0x140>(v);
  return ((readlane_f64(v, 0) + readlane_f64(v, 16)) + readlane_f64(v, 32)) + readlane_f64(v, 48);
}

__device__ __forceinline__ double wave_max(double v) {
  v = fmax(v, dpp_f64<0xB1>(v));
  v = fmax(v, dpp_f64<0x4E>(v));
  v = fmax(v, dpp_f64<0x141>(v));
  v = fmax(v, dpp_f64<0x140>(v));
  return fmax(fmax(readlane_f64(v, 0), readlane_f64(v, 16)), fmax(readlane_f64(v, 32), readlane_f64(v, 48)));
}

// Keys (and the values the weights use) of this lane's experts.
template <int EPL>
__device__ __forceinline__ void gate_keys(const float* lg, const float* bias, int E, int mode, double* key,
                                          double* lv) {
  const int lane = lane_id();
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
}

// Arg-max selection: k rounds of a cross-lane arg-max over the keys held in
// registers.  Its work per token grows with k * log2(64), not with E, so it
// wins once there are many experts per lane.  lg: this token's E logits;
// ids/w (and the optional copies ids2/w2): this token's k outputs.
template <int EPL>
__device__ __forceinline__ void gate_argmax_row(const float* lg, const float* bias, int E, int k, int mode,
                                                int renorm, float scale, int32_t* ids, float* w, int32_t* ids2,
                                                float* w2) {
  const int lane = lane_id();
  double key[EPL], lv[EPL];  // lv: logit in fp64 (softmax) or sigmoid score (sigmoid)
  gate_keys<EPL>(lg, bias, E, mode, key, lv);

  // taken: bit i set once expert lane + 64 i has been selected (or does not
  // exist).  A key of -inf (a masked expert) still competes: the first
  // untaken expert a lane sees is its candidate even at -inf, so a token with
  // fewer than k finite keys picks its remaining experts by lowest index, as
  // a stable sort on the keys does.
  uint32_t taken = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i)
    if (lane + 64 * i >= E) taken |= 1u << i;
  int my_id = 0;
  double my_v = 0.0;
  for (int j = 0; j < k; ++j) {
    double bv = -INFINITY;
    int be = 0x7fffffff;
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (!(taken >> i & 1) && (key[i] > bv || be == 0x7fffffff)) {  // strict: lower index kept
        bv = key[i];
        be = lane + 64 * i;
      }
    wave_argmax(bv, be);
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (lane + 64 * i == be) taken |= 1u << i;
    // the owner lane (be % 64: be is the same in every lane) broadcasts the
    // selected expert's logit / score
    double v = 0.0;
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (lane + 64 * i == be) v = lv[i];
    v = readlane_f64(v, be & 63);
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
    ids[lane] = my_id;
    w[lane] = static_cast<float>(wt);
    if (ids2) ids2[lane] = my_id;
    if (w2) w2[lane] = static_cast<float>(wt);
  }
}

// Rank selection: every key goes to LDS; lane l counts, for each key it owns,
// the keys that beat it (larger, or equal at a lower expert index).  That
// rank is the key's slot in descending order, so the k winners write their
// id directly; no sequential arg-max rounds.  Keys stay fp64 throughout.
// skey/sval: EPL*64 doubles of LDS, sel: MOE_GATE_MAX_K doubles, private to
// this wave.  Only waves of one token may call it together (no barrier).
template <int EPL>
__device__ __forceinline__ void gate_rank_row(const float* lg, const float* bias, int E, int k, int mode,
                                              int renorm, float scale, int32_t* ids, float* w, int32_t* ids2,
                                              float* w2, double* skey, double* sval, double* sel) {
  const int lane = lane_id();
  double key[EPL], lv[EPL];
  gate_keys<EPL>(lg, bias, E, mode, key, lv);
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    skey[lane + 64 * i] = key[i];
    sval[lane + 64 * i] = lv[i];
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

  int rank[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) rank[i] = 0;
  // every one of the wave's EPL*64 key slots, two per 16-byte read: slots
  // past E hold -inf at indices above every real expert, so they never beat
  // a real key and the ranks are those over the E experts
#pragma unroll 8
  for (int e2 = 0; e2 < EPL * 64; e2 += 2) {
    const double2 k2 = *reinterpret_cast<const double2*>(skey + e2);  // same address in every lane: a broadcast read
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = lane + 64 * i;
      rank[i] += (k2.x > key[i]) || (k2.x == key[i] && e2 < e);
      rank[i] += (k2.y > key[i]) || (k2.y == key[i] && e2 + 1 < e);
    }
  }
  __builtin_amdgcn_wave_barrier();  // every lane is done reading the keys
  int32_t* slot_id = reinterpret_cast<int32_t*>(skey);  // reused: id of slot j
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = lane + 64 * i;
    if (e < E && rank[i] < k) {
      slot_id[rank[i]] = e;
      sel[rank[i]] = lv[i];
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

  // lane j < k holds selected slot j; the sums and maxima are wave
  // reductions (one exp per lane), every lane taking part
  const bool on = lane < k;
  const double my_v = on ? sel[lane] : 0.0;
  double wt;
  if (mode == 0) {
    if (renorm) {
      const double m = wave_max(on ? my_v : -INFINITY);
      const double z = on ? exp(my_v - m) : 0.0;
      wt = z / wave_sum(z);
    } else {
      double m = -INFINITY;
#pragma unroll
      for (int i = 0; i < EPL; ++i) m = fmax(m, lv[i]);
      m = wave_max(m);
      double zs = 0.0;
#pragma unroll
      for (int i = 0; i < EPL; ++i)
        if (lane + 64 * i < E) zs += exp(lv[i] - m);
      wt = exp(my_v - m) / wave_sum(zs);
    }
  } else {
    wt = renorm ? my_v / wave_sum(my_v) : my_v;
  }
  if (!on) return;
  wt *= static_cast<double>(scale);
  const int my_id = slot_id[lane];
  ids[lane] = my_id;
  w[lane] = static_cast<float>(wt);
  if (ids2) ids2[lane] = my_id;
  if (w2) w2[lane] = static_cast<float>(wt);
}

}  // namespace moe
