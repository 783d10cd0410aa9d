// Router GEMM fused with the MoE Gate (the step in front of the Gate node of
// the paper's MoE skeleton, Fig. 1):
//   logits[t, e] = sum_h hidden[t, h] * w_router[e, h]     (bf16 in, fp32 accumulate)
// followed, in the same kernel, by the gate's top-k selection and routing
// weights on those fp32 logits (gate_select.hpp), so the [T, E] logits never
// make a round trip through HBM and decode saves a launch.
//
// One workgroup per 16-token tile, 4 * KS waves.  Wave w computes the
// 16-expert column tiles (w % 4) + 4 j (EPL of them: 64 * EPL >= E) over K
// slice w / 4 with v_mfma_f32_16x16x32_bf16, the K loop software-pipelined U
// steps ahead (splitting K over more waves shortens each wave's chain of
// dependent loads, which bounds this kernel at small T); the slices' partial
// logits are summed in slice order in LDS, then wave w selects for tokens
// w, w + 4 KS, ...
#include "gate_select.hpp"
#include "launch.hpp"

namespace moe {

#ifndef MOE_GATE_RANK_MAX_EPL
#define MOE_GATE_RANK_MAX_EPL 1
#endif

template <int EPL, int TT, int KS, int U>
__global__ __launch_bounds__(256 * KS) void router_gate_kernel(
    const uint16_t* __restrict__ hidden, const uint16_t* __restrict__ wr, int T, int H, int E, int k, int mode,
    int renorm, float scale, const float* __restrict__ bias, float* __restrict__ logits_out,
    int32_t* __restrict__ ids, float* __restrict__ w, int32_t* __restrict__ ids2, float* __restrict__ w2) {
  constexpr bool RANK = EPL <= MOE_GATE_RANK_MAX_EPL;
  constexpr int NW = 4 * KS;         // waves: 4 column-tile groups x KS slices of K
  constexpr int TM = 16 * TT;        // tokens per workgroup
  constexpr int LDE = 64 * EPL + 4;  // LDS row stride of the logits (floats)
  __shared__ float part[KS][TM][LDE];  // per-slice partial logits; slice 0 then holds the sums
  __shared__ double skey[RANK ? NW : 1][RANK ? EPL * 64 : 1];
  __shared__ double sval[RANK ? NW : 1][RANK ? EPL * 64 : 1];
  __shared__ double ssel[RANK ? NW : 1][RANK ? MOE_GATE_MAX_K : 1];

  const int t0 = blockIdx.x * TM;
  const int lane = lane_id(), wv = threadIdx.x >> 6;
  const int tg = wv % 4, ks = wv / 4;  // column-tile group, K slice
  const int r16 = lane & 15, kg = lane >> 4;
  const int hs = H / KS, h0 = ks * hs;  // this wave's K slice (a multiple of 32 elements)

  // A: token rows t0 + 16 i + r16 (tokens past T re-read the last one; never stored)
  const uint16_t* arow[TT];
#pragma unroll
  for (int i = 0; i < TT; ++i) arow[i] = hidden + static_cast<size_t>(min(t0 + 16 * i + r16, T - 1)) * H + h0 + 8 * kg;
  // B: expert row (tg + 4 j) * 16 + r16 of tile j; rows past E read row 0 and are zeroed
  const uint16_t* brow[EPL];
  bool bval[EPL];
#pragma unroll
  for (int j = 0; j < EPL; ++j) {
    const int e = (tg + 4 * j) * 16 + r16;
    bval[j] = e < E;
    brow[j] = wr + static_cast<size_t>(bval[j] ? e : 0) * H + h0 + 8 * kg;
  }

  f32x4 acc[TT][EPL];
#pragma unroll
  for (int i = 0; i < TT; ++i)
#pragma unroll
    for (int j = 0; j < EPL; ++j) acc[i][j] = f32x4{};
  const int nst = hs / (32 * U);  // pipelined stages of U K-steps; the rest one step at a time
  u32x4 a0[U][TT], b0[U][EPL], a1[U][TT], b1[U][EPL];
#define MOE_ROUTER_LOAD(A, Bv, h_)                                                                  \
  do {                                                                                              \
    _Pragma("unroll") for (int u = 0; u < U; ++u) {                                                 \
      _Pragma("unroll") for (int i = 0; i < TT; ++i) A[u][i] = ld16(arow[i] + (h_) + 32 * u);      \
      _Pragma("unroll") for (int j = 0; j < EPL; ++j) Bv[u][j] = ld16(brow[j] + (h_) + 32 * u);     \
    }                                                                                               \
  } while (0)
#define MOE_ROUTER_MMA(A, Bv)                                                                       \
  do {                                                                                              \
    _Pragma("unroll") for (int u = 0; u < U; ++u)                                                   \
        _Pragma("unroll") for (int j = 0; j < EPL; ++j) {                                           \
      const bf16x8 b = as_bf16x8(bval[j] ? Bv[u][j] : u32x4{});                                     \
      _Pragma("unroll") for (int i = 0; i < TT; ++i) acc[i][j] = mfma16x16x32(as_bf16x8(A[u][i]), b, acc[i][j]); \
    }                                                                                               \
  } while (0)
  if (nst > 0) MOE_ROUTER_LOAD(a0, b0, 0);
  for (int s = 0; s < nst; s += 2) {
    if (s + 1 < nst) MOE_ROUTER_LOAD(a1, b1, (s + 1) * 32 * U);
    MOE_ROUTER_MMA(a0, b0);
    if (s + 2 < nst) MOE_ROUTER_LOAD(a0, b0, (s + 2) * 32 * U);
    if (s + 1 < nst) MOE_ROUTER_MMA(a1, b1);
  }
#undef MOE_ROUTER_LOAD
#undef MOE_ROUTER_MMA
  for (int h = nst * 32 * U; h < hs; h += 32) {
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const bf16x8 b = as_bf16x8(bval[j] ? ld16(brow[j] + h) : u32x4{});
#pragma unroll
      for (int i = 0; i < TT; ++i) acc[i][j] = mfma16x16x32(as_bf16x8(ld16(arow[i] + h)), b, acc[i][j]);
    }
  }

  // D element v of a 16x16 tile: token 4*(lane/16) + v, expert lane%16 of the tile
#pragma unroll
  for (int j = 0; j < EPL; ++j) {
    const int e = (tg + 4 * j) * 16 + r16;
    if (e >= E) continue;
#pragma unroll
    for (int i = 0; i < TT; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) part[ks][16 * i + 4 * kg + v][e] = acc[i][j][v];
  }
  __syncthreads();
  if (KS > 1) {  // sum the slices in slice order into part[0]
    for (int idx = threadIdx.x; idx < TM * E; idx += 256 * KS) {
      const int tl = idx / E, e = idx % E;
      float v = part[0][tl][e];
#pragma unroll
      for (int q = 1; q < KS; ++q) v += part[q][tl][e];
      part[0][tl][e] = v;
    }
    __syncthreads();
  }
  if (logits_out) {
    for (int idx = threadIdx.x; idx < TM * E; idx += 256 * KS) {
      const int tl = idx / E, e = idx % E;
      if (t0 + tl < T) logits_out[static_cast<size_t>(t0 + tl) * E + e] = part[0][tl][e];
    }
  }

  for (int tl = wv; tl < TM; tl += NW) {
    const int t = t0 + tl;
    if (t >= T) break;  // uniform per wave
    const size_t o = static_cast<size_t>(t) * k;
    if constexpr (RANK)
      gate_rank_row<EPL>(&part[0][tl][0], bias, E, k, mode, renorm, scale, ids + o, w + o,
                         ids2 ? ids2 + o : nullptr, w2 ? w2 + o : nullptr, skey[wv], sval[wv], ssel[wv]);
    else
      gate_argmax_row<EPL>(&part[0][tl][0], bias, E, k, mode, renorm, scale, ids + o, w + o,
                           ids2 ? ids2 + o : nullptr, w2 ? w2 + o : nullptr);
  }
}

hipError_t launch_router_gate(const uint16_t* hidden, const uint16_t* wr, int T, int H, int E, int k, int mode,
                              int renorm, float scale, const float* bias, float* logits_out, int32_t* ids,
                              float* w, int32_t* ids2, float* w2, hipStream_t s) {
  const int epl = (E + 63) / 64;
  // KS slices of K per column-tile group (more waves in flight, shorter load
  // chains), U K-steps of 32 loaded ahead per stage; the partial logits of
  // all slices fit in LDS.  H % 128 == 0, so every slice is whole K-steps.
  // One 16-token tile per workgroup: a workgroup that owns whole logits rows
  // reads the whole router matrix, so its time is bounded by one CU's read
  // rate whatever its token count, and 16-token tiles keep the most CUs busy
  // (64-token tiles measured 2.5x slower at 4096 tokens).
#define MOE_ROUTER_CASE(N, TT_, KS_, U_)                                                              \
  hipLaunchKernelGGL((router_gate_kernel<N, TT_, KS_, U_>), dim3((T + 16 * TT_ - 1) / (16 * TT_)), \
                     dim3(256 * KS_), 0, s, hidden, wr, T, H, E, k, mode, renorm, scale, bias, logits_out, ids, w, \
                     ids2, w2)
  if (epl <= 1) MOE_ROUTER_CASE(1, 1, 4, 4);
  else if (epl <= 2) MOE_ROUTER_CASE(2, 1, 4, 2);
  else if (epl <= 4) MOE_ROUTER_CASE(4, 1, 2, 2);
  else if (epl <= 8) MOE_ROUTER_CASE(8, 1, 2, 2);
  else MOE_ROUTER_CASE(16, 1, 1, 1);
#undef MOE_ROUTER_CASE
  return hipGetLastError();
}

}  // namespace moe
