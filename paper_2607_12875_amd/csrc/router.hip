// Router GEMM in front of the MoE Gate (the step before the Gate node of the
// paper's MoE skeleton, Fig. 1):
//   logits[t, e] = sum_h hidden[t, h] * w_router[e, h]     (bf16 in, fp32 accumulate)
// followed by the gate's top-k selection and routing weights on those fp32
// logits (gate_select.hpp).  Two forms, by batch size:
//  * up to 64 tokens (decode), two launches: the logits GEMM spread over many
//    workgroups in K slices (a workgroup that owned whole logits rows would
//    read the whole router matrix and be bound by one CU's read rate: 40 us on
//    a 16-token decode step), then one wave per token that sums the slices in
//    slice order -- a fixed order, so the logits are the same on every run --
//    and selects;
//  * above, one kernel, one workgroup per 16-token tile (router_gate_kernel):
//    there are enough tiles to occupy the CUs, and the [T, E] logits stay in
//    LDS.
//
// router_gate_kernel: 4 * KS waves.  Wave w computes the
// 16-expert column tiles (w % 4) + 4 j (EPL of them: 64 * EPL >= E) over K
// slice w / 4 with v_mfma_f32_16x16x32_bf16, the K loop software-pipelined U
// steps ahead (splitting K over more waves shortens each wave's chain of
// dependent loads); the slices' partial logits are summed in slice order in
// LDS, then wave w selects for tokens w, w + 4 KS, ...
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
  __shared__ __attribute__((aligned(16))) double skey[RANK ? NW : 1][RANK ? EPL * 64 : 1];
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

// router_partial_kernel: workgroup (token tile, 64-expert group, K slice);
// wave w computes the 16 TT tokens x 16 experts tile of experts
// 64 g + 16 w over K slice ks with v_mfma_f32_16x16x32_bf16 (fragments
// loaded straight from HBM/L2 into registers; the four waves of a workgroup
// share the token rows through L1) and stores the fp32 partial logits
// P[ks][t][e].  Every K slice is a whole number of 32-element MFMA steps.
template <int TT, int U>
__global__ __launch_bounds__(256) void router_partial_kernel(const uint16_t* __restrict__ hidden,
                                                             const uint16_t* __restrict__ wr, int T, int H, int E,
                                                             int hs, float* __restrict__ part) {
  const int lane = lane_id(), wv = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int t0 = blockIdx.x * 16 * TT, ks = blockIdx.z, h0 = ks * hs;
  const int e = blockIdx.y * 64 + wv * 16 + r16;  // this lane's expert (B row)
  const bool ev = e < E;
  if (blockIdx.y * 64 + wv * 16 >= E) return;  // a wave with no expert of its own (uniform)
  const uint16_t* arow[TT];
#pragma unroll
  for (int i = 0; i < TT; ++i) arow[i] = hidden + static_cast<size_t>(min(t0 + 16 * i + r16, T - 1)) * H + h0 + 8 * kg;
  const uint16_t* brow = wr + static_cast<size_t>(ev ? e : 0) * H + h0 + 8 * kg;
  f32x4 acc[TT];
#pragma unroll
  for (int i = 0; i < TT; ++i) acc[i] = f32x4{};
  // U K steps per iteration, the next U steps' fragments loaded ahead
  const int n = hs / 32;
  u32x4 a[2][U][TT], b[2][U];
  auto load = [&](int buf, int st) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int h = (st + u) * 32;
      const bool in = st + u < n;
#pragma unroll
      for (int i = 0; i < TT; ++i) a[buf][u][i] = in ? ld16(arow[i] + h) : u32x4{};
      b[buf][u] = in && ev ? ld16(brow + h) : u32x4{};
    }
  };
  load(0, 0);
  for (int st = 0, buf = 0; st < n; st += U, buf ^= 1) {
    if (st + U < n) load(buf ^ 1, st + U);
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int i = 0; i < TT; ++i) acc[i] = mfma16x16x32(as_bf16x8(a[buf][u][i]), as_bf16x8(b[buf][u]), acc[i]);
  }
  // D element v of a 16x16 tile: token 4*(lane/16) + v, expert lane%16 of the tile
  if (!ev) return;
#pragma unroll
  for (int i = 0; i < TT; ++i)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int t = t0 + 16 * i + 4 * kg + v;
      if (t < T) part[(static_cast<size_t>(ks) * T + t) * E + e] = acc[i][v];
    }
}

// One wave per token: logits = the KS partials summed in slice order (fp32),
// written out if asked, then the gate's selection and weights on them.
constexpr int kRouterMaxKS = 32;  // most K slices of the split router

template <int EPL>
__global__ __launch_bounds__(256) void router_select_kernel(const float* __restrict__ part, int KS, int T, int E,
                                                            int k, int mode, int renorm, float scale,
                                                            const float* __restrict__ bias,
                                                            float* __restrict__ logits_out, int32_t* __restrict__ ids,
                                                            float* __restrict__ w, int32_t* __restrict__ ids2,
                                                            float* __restrict__ w2) {
  constexpr bool RANK = EPL <= MOE_GATE_RANK_MAX_EPL;
  __shared__ float lg[4][EPL * 64];
  __shared__ __attribute__((aligned(16))) double skey[RANK ? 4 : 1][RANK ? EPL * 64 : 1];
  __shared__ double sval[RANK ? 4 : 1][RANK ? EPL * 64 : 1];
  __shared__ double ssel[RANK ? 4 : 1][RANK ? MOE_GATE_MAX_K : 1];
  const int wv = threadIdx.x >> 6, lane = lane_id();
  const int t = blockIdx.x * 4 + wv;
  if (t >= T) return;  // uniform per wave
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = lane + 64 * i;
    if (e >= E) continue;
    // every slice's partial is requested before the first is added (one
    // memory round trip; slots past KS re-read the last slice, so there is no
    // branch between the loads), then they are added in slice order (adding
    // +0 for the slots past KS leaves v unchanged: v is never -0)
    float x[kRouterMaxKS];
#pragma unroll
    for (int j = 0; j < kRouterMaxKS; ++j) x[j] = part[(static_cast<size_t>(min(j, KS - 1)) * T + t) * E + e];
    float v = 0.f;
#pragma unroll
    for (int j = 0; j < kRouterMaxKS; ++j) v += j < KS ? x[j] : 0.f;
    lg[wv][e] = v;  // read back below by this same lane only
    if (logits_out) logits_out[static_cast<size_t>(t) * E + e] = v;
  }
  const size_t o = static_cast<size_t>(t) * k;
  if constexpr (RANK)
    gate_rank_row<EPL>(lg[wv], bias, E, k, mode, renorm, scale, ids + o, w + o, ids2 ? ids2 + o : nullptr,
                       w2 ? w2 + o : nullptr, skey[wv], sval[wv], ssel[wv]);
  else
    gate_argmax_row<EPL>(lg[wv], bias, E, k, mode, renorm, scale, ids + o, w + o, ids2 ? ids2 + o : nullptr,
                         w2 ? w2 + o : nullptr);
}

// Rows of the logits product as one expert segment of the grouped GEMM:
// position p holds token p (p < T) or the pad id T, offsets {0, cap}.
__global__ __launch_bounds__(256) void router_rows_kernel(int T, int cap, int32_t* __restrict__ ids,
                                                          int32_t* __restrict__ offs) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < cap) ids[i] = i < T ? i : T;
  if (i == 0) {
    offs[0] = 0;
    offs[1] = cap;
  }
}

namespace {
constexpr int kRouterSplitMaxT = 64;  // the two-launch form's 16-token tiles up to this many tokens
#ifndef MOE_ROUTER_GEMM_MIN_TE
#define MOE_ROUTER_GEMM_MIN_TE (1L << 20)
#endif
// Many tokens times many experts: the logits as a plain GEMM on the tiled
// bf16 kernel (128-token tiles, every workgroup reading its weight tile once
// per K step), then the gate on them.  The single kernel below makes each
// 16-token workgroup read the whole router matrix, which a large E·H makes
// bound by one CU's read rate (307 us on 8192 tokens x 256 experts x 7168).
bool router_as_gemm(int T, int E) {
  return T > kRouterSplitMaxT && E % 8 == 0 && static_cast<long>(T) * E >= MOE_ROUTER_GEMM_MIN_TE;
}
size_t align256(size_t b) { return (b + 255) / 256 * 256; }
size_t router_gemm_cap(int T) {
  const int bm = bf16_tiled_block_m();
  return static_cast<size_t>((T + bm - 1) / bm) * bm;
}
// From 65 to kRouterMidMaxT tokens the two-launch form takes 64-token tiles
// (four 16-token tiles per workgroup, each weight fragment used four times):
// there the single kernel has too few 16-token workgroups to fill the device
// (router stage, two-launch / single kernel: 18.6 / 38.6 us at 256 tokens and
// 64 experts, 32.7 / 57.5 at 512 and 128, 30.6 / 42.4 at 1024 and 64;
// at 2048 tokens the single kernel is ahead).
constexpr int kRouterMidMaxT = 1024;
constexpr int kMidTT = 4;
bool router_split(int T) { return T <= kRouterMidMaxT; }
// K slices of the split router: enough workgroups to spread the router matrix
// over the CUs, slices of at least 128 elements, at most 32 of them.
int router_ks(int T, int H, int E) {
  const int tt = T > kRouterSplitMaxT ? kMidTT : 1;
  const long tiles = static_cast<long>((T + 16 * tt - 1) / (16 * tt)) * ((E + 63) / 64);
  int ks = 1;
  while (ks < kRouterMaxKS && tiles * ks < 256 && H % (64 * ks) == 0 && H / (2 * ks) >= 128) ks *= 2;
  return ks;
}
}  // namespace

size_t router_workspace_bytes(int T, int H, int E) {
  if (router_as_gemm(T, E))  // row ids, segment offsets, logits
    return align256(router_gemm_cap(T) * sizeof(int32_t)) + 256 + align256(static_cast<size_t>(T) * E * sizeof(float));
  if (!router_split(T)) return 0;
  return static_cast<size_t>(router_ks(T, H, E)) * T * E * sizeof(float);
}

hipError_t launch_router_gate(const uint16_t* hidden, const uint16_t* wr, int T, int H, int E, int k, int mode,
                              int renorm, float scale, const float* bias, float* logits_out, int32_t* ids,
                              float* w, int32_t* ids2, float* w2, void* ws, hipStream_t s) {
  const int epl = (E + 63) / 64;
  if (router_as_gemm(T, E)) {
    const size_t cap = router_gemm_cap(T);
    int32_t* rows = static_cast<int32_t*>(ws);
    int32_t* offs = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + align256(cap * sizeof(int32_t)));
    float* lg = reinterpret_cast<float*>(reinterpret_cast<char*>(offs) + 256);
    // the product's y stores are 16-byte: a caller's logits buffer is written
    // directly when it is 16-byte aligned, else the gate reads the workspace
    // copy and it is copied out after
    const bool direct = logits_out && reinterpret_cast<uintptr_t>(logits_out) % 16 == 0;
    hipLaunchKernelGGL(router_rows_kernel, dim3(static_cast<unsigned>((cap + 255) / 256)), dim3(256), 0, s, T,
                       static_cast<int>(cap), rows, offs);
    GroupedGemm g{};
    g.x = hidden;  // unread by the second product
    g.sorted_ids = rows;
    g.offsets = offs;
    g.T = T;
    g.H = E;  // output columns: the experts
    g.E = 1;  // one segment: every token against the whole router matrix
    g.I = H;  // K
    g.top_k = 1;
    g.n_routed = T;
    g.max_rows = static_cast<int>(cap);
    g.w2 = wr;
    g.inter = const_cast<uint16_t*>(hidden);  // A rows: the hidden rows in order (pad rows are never read)
    g.y = direct ? logits_out : lg;
    hipError_t err = launch_gemm2_bf16_tiled(g, s);
    if (err != hipSuccess) return err;
    err = launch_gate_topk(direct ? logits_out : lg, bias, T, E, k, mode, renorm, scale, ids, w, ids2, w2, s);
    if (err != hipSuccess || !logits_out || direct) return err;
    return hipMemcpyAsync(logits_out, lg, static_cast<size_t>(T) * E * sizeof(float), hipMemcpyDeviceToDevice, s);
  }
  if (!router_split(T)) {
    // KS slices of K per column-tile group, U K-steps of 32 loaded ahead per
    // stage; the partial logits of all slices fit in LDS.  H % 128 == 0, so
    // every slice is whole K-steps.  16-token tiles keep the most CUs busy
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
  const int KS = router_ks(T, H, E), hs = H / KS;
  float* part = static_cast<float*>(ws);
  if (T > kRouterSplitMaxT) {
    const dim3 gm((T + 16 * kMidTT - 1) / (16 * kMidTT), (E + 63) / 64, KS);
    hipLaunchKernelGGL((router_partial_kernel<kMidTT, 4>), gm, dim3(256), 0, s, hidden, wr, T, H, E, hs, part);
  } else {
    const dim3 g1((T + 15) / 16, (E + 63) / 64, KS);
    // all of a short slice's K steps in flight at once
    if (hs <= 128) hipLaunchKernelGGL((router_partial_kernel<1, 4>), g1, dim3(256), 0, s, hidden, wr, T, H, E, hs, part);
    else hipLaunchKernelGGL((router_partial_kernel<1, 8>), g1, dim3(256), 0, s, hidden, wr, T, H, E, hs, part);
  }
  const dim3 g2((T + 3) / 4);
#define MOE_ROUTER_SEL(N)                                                                                  \
  hipLaunchKernelGGL(router_select_kernel<N>, g2, dim3(256), 0, s, part, KS, T, E, k, mode, renorm, scale, \
                     bias, logits_out, ids, w, ids2, w2)
  if (epl <= 1) MOE_ROUTER_SEL(1);
  else if (epl <= 2) MOE_ROUTER_SEL(2);
  else if (epl <= 4) MOE_ROUTER_SEL(4);
  else if (epl <= 8) MOE_ROUTER_SEL(8);
  else MOE_ROUTER_SEL(16);
#undef MOE_ROUTER_SEL
  return hipGetLastError();
}

}  // namespace moe
