// Weight Sum (the last node of the MoE skeleton, Fig. 1) and the per-(row,
// 128-column) e4m3 activation quantisation the fp8 expert route needs (the
// format semantics Sec. 6.2 asks a quantised route to carry).
#include "common.hpp"
#include "launch.hpp"

namespace moe {

// out[t, h] = sum_j w[t, j] * y[inv_pos[t*k + j], h], j ascending, fp32
// accumulation.  Each thread owns 8 consecutive columns: one 16-byte load per
// routed row, one or two 16-byte stores.
template <bool Y_F32, bool OUT_BF16>
__global__ __launch_bounds__(256) void combine_kernel(
    const void* __restrict__ y, const float* __restrict__ w, const int32_t* __restrict__ inv_pos,
    int T, int H, int k, void* __restrict__ out) {
  const int t = blockIdx.y;
  const int h = (blockIdx.x * 256 + threadIdx.x) * 8;
  if (h >= H) return;
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  for (int j = 0; j < k; ++j) {
    const float wt = w[static_cast<size_t>(t) * k + j];
    const int p = inv_pos[static_cast<size_t>(t) * k + j];
    if (Y_F32) {
      const float4* src = reinterpret_cast<const float4*>(static_cast<const float*>(y) +
                                                          static_cast<size_t>(p) * H + h);
      const float4 a = src[0], b = src[1];
      const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] = fmaf(wt, v[i], acc[i]);
    } else {
      const uint4 v = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(y) +
                                                      static_cast<size_t>(p) * H + h);
      const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[2 * i] = fmaf(wt, __uint_as_float(u[i] << 16), acc[2 * i]);
        acc[2 * i + 1] = fmaf(wt, __uint_as_float(u[i] & 0xFFFF0000u), acc[2 * i + 1]);
      }
    }
  }
  if (OUT_BF16) {
    uint4 o;
    o.x = pack_bf16x2(acc[0], acc[1]);
    o.y = pack_bf16x2(acc[2], acc[3]);
    o.z = pack_bf16x2(acc[4], acc[5]);
    o.w = pack_bf16x2(acc[6], acc[7]);
    *reinterpret_cast<uint4*>(static_cast<uint16_t*>(out) + static_cast<size_t>(t) * H + h) = o;
  } else {
    float4* o = reinterpret_cast<float4*>(static_cast<float*>(out) + static_cast<size_t>(t) * H + h);
    o[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
    o[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
  }
}

hipError_t launch_combine(const void* y, bool y_f32, const float* w, const int32_t* inv_pos, int T,
                          int H, int k, bool out_bf16, void* out, hipStream_t s) {
  const dim3 grid((H / 8 + 255) / 256, T), block(256);
#define MOE_COMBINE(YF, OB) \
  hipLaunchKernelGGL((combine_kernel<YF, OB>), grid, block, 0, s, y, w, inv_pos, T, H, k, out)
  if (y_f32) {
    if (out_bf16) MOE_COMBINE(true, true); else MOE_COMBINE(true, false);
  } else {
    if (out_bf16) MOE_COMBINE(false, true); else MOE_COMBINE(false, false);
  }
#undef MOE_COMBINE
  return hipGetLastError();
}

// Per (row, 128-column group): s = max(amax, 1e-10) / 448 with an IEEE fp32
// divide, q = e4m3(RNE(x / s)) after saturating x / s to +-448.  Sixteen lanes
// own one group (8 columns each); amax is reduced with lane shuffles.
__global__ __launch_bounds__(256) void act_quant_kernel(
    const uint16_t* __restrict__ x, int M, int K, uint8_t* __restrict__ q, float* __restrict__ s) {
  const long idx = static_cast<long>(blockIdx.x) * 256 + threadIdx.x;  // one per 8 columns
  const long total = static_cast<long>(M) * (K / 8);
  const bool live = idx < total;
  uint4 v = make_uint4(0, 0, 0, 0);
  if (live) v = *reinterpret_cast<const uint4*>(x + idx * 8);
  const uint32_t u[4] = {v.x, v.y, v.z, v.w};
  float f[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(u[i] << 16);
    f[2 * i + 1] = __uint_as_float(u[i] & 0xFFFF0000u);
  }
  float amax = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) amax = fmaxf(amax, fabsf(f[i]));
#pragma unroll
  for (int off = 1; off < 16; off <<= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
  const float sc = fmaxf(amax, 1e-10f) / 448.0f;
  if (!live) return;
  uint32_t lo = 0, hi = 0;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    lo |= f32x2_to_e4m3(sat_e4m3(f[2 * i] / sc), sat_e4m3(f[2 * i + 1] / sc)) << (16 * i);
    hi |= f32x2_to_e4m3(sat_e4m3(f[4 + 2 * i] / sc), sat_e4m3(f[5 + 2 * i] / sc)) << (16 * i);
  }
  *reinterpret_cast<uint2*>(q + idx * 8) = make_uint2(lo, hi);
  if ((threadIdx.x & 15) == 0) s[idx / 16] = sc;
}

hipError_t launch_act_quant(const uint16_t* x, int M, int K, uint8_t* q, float* s, hipStream_t st) {
  const long total = static_cast<long>(M) * (K / 8);
  const dim3 grid(static_cast<unsigned>((total + 255) / 256)), block(256);
  hipLaunchKernelGGL(act_quant_kernel, grid, block, 0, st, x, M, K, q, s);
  return hipGetLastError();
}

}  // namespace moe
