// Weight Sum (the last node of the MoE skeleton, Fig. 1) and the per-(row,
// 128-column) e4m3 activation quantisation the fp8 expert route needs (the
// format semantics Sec. 6.2 asks a quantised route to carry).
#include "common.hpp"
#include "launch.hpp"

namespace moe {

// out[t, h] = sum_j w[t, j] * y[inv_pos[t*k + j], h], j ascending, fp32
// accumulation.  Each thread owns 8 consecutive columns of one token (threads
// laid over all T * H/8 column groups, so no workgroup is left part-empty).
// The slots' positions and weights are read first, then every slot's row
// piece is requested before any is summed (a row load issued behind an index
// load would wait for all earlier row loads: the counts complete in order).
// KC > 0: k == KC, all slots at once; KC == 0: any k, eight slots at a time
// (slots past k re-read the last row and are not summed).  y is read and out
// written exactly once, with non-temporal hints.
template <bool Y_F32, bool OUT_BF16, int KC>
__global__ __launch_bounds__(256) void combine_kernel(
    const void* __restrict__ y, const float* __restrict__ w, const int32_t* __restrict__ inv_pos,
    int T, int H, int k, void* __restrict__ out) {
  constexpr int CH = KC > 0 ? KC : 8;
  typedef float f4 __attribute__((ext_vector_type(4)));
  const int hg = H / 8;
  const long idx = static_cast<long>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= static_cast<long>(T) * hg) return;
  const int t = static_cast<int>(idx / hg), h = static_cast<int>(idx % hg) * 8;
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  for (int j0 = 0; j0 < k; j0 += CH) {
    float wt[CH];
    int pos[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const size_t o = static_cast<size_t>(t) * k + (KC > 0 ? c : min(j0 + c, k - 1));
      wt[c] = w[o];
      pos[c] = inv_pos[o];
    }
    f4 va[CH], vb[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const size_t p = static_cast<size_t>(pos[c]);
      if (Y_F32) {
        const f4* src = reinterpret_cast<const f4*>(static_cast<const float*>(y) + p * H + h);
        va[c] = __builtin_nontemporal_load(src);
        vb[c] = __builtin_nontemporal_load(src + 1);
      } else {
        va[c] = __builtin_nontemporal_load(reinterpret_cast<const f4*>(static_cast<const uint16_t*>(y) + p * H + h));
      }
    }
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      if (KC == 0 && j0 + c >= k) break;
      if (Y_F32) {
        const float v[8] = {va[c].x, va[c].y, va[c].z, va[c].w, vb[c].x, vb[c].y, vb[c].z, vb[c].w};
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = fmaf(wt[c], v[i], acc[i]);
      } else {
        const uint32_t u[4] = {__float_as_uint(va[c].x), __float_as_uint(va[c].y), __float_as_uint(va[c].z),
                               __float_as_uint(va[c].w)};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc[2 * i] = fmaf(wt[c], __uint_as_float(u[i] << 16), acc[2 * i]);
          acc[2 * i + 1] = fmaf(wt[c], __uint_as_float(u[i] & 0xFFFF0000u), acc[2 * i + 1]);
        }
      }
    }
  }
  if (OUT_BF16) {
    const u32x4 o = {pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]), pack_bf16x2(acc[4], acc[5]),
                     pack_bf16x2(acc[6], acc[7])};
    __builtin_nontemporal_store(o, reinterpret_cast<u32x4*>(static_cast<uint16_t*>(out) + static_cast<size_t>(t) * H + h));
  } else {
    f32x4* o = reinterpret_cast<f32x4*>(static_cast<float*>(out) + static_cast<size_t>(t) * H + h);
    __builtin_nontemporal_store(f32x4{acc[0], acc[1], acc[2], acc[3]}, o);
    __builtin_nontemporal_store(f32x4{acc[4], acc[5], acc[6], acc[7]}, o + 1);
  }
}

hipError_t launch_combine(const void* y, bool y_f32, const float* w, const int32_t* inv_pos, int T,
                          int H, int k, bool out_bf16, void* out, hipStream_t s) {
  const long n = static_cast<long>(T) * (H / 8);
  const dim3 grid(static_cast<unsigned>((n + 255) / 256)), block(256);
#define MOE_COMBINE_K(YF, OB, KC) \
  hipLaunchKernelGGL((combine_kernel<YF, OB, KC>), grid, block, 0, s, y, w, inv_pos, T, H, k, out)
#define MOE_COMBINE(YF, OB)                        \
  do {                                             \
    if (k == 6) MOE_COMBINE_K(YF, OB, 6);          \
    else if (k == 8) MOE_COMBINE_K(YF, OB, 8);     \
    else MOE_COMBINE_K(YF, OB, 0);                 \
  } while (0)
  if (y_f32) {
    if (out_bf16) MOE_COMBINE(true, true); else MOE_COMBINE(true, false);
  } else {
    if (out_bf16) MOE_COMBINE(false, true); else MOE_COMBINE(false, false);
  }
#undef MOE_COMBINE
#undef MOE_COMBINE_K
  return hipGetLastError();
}

// Value of the lane that the DPP control CTRL pairs with this one (a VALU
// lane permute, no LDS round trip): quad_perm [1,0,3,2] (0xB1) and [2,3,0,1]
// (0x4E) pair lanes at distance 1 and 2, row_half_mirror (0x141) the two
// quads of each half of a 16-lane row, row_mirror (0x140) the two halves.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Per (row, 128-column group): s = max(amax, 1e-10) / 448 with an IEEE fp32
// divide, q = e4m3(RNE(x / s)) after saturating x / s to +-448.  Sixteen lanes
// (one DPP row) own one group (8 columns each); amax is reduced over the row
// with four DPP steps.  The
// quotients come from one divide per lane, r = 1 / s, and a residual step per
// element: q0 = x r, q = q0 + fma(-q0, s, x) r.  That q can differ from the
// IEEE quotient in its last fp32 bit, but for bf16 x it always lands on the
// same e4m3 code: checked on the device against the divide for every
// positive bf16 amax and every bf16 |x| <= amax, about 1.06e9 pairs (the
// steps are symmetric in sign but for a zero, whose sign is copied back).
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
  amax = fmaxf(amax, dpp_f32<0xB1>(amax));
  amax = fmaxf(amax, dpp_f32<0x4E>(amax));
  amax = fmaxf(amax, dpp_f32<0x141>(amax));
  amax = fmaxf(amax, dpp_f32<0x140>(amax));
  const float sc = fmaxf(amax, 1e-10f) / 448.0f;
  if (!live) return;
  const float r = 1.0f / sc;
  float qv[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float q0 = f[i] * r;
    // (the residual step turns -0 into +0; the quotient keeps x's sign)
    qv[i] = sat_e4m3(__builtin_copysignf(fmaf(fmaf(-q0, sc, f[i]), r, q0), f[i]));
  }
  uint32_t lo = 0, hi = 0;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    lo |= f32x2_to_e4m3(qv[2 * i], qv[2 * i + 1]) << (16 * i);
    hi |= f32x2_to_e4m3(qv[4 + 2 * i], qv[5 + 2 * i]) << (16 * i);
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

// Per (row, 32-column block), the OCP MX rule for e4m3 elements: the shared
// scale X = 2^(floor(log2 amax) - 8) is kept as its E8M0 byte, which is the
// fp32 exponent field of amax minus 8, floored at 0 (an all-zero or tiny block
// takes 2^-127); elements e4m3(RNE(x / X)) saturated to +-448, where x / X is
// the exact product x * 2^(127 - byte).  Four lanes own one block.
__global__ __launch_bounds__(256) void act_quant_mx_kernel(
    const uint16_t* __restrict__ x, int M, int K, uint8_t* __restrict__ q, uint8_t* __restrict__ sx) {
  const long idx = static_cast<long>(blockIdx.x) * 256 + threadIdx.x;  // one per 8 columns
  const long total = static_cast<long>(M) * (K / 8);
  const bool live = idx < total;  // uniform over each block's four lanes (K % 32 == 0)
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
  amax = fmaxf(amax, dpp_f32<0xB1>(amax));
  amax = fmaxf(amax, dpp_f32<0x4E>(amax));
  if (!live) return;
  const uint32_t byte = mx_e8m0_of_amax(amax);
  const float mul = __uint_as_float((254u - byte) << 23);  // 2^(127 - byte), a normal fp32
  uint32_t lo = 0, hi = 0;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    lo |= f32x2_to_e4m3(sat_e4m3(f[2 * i] * mul), sat_e4m3(f[2 * i + 1] * mul)) << (16 * i);
    hi |= f32x2_to_e4m3(sat_e4m3(f[4 + 2 * i] * mul), sat_e4m3(f[5 + 2 * i] * mul)) << (16 * i);
  }
  *reinterpret_cast<uint2*>(q + idx * 8) = make_uint2(lo, hi);
  if ((threadIdx.x & 3) == 0) sx[idx / 4] = static_cast<uint8_t>(byte);
}

hipError_t launch_act_quant_mx(const uint16_t* x, int M, int K, uint8_t* q, uint8_t* sx, hipStream_t st) {
  const long total = static_cast<long>(M) * (K / 8);
  const dim3 grid(static_cast<unsigned>((total + 255) / 256)), block(256);
  hipLaunchKernelGGL(act_quant_mx_kernel, grid, block, 0, st, x, M, K, q, sx);
  return hipGetLastError();
}

// Per (row, 128-column group): -136 times the fp32 sum of the group's values,
// the term the int4 GEMM1 takes off its biased codes (136 + q).  Sixteen
// lanes (one DPP row) own one group, as in the quantiser above.
__global__ __launch_bounds__(256) void group_sum_kernel(const uint16_t* __restrict__ x, int M, int K,
                                                         float* __restrict__ out) {
  const long idx = static_cast<long>(blockIdx.x) * 256 + threadIdx.x;  // one per 8 columns
  const long total = static_cast<long>(M) * (K / 8);
  const bool live = idx < total;
  uint4 v = make_uint4(0, 0, 0, 0);
  if (live) v = *reinterpret_cast<const uint4*>(x + idx * 8);
  const uint32_t u[4] = {v.x, v.y, v.z, v.w};
  float sum = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) sum += __uint_as_float(u[i] << 16) + __uint_as_float(u[i] & 0xFFFF0000u);
  sum += dpp_f32<0xB1>(sum);
  sum += dpp_f32<0x4E>(sum);
  sum += dpp_f32<0x141>(sum);
  sum += dpp_f32<0x140>(sum);
  if (live && (threadIdx.x & 15) == 0) out[idx / 16] = -136.0f * sum;
}

hipError_t launch_group_sum(const uint16_t* x, int M, int K, float* out, hipStream_t st) {
  const long total = static_cast<long>(M) * (K / 8);
  const dim3 grid(static_cast<unsigned>((total + 255) / 256)), block(256);
  hipLaunchKernelGGL(group_sum_kernel, grid, block, 0, st, x, M, K, out);
  return hipGetLastError();
}

}  // namespace moe
