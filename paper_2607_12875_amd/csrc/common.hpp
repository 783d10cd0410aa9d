// Shared device helpers for the gfx950 (CDNA4) MoE kernels: vector types,
// bf16 / e4m3 conversions, MFMA wrappers and wavefront reductions.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));  // native 16-byte vector (HIP's uint4 is a struct)

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round-to-nearest-even fp32 -> bf16 (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return static_cast<uint32_t>(f32_to_bf16(lo)) | (static_cast<uint32_t>(f32_to_bf16(hi)) << 16);
}

// Two fp32 -> two OCP e4m3fn codes in the low 16 bits (round to nearest even;
// callers saturate to +-448 first).
__device__ __forceinline__ uint32_t f32x2_to_e4m3(float a, float b) {
  return static_cast<uint32_t>(__builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false)) & 0xFFFFu;
}

__device__ __forceinline__ float sat_e4m3(float x) {
  return fminf(fmaxf(x, -448.0f), 448.0f);
}

// D(16x16, fp32) += A(16x32, bf16) * B(32x16, bf16).
// Lane l holds A row (l % 16), B column (l % 16), eight consecutive k of the
// k-group (l / 16); D rows 4*(l/16) + i, column l % 16.
__device__ __forceinline__ f32x4 mfma16x16x32(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// D(32x32, fp32) += A(32x16, bf16) * B(16x32, bf16).
// Lane l holds A row (l % 32), B column (l % 32), eight consecutive k of the
// k-group (l / 32); D element v: row 8*(v/4) + 4*(l/32) + v%4, column l % 32.
__device__ __forceinline__ f32x16 mfma32x32x16(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// D(16x16, fp32) += A(16x128, e4m3) * B(128x16, e4m3); lane l holds 32
// consecutive k of k-group (l / 16) for row / column (l % 16).
__device__ __forceinline__ f32x4 mfma16x16x128_fp8(const i32x8& a, const i32x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// D(32x32, fp32) += A(32x64, e4m3) * B(64x32, e4m3); lane l holds 32
// consecutive k of k-group (l / 32) for row / column (l % 32).
__device__ __forceinline__ f32x16 mfma32x32x64_fp8(const i32x8& a, const i32x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ bf16x8 as_bf16x8(const u32x4& v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, const u32x4& v) { *reinterpret_cast<u32x4*>(p) = v; }

// SiLU(g) * u in fp32 with the hardware reciprocal (v_rcp_f32, about 1 ulp)
// in place of an IEEE divide; g -> -inf gives rcp(inf) = 0, so -0 * u.
__device__ __forceinline__ float silu_mul(float g, float u) {
  return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
}

// Eight OCP MX E2M1 codes (one 32-bit word, byte b holding elements 2b in the
// low nibble and 2b+1 in the high one) -> eight bf16 values times the block
// scale.  v_cvt_scalef32_pk_bf16_fp4 applies its fp32 scale operand through
// the exponent field only, so an E8M0 scale byte s is passed as float(s << 23).
// Each result word is the bf16 pair (element 2b, element 2b+1), taken as a
// whole word.
__device__ __forceinline__ u32x4 mxfp4x8_to_bf16(uint32_t w, float sc) {
  u32x4 r;
  r.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 0));
  r.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 1));
  r.z = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 2));
  r.w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, sc, 3));
  return r;
}

// E8M0 byte of the OCP MX scale X = 2^(floor(log2 amax) - 8) for e4m3
// elements (8: the exponent of e4m3's largest power of two), from the fp32
// exponent field of amax >= 0, floored at byte 0 (2^-127); amax = 0 and
// subnormal amax give 0.
__device__ __forceinline__ uint32_t mx_e8m0_of_amax(float amax) {
  const int ef = static_cast<int>(__float_as_uint(amax) >> 23);
  return static_cast<uint32_t>(ef > 8 ? ef - 8 : 0);
}

// D(32x32, fp32) += A(32x64, OCP MX E2M1) * B(64x32, OCP MX e4m3), both
// with E8M0 block scales per 32 k applied by the instruction (layout measured
// on gfx950 with an in-bounds probe on random data).  Lane l serves row /
// column (l % 32); lane group g = l / 32 supplies the scale of K block g
// (byte OS of sa / sb, biased by 127) for both operands.  A (E2M1, a.s0..s3;
// a.s4..s7 unused): the lane's 32 nibbles are block g (element 2b in the low
// nibble of byte b).  B (e4m3): the lane's bytes 0..15 are elements
// [16 g, 16 g + 16) of block 0, bytes 16..31 the same elements of block 1.
// D element v: row 8*(v/4) + 4*(l/32) + v%4, column l % 32.
template <int OS>
__device__ __forceinline__ f32x16 mfma32x32x64_f4f8(const i32x8& a, const i32x8& b, int sa, int sb,
                                                     const f32x16& c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 4, 0, OS, sa, OS, sb);
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// Index e with off[e] <= p < off[e+1] (off non-decreasing, off[0] = 0 <= p < off[E]).
__device__ __forceinline__ int find_segment(const int32_t* __restrict__ off, int E, int p) {
  int lo = 0, hi = E;  // invariant: off[lo] <= p < off[hi]
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (off[mid] <= p) lo = mid; else hi = mid;
  }
  return lo;
}

}  // namespace moe
