// Achievable-peak probes for the roofline denominators: an MFMA-only loop
// (bf16 32x32x16 or fp8 32x32x64, register operands, no memory traffic in the
// loop) and a streaming copy.  The bench reports what they reach on the box
// beside the published peaks its fractions are priced against.
#include "common.hpp"
#include "moe_peaks.h"

namespace moe {

namespace {

constexpr int kPeakWavesPerCu = 8;  // two waves per SIMD keep the matrix pipe fed
constexpr int kPeakChains = 4;      // independent accumulators per wave

// Each wave runs `iters` rounds of kPeakChains independent MFMAs; the
// accumulators are summed into one float per wave at the end (so the loop is
// not removed).  Operands come from the lane id: their values are irrelevant.
template <bool FP8>
__global__ __launch_bounds__(64 * kPeakWavesPerCu) void mfma_loop_kernel(int iters, float* __restrict__ sink) {
  const int lane = lane_id();
  f32x16 acc[kPeakChains];
#pragma unroll
  for (int c = 0; c < kPeakChains; ++c) acc[c] = f32x16{};
  if constexpr (FP8) {
    i32x8 a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      a[i] = 0x38383838 + lane + i;  // small positive e4m3 codes
      b[i] = 0x30303030 + lane - i;
    }
    for (int it = 0; it < iters; ++it)
#pragma unroll
      for (int c = 0; c < kPeakChains; ++c) acc[c] = mfma32x32x64_fp8(a, b, acc[c]);
  } else {
    bf16x8 a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      a[i] = static_cast<__bf16>(0.001f * (lane + i));
      b[i] = static_cast<__bf16>(0.002f * (lane - i));
    }
    for (int it = 0; it < iters; ++it)
#pragma unroll
      for (int c = 0; c < kPeakChains; ++c) acc[c] = mfma32x32x16(a, b, acc[c]);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kPeakChains; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += acc[c][v];
  if (lane == 0) sink[blockIdx.x * kPeakWavesPerCu + (threadIdx.x >> 6)] = s;
}

// Every 16-byte element of src read once: each wave streams its own
// contiguous chunk of per_wave elements (one 1 KB row of the chunk per
// instruction, eight in flight, non-temporal), folding it with XOR into one
// word per workgroup (so no load is removed).  Chunks per wave measured
// ~7 % above a grid-stride read on MI355X.
__global__ __launch_bounds__(256) void read_kernel(const u32x4* __restrict__ src, size_t n, size_t per_wave,
                                                   uint32_t* __restrict__ sink) {
  constexpr int U = 8;
  const size_t w = (static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x) / 64;
  const size_t b = w * per_wave, e = b + per_wave < n ? b + per_wave : n;
  uint32_t x = 0;
  size_t i = b + (threadIdx.x & 63);
  for (; i + (U - 1) * 64 < e; i += U * 64) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(src + i + u * 64);
#pragma unroll
    for (int u = 0; u < U; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < e; i += 64) {
    const u32x4 v = src[i];
    x ^= v.x ^ v.y ^ v.z ^ v.w;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x ^= __shfl_xor(x, off);
  if ((threadIdx.x & 63) == 0) atomicXor(sink + blockIdx.x, x);
}

// dst[i] = src[i] over n 16-byte elements, grid-stride.
__global__ __launch_bounds__(256) void copy_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst, size_t n) {
  const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
  for (size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) dst[i] = src[i];
}

int cu_count_peak() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    n = 256;
  return n;
}

}  // namespace
}  // namespace moe

extern "C" {

long long moe_peak_mfma_flops_per_launch(int fp8, int iters) {
  if (iters < 1) return 0;
  const long long per_mfma = fp8 ? 2LL * 32 * 32 * 64 : 2LL * 32 * 32 * 16;
  return static_cast<long long>(moe::cu_count_peak()) * moe::kPeakWavesPerCu * iters * moe::kPeakChains * per_mfma;
}

int moe_peak_sink_elems(void) { return moe::cu_count_peak() * 8; }

moe_status moe_peak_mfma(int fp8, int iters, float* sink, hipStream_t stream) {
  if (!sink) return MOE_ERR_NULL;
  if (iters < 1 || (fp8 != 0 && fp8 != 1)) return MOE_ERR_SHAPE;
  const dim3 grid(static_cast<unsigned>(moe::cu_count_peak())), block(64 * moe::kPeakWavesPerCu);
  if (fp8) hipLaunchKernelGGL(moe::mfma_loop_kernel<true>, grid, block, 0, stream, iters, sink);
  else hipLaunchKernelGGL(moe::mfma_loop_kernel<false>, grid, block, 0, stream, iters, sink);
  return hipGetLastError() == hipSuccess ? MOE_OK : MOE_ERR_HIP;
}

moe_status moe_peak_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t stream) {
  if (!src || !sink) return MOE_ERR_NULL;
  if (bytes % 16 != 0) return MOE_ERR_SHAPE;
  if (reinterpret_cast<uintptr_t>(src) % 16 != 0) return MOE_ERR_ALIGN;
  if (bytes == 0) return MOE_OK;
  const unsigned wgs = static_cast<unsigned>(moe::cu_count_peak() * 4);  // <= moe_peak_sink_elems()
  const size_t n = bytes / 16, waves = static_cast<size_t>(wgs) * 4;
  hipLaunchKernelGGL(moe::read_kernel, dim3(wgs), dim3(256), 0, stream, static_cast<const moe::u32x4*>(src), n,
                     (n + waves - 1) / waves, sink);
  return hipGetLastError() == hipSuccess ? MOE_OK : MOE_ERR_HIP;
}

moe_status moe_peak_copy(const void* src, void* dst, size_t bytes, hipStream_t stream) {
  if (!src || !dst) return MOE_ERR_NULL;
  if (bytes % 16 != 0) return MOE_ERR_SHAPE;
  if ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) % 16 != 0) return MOE_ERR_ALIGN;
  if (bytes == 0) return MOE_OK;
  const dim3 grid(static_cast<unsigned>(moe::cu_count_peak() * 8)), block(256);
  hipLaunchKernelGGL(moe::copy_kernel, grid, block, 0, stream, static_cast<const moe::u32x4*>(src),
                     static_cast<moe::u32x4*>(dst), bytes / 16);
  return hipGetLastError() == hipSuccess ? MOE_OK : MOE_ERR_HIP;
}

}  // extern "C"
