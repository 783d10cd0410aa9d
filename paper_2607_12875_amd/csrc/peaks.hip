// Achievable-peak probes for the roofline denominators: an MFMA-only loop
// (bf16 32x32x16 or fp8 32x32x64, register operands, no memory traffic in the
// loop), a streaming read and a streaming copy; and two per-CU probes of the
// paths the tiled GEMMs stage their operands through (global -> LDS copies,
// LDS fragment reads).  The bench reports what they reach on the device beside
// the published peaks its fractions are priced against.  Every probe
// computes its addresses outside the timed loop or with a few 32-bit
// operations, so it times the memory path rather than its own arithmetic.
#include "common.hpp"
#include "lds_dma.hpp"
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

// global -> LDS copies (global_load_lds_dwordx4, 1 KB per instruction) by the
// first `waves` of a workgroup's 16 waves, one workgroup per CU.  Workgroup b
// reads region b % 8 of `region` bytes (a power of two; with round-robin
// dispatch the workgroups of one XCD share a region, so a small region stays
// in that XCD's L2).  Each step every issuing wave issues NC copies into a
// 64 KB LDS ring and then waits until at most NC are outstanding, so one
// step's copies stay in flight across the workgroup barrier, as in the
// GEMMs' pipelines.
template <int NC>
__global__ __launch_bounds__(1024) void lds_copy_kernel(const uint8_t* __restrict__ src, uint32_t region_mask,
                                                        int waves, int steps) {
  __shared__ __attribute__((aligned(1024))) uint8_t ring[64 * 1024];
  const int wave = threadIdx.x >> 6, lane = lane_id();
  if (wave >= waves) {
    for (int s = 0; s < steps; ++s) __syncthreads();
    return;
  }
  // region_mask: region - 1 with the low 10 bits cleared (copies start on 1 KB boundaries)
  const size_t region = static_cast<size_t>(region_mask | 1023u) + 1;
  const uint8_t* base = src + static_cast<size_t>(blockIdx.x % 8) * region + lane * 16;
  const uint32_t ring0 = lds_addr(&ring[0]);
  uint32_t blk = (blockIdx.x * 977u + wave) & 0xFFFFFu;
  for (int s = 0; s < steps; ++s) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      dma16(base + ((blk * 1024u) & region_mask), ring0 + ((c * waves + wave) & 63) * 1024);
      blk += waves;
    }
    vm_wait<NC>();
    __syncthreads();
  }
  vm_wait<0>();
}

// ds_read_b128 in the tiled GEMMs' fragment pattern (128-byte rows, 16-byte
// chunk c of row r at slot c ^ ((r >> 1) & 7), lanes l and l + 32 on
// neighbouring chunks of one row), 16 reads in flight per wave, addresses
// precomputed.  The reads are issued as inline asm so that nothing consumes
// them inside the loop; one word per workgroup goes to sink at the end.
__global__ __launch_bounds__(1024) void lds_read_kernel(int iters, uint32_t* __restrict__ sink) {
  __shared__ __attribute__((aligned(1024))) u32x4 tile[4096];  // 512 rows of 128 bytes
  for (int i = threadIdx.x; i < 4096; i += blockDim.x) tile[i] = u32x4{static_cast<unsigned>(i), 1u, 2u, 3u};
  __syncthreads();
  const int lane = lane_id(), wave = threadIdx.x >> 6;
  uint32_t addr[16];
#pragma unroll
  for (int c = 0; c < 16; ++c) {
    const int r = (wave * 32 + (lane & 31) + c * 32) & 511;
    const int ch = ((c & 3) * 2 + (lane >> 5)) ^ ((r >> 1) & 7);
    addr[c] = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(&tile[r * 8 + ch]));
  }
  u32x4 v[16];
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < 16; ++c) asm volatile("ds_read_b128 %0, %1" : "=v"(v[c]) : "v"(addr[c]));
    lds_wait();
#pragma unroll
    for (int c = 0; c < 16; ++c) asm volatile("" ::"v"(v[c]));  // sixteen distinct destinations
  }
  u32x4 x = v[0];
#pragma unroll
  for (int c = 1; c < 16; ++c) x ^= v[c];
  if (threadIdx.x == 0) sink[blockIdx.x] = x.x ^ x.y ^ x.z ^ x.w;
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

long long moe_peak_lds_copy_bytes_per_launch(int waves, int copies, int steps) {
  if (waves < 1 || waves > 16 || (copies != 4 && copies != 8 && copies != 16) || steps < 1) return 0;
  return static_cast<long long>(moe::cu_count_peak()) * waves * copies * steps * 1024LL;
}

moe_status moe_peak_lds_copy(const void* src, size_t region_bytes, int waves, int copies, int steps,
                             hipStream_t stream) {
  if (!src) return MOE_ERR_NULL;
  if (waves < 1 || waves > 16 || (copies != 4 && copies != 8 && copies != 16) || steps < 1 ||
      region_bytes < (64u << 10) || region_bytes > (256u << 20) || (region_bytes & (region_bytes - 1)) != 0)
    return MOE_ERR_SHAPE;
  if (reinterpret_cast<uintptr_t>(src) % 16 != 0) return MOE_ERR_ALIGN;
  const dim3 grid(static_cast<unsigned>(moe::cu_count_peak())), block(1024);
  const auto* p = static_cast<const uint8_t*>(src);
  const uint32_t mask = static_cast<uint32_t>(region_bytes - 1) & ~1023u;  // 1 KB-aligned copy starts
  if (copies == 4) hipLaunchKernelGGL(moe::lds_copy_kernel<4>, grid, block, 0, stream, p, mask, waves, steps);
  else if (copies == 8) hipLaunchKernelGGL(moe::lds_copy_kernel<8>, grid, block, 0, stream, p, mask, waves, steps);
  else hipLaunchKernelGGL(moe::lds_copy_kernel<16>, grid, block, 0, stream, p, mask, waves, steps);
  return hipGetLastError() == hipSuccess ? MOE_OK : MOE_ERR_HIP;
}

long long moe_peak_lds_read_bytes_per_launch(int waves, int iters) {
  if (waves < 1 || waves > 16 || iters < 1) return 0;
  return static_cast<long long>(moe::cu_count_peak()) * waves * 64 * 16 * 16 * static_cast<long long>(iters);
}

moe_status moe_peak_lds_read(int waves, int iters, uint32_t* sink, hipStream_t stream) {
  if (!sink) return MOE_ERR_NULL;
  if (waves < 1 || waves > 16 || iters < 1) return MOE_ERR_SHAPE;
  hipLaunchKernelGGL(moe::lds_read_kernel, dim3(static_cast<unsigned>(moe::cu_count_peak())), dim3(64 * waves), 0,
                     stream, iters, sink);
  return hipGetLastError() == hipSuccess ? MOE_OK : MOE_ERR_HIP;
}

}  // extern "C"
