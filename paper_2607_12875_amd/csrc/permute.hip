// Permute / align: group the T*k routed rows by expert (the data movement
// inside the paper's "Fused MoE" node, Fig. 1 / Fig. 3).
//
// Flat ids f = t*k + j are cut into chunks of C consecutive ids, one
// workgroup per chunk.
//   count pass   per chunk, an LDS-atomic histogram over experts -> counts[c][e]
//   scatter pass every chunk block rebuilds the global layout it needs:
//                totals per expert, segment sizes padded to block_m, an
//                exclusive scan over experts (wave scan + LDS), and the base of
//                its own chunk inside each segment (counts of earlier chunks).
//                The stable rank of each id inside its chunk comes from an LDS
//                bitmap: bit i of row e is set when chunk element i routes to
//                e; rank = popcount of the bits below i.  No ordering depends
//                on atomics, so the result is bit-identical on every run.
// With a single chunk the count pass is skipped and totals come from the
// bitmap itself.
#include "common.hpp"
#include "launch.hpp"

namespace moe {

constexpr int kPermThreads = 1024;
constexpr int kBitmapWords = 8192;  // 32 KiB of LDS: E * C/32 words

int permute_chunk(int E) { return E <= 256 ? 1024 : (E <= 512 ? 512 : 256); }

__global__ __launch_bounds__(kPermThreads) void permute_count_kernel(
    const int32_t* __restrict__ ids, int n, int E, int C, int32_t* __restrict__ counts) {
  __shared__ int hist[1024];
  for (int e = threadIdx.x; e < E; e += blockDim.x) hist[e] = 0;
  __syncthreads();
  const int f = blockIdx.x * C + threadIdx.x;
  if (threadIdx.x < C && f < n) {
    const int e = ids[f];
    if (e >= 0 && e < E) atomicAdd(&hist[e], 1);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x) counts[blockIdx.x * E + e] = hist[e];
}

// Inclusive scan inside each 16-lane row of the wave with DPP shifts
// (row_shr:n, 0x110 + n; lanes whose source falls before the row read 0):
// VALU lane moves in place of ds_bpermute round trips.
__device__ __forceinline__ int row_inclusive_scan(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, true);
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, true);
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, true);
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, true);
  return v;
}

// Inclusive scan of one int per thread across the block (blockDim = 1024):
// rows of 16 lanes, then the rows of each wave joined with row_bcast:15
// (0x142: lane 15 of rows 0 and 2 added to rows 1 and 3) and row_bcast:31
// (0x143: lane 31 added to rows 2 and 3), then the waves through LDS.
__device__ __forceinline__ int block_inclusive_scan(int v, int* wave_tot) {
  const int lane = lane_id(), wv = threadIdx.x >> 6;
  v = row_inclusive_scan(v);
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);
  if (lane == 63) wave_tot[wv] = v;
  __syncthreads();
  if (wv == 0) {
    static_assert(kPermThreads / 64 <= 16, "the wave totals fit one row");
    int t = lane < (kPermThreads / 64) ? wave_tot[lane] : 0;
    t = row_inclusive_scan(t);
    if (lane < (kPermThreads / 64)) wave_tot[lane] = t;
  }
  __syncthreads();
  if (wv > 0) v += wave_tot[wv - 1];
  return v;
}

__global__ __launch_bounds__(kPermThreads) void permute_scatter_kernel(
    const int32_t* __restrict__ ids, int n, int E, int C, int block_m, int nchunks,
    const int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
    int32_t* __restrict__ sorted_ids, int32_t* __restrict__ inv_pos, int cap) {
  __shared__ __attribute__((aligned(16))) uint32_t bitmap[kBitmapWords];
  __shared__ int base[1024];
  __shared__ int wave_tot[16];
  __shared__ int total_padded;
  const int W = C / 32;  // bitmap words per expert
  const int tid = threadIdx.x;
  const int c = blockIdx.x;

  for (int i = tid; i < E * W; i += kPermThreads) bitmap[i] = 0;
  __syncthreads();
  const int f = c * C + tid;
  int my_e = -1;
  if (tid < C && f < n) {
    my_e = ids[f];
    if (my_e >= 0 && my_e < E) atomicOr(&bitmap[my_e * W + (tid >> 5)], 1u << (tid & 31));
    else my_e = -1;
  }
  __syncthreads();

  // per-expert totals and the count of this expert in earlier chunks
  int tot = 0, pre = 0;
  if (tid < E) {
    if (counts == nullptr) {
      for (int w = 0; w < W; ++w) tot += __popc(bitmap[tid * W + w]);
    } else {
      // every chunk's count of expert tid, up to 64 loads in flight at a time
      // (one round of memory latency up to 64 chunks, i.e. 65536 routed rows;
      // indices clamped so the loads issue unconditionally)
      for (int c0 = 0; c0 < nchunks; c0 += 64) {
        int v[64];
#pragma unroll
        for (int u = 0; u < 64; ++u) v[u] = counts[min(c0 + u, nchunks - 1) * E + tid];
#pragma unroll
        for (int u = 0; u < 64; ++u) {
          const int cc = c0 + u;
          if (cc < nchunks) tot += v[u];
          if (cc < c) pre += v[u];
        }
      }
    }
  }
  const int padded = (tot + block_m - 1) / block_m * block_m;
  const int incl = block_inclusive_scan(tid < E ? padded : 0, wave_tot);
  const int seg0 = incl - padded;  // exclusive offset of expert tid
  if (tid < E) base[tid] = seg0 + pre;
  if (tid == E - 1) total_padded = incl;
  if (c == 0 && tid < E) {
    offsets[tid] = seg0;
    for (int p = seg0 + tot; p < seg0 + padded; ++p) sorted_ids[p] = n;
    if (tid == E - 1) offsets[E] = incl;
  }
  __syncthreads();
  if (c == 0)  // pads after the last segment, up to the capacity
    for (int p = total_padded + tid; p < cap; p += kPermThreads) sorted_ids[p] = n;

  if (my_e >= 0) {
    const uint32_t* row = bitmap + my_e * W;  // 16-byte aligned: W is a multiple of 4
    const int wi = tid >> 5;
    int rank = __popc(row[wi] & ((1u << (tid & 31)) - 1u));
    for (int w = 0; w + 4 <= wi; w += 4) {  // the whole words below, four per read
      const u32x4 q = *reinterpret_cast<const u32x4*>(row + w);
      rank += __popc(q.x) + __popc(q.y) + __popc(q.z) + __popc(q.w);
    }
    for (int w = wi & ~3; w < wi; ++w) rank += __popc(row[w]);
    const int pos = base[my_e] + rank;
    sorted_ids[pos] = f;
    inv_pos[f] = pos;
  } else if (tid < C && f < n) {
    inv_pos[f] = -1;
  }
}

size_t permute_workspace_bytes(int T, int k, int E) {
  const long n = static_cast<long>(T) * k;
  const int C = permute_chunk(E);
  const long nchunks = (n + C - 1) / C;
  if (nchunks <= 1) return 0;
  return static_cast<size_t>((nchunks * E * 4 + 255) / 256 * 256);
}

hipError_t launch_permute(const int32_t* ids, int T, int k, int E, int block_m, int32_t* offsets,
                          int32_t* sorted_ids, int32_t* inv_pos, int cap, void* ws,
                          hipStream_t s) {
  const int n = T * k;
  const int C = permute_chunk(E);
  const int nchunks = n == 0 ? 1 : (n + C - 1) / C;
  int32_t* counts = nullptr;
  if (nchunks > 1) {
    counts = static_cast<int32_t*>(ws);
    hipLaunchKernelGGL(permute_count_kernel, dim3(nchunks), dim3(kPermThreads), 0, s, ids, n, E,
                       C, counts);
  }
  hipLaunchKernelGGL(permute_scatter_kernel, dim3(nchunks), dim3(kPermThreads), 0, s, ids, n, E,
                     C, block_m, nchunks, counts, offsets, sorted_ids, inv_pos, cap);
  return hipGetLastError();
}

}  // namespace moe
