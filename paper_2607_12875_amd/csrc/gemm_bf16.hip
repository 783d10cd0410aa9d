// Grouped expert GEMMs for bf16 weights (the "Fused MoE" node, Fig. 1 /
// Fig. 3): per expert e, over the rows of its permuted segment,
//   GEMM1  a = SiLU(x W1[e,:I]^T) * (x W1[e,I:]^T)   (SiLU*up fused in the epilogue)
//   GEMM2  y = a W2[e]^T
// Weights are [N,K] with K contiguous, so both products read B rows along K.
//
// Two kernel families:
//  * tiled  (rows per expert >> 16): BM x BN output tile per workgroup, BK=64
//    slices of A and B staged through LDS (double buffered, 16-byte chunks
//    XOR-swizzled by row so the MFMA fragment reads are bank-conflict free),
//    v_mfma_f32_32x32x16_bf16 with fp32 accumulation.
//  * skinny (decode: a few rows per expert): 16-row tile, the K range split
//    over the four waves, weight fragments streamed from HBM straight into
//    registers (no reuse to stage for), v_mfma_f32_16x16x32_bf16, partial sums
//    reduced through LDS.
// Segments are padded to the row tile, so every tile belongs to one expert;
// tiles past the last segment exit at once.
#include "common.hpp"
#include "launch.hpp"

namespace moe {

// ----------------------------------------------------------------- tiled
template <int BM, int BN, int WM, int WN, bool GEMM1>
__global__ __launch_bounds__(WM * WN * 64) void gemm_bf16_tiled(GroupedGemm g) {
  constexpr int NT = WM * WN * 64;
  constexpr int BK = 64;
  constexpr int NB = GEMM1 ? 2 * BN : BN;   // B tile rows (gate + up for GEMM1)
  constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
  constexpr int A_CH = BM * 8 / NT, B_CH = NB * 8 / NT;  // 16-byte chunks per thread
  static_assert(A_CH * NT == BM * 8 && B_CH * NT == NB * 8, "tile/thread mismatch");
  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * BK];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][NB * BK];

  const int m0 = blockIdx.x * BM;
  if (m0 >= g.offsets[g.E]) return;
  const int e = find_segment(g.offsets, g.E, m0);
  const int n0 = blockIdx.y * BN;
  const int K = GEMM1 ? g.H : g.I;
  const int tid = threadIdx.x, lane = lane_id(), wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  // global row pointers of this thread's A and B chunks
  const uint16_t* a_ptr[A_CH];
  const uint16_t* b_ptr[B_CH];
  int a_lds[A_CH], b_lds[B_CH];
#pragma unroll
  for (int i = 0; i < A_CH; ++i) {
    const int q = tid + i * NT, r = q >> 3, c = q & 7;
    const uint16_t* row;
    if (GEMM1) {
      const int sid = g.sorted_ids[m0 + r];
      const int tok = sid < g.n_routed ? sid / g.top_k : 0;
      row = static_cast<const uint16_t*>(g.x) + static_cast<size_t>(tok) * g.H;
    } else {
      row = static_cast<const uint16_t*>(g.inter) + static_cast<size_t>(m0 + r) * g.I;
    }
    a_ptr[i] = row + c * 8;
    a_lds[i] = r * BK + ((c ^ (r & 7)) << 3);
  }
  const uint16_t* wbase = static_cast<const uint16_t*>(GEMM1 ? g.w1 : g.w2) +
                          static_cast<size_t>(e) * (GEMM1 ? 2 * g.I : g.H) * K;
#pragma unroll
  for (int i = 0; i < B_CH; ++i) {
    const int q = tid + i * NT, r = q >> 3, c = q & 7;
    int n;
    if (GEMM1) n = r < BN ? n0 + r : g.I + n0 + (r - BN);
    else n = n0 + r;
    b_ptr[i] = wbase + static_cast<size_t>(n) * K + c * 8;
    b_lds[i] = r * BK + ((c ^ (r & 7)) << 3);
  }

  f32x16 acc[TM][TN], acc_u[TM][GEMM1 ? TN : 1];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      acc[i][j] = f32x16{};
      if (GEMM1) acc_u[i][j] = f32x16{};
    }

  uint4 ra[A_CH], rb[B_CH];
  auto load = [&](int k0) {
#pragma unroll
    for (int i = 0; i < A_CH; ++i) ra[i] = *reinterpret_cast<const uint4*>(a_ptr[i] + k0);
#pragma unroll
    for (int i = 0; i < B_CH; ++i) rb[i] = *reinterpret_cast<const uint4*>(b_ptr[i] + k0);
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < A_CH; ++i) *reinterpret_cast<uint4*>(&As[buf][a_lds[i]]) = ra[i];
#pragma unroll
    for (int i = 0; i < B_CH; ++i) *reinterpret_cast<uint4*>(&Bs[buf][b_lds[i]]) = rb[i];
  };

  const int nk = K / BK;
  load(0);
  store(0);
  __syncthreads();
  const int l32 = lane & 31, kg = lane >> 5;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load((kt + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int ch = 2 * kk + kg;
      bf16x8 a[TM], b[TN], bu[GEMM1 ? TN : 1];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = wm * (BM / WM) + i * 32 + l32;
        a[i] = as_bf16x8(*reinterpret_cast<const uint4*>(&As[buf][r * BK + ((ch ^ (r & 7)) << 3)]));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = wn * (BN / WN) + j * 32 + l32;
        b[j] = as_bf16x8(*reinterpret_cast<const uint4*>(&Bs[buf][r * BK + ((ch ^ (r & 7)) << 3)]));
        if (GEMM1) {
          const int ru = BN + r;
          bu[j] = as_bf16x8(*reinterpret_cast<const uint4*>(&Bs[buf][ru * BK + ((ch ^ (ru & 7)) << 3)]));
        }
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          acc[i][j] = mfma32x32x16(a[i], b[j], acc[i][j]);
          if (GEMM1) acc_u[i][j] = mfma32x32x16(a[i], bu[j], acc_u[i][j]);
        }
    }
    if (kt + 1 < nk) store(buf ^ 1);
    __syncthreads();
  }

  // epilogue: D element v of a 32x32 tile is (row 8*(v/4) + 4*(lane/32) + v%4, col lane%32)
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + wm * (BM / WM) + i * 32 + 8 * (v >> 2) + 4 * kg + (v & 3);
        const int col = n0 + wn * (BN / WN) + j * 32 + l32;
        if (GEMM1) {
          static_cast<uint16_t*>(g.inter)[static_cast<size_t>(row) * g.I + col] =
              f32_to_bf16(silu_mul(acc[i][j][v], acc_u[i][j][v]));
        } else if (g.sorted_ids[row] < g.n_routed) {  // pad rows are never read
          static_cast<float*>(g.y)[static_cast<size_t>(row) * g.H + col] = acc[i][j][v];
        }
      }
}

// ----------------------------------------------------------------- skinny
// NSUB 16-column weight subtiles per workgroup (GEMM1: NSUB/2 gate + NSUB/2
// up subtiles covering the same act columns).
template <int NSUB, int UNROLL, bool GEMM1>
__global__ __launch_bounds__(256) void gemm_bf16_skinny(GroupedGemm g) {
  constexpr int BM = 16;
  constexpr int BN = GEMM1 ? NSUB / 2 * 16 : NSUB * 16;  // output columns
  __shared__ f32x4 red[3][NSUB][64];

  const int m0 = blockIdx.x * BM;
  if (m0 >= g.offsets[g.E]) return;
  const int e = find_segment(g.offsets, g.E, m0);
  const int n0 = blockIdx.y * BN;
  const int K = GEMM1 ? g.H : g.I;
  const int lane = lane_id(), wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;

  const uint16_t* arow;
  if (GEMM1) {
    const int sid = g.sorted_ids[m0 + r16];
    const int tok = sid < g.n_routed ? sid / g.top_k : 0;
    arow = static_cast<const uint16_t*>(g.x) + static_cast<size_t>(tok) * g.H;
  } else {
    arow = static_cast<const uint16_t*>(g.inter) + static_cast<size_t>(m0 + r16) * g.I;
  }
  const uint16_t* wbase = static_cast<const uint16_t*>(GEMM1 ? g.w1 : g.w2) +
                          static_cast<size_t>(e) * (GEMM1 ? 2 * g.I : g.H) * K;
  const uint16_t* brow[NSUB];
#pragma unroll
  for (int s = 0; s < NSUB; ++s) {
    int n;
    if (GEMM1) n = s < NSUB / 2 ? n0 + s * 16 + r16 : g.I + n0 + (s - NSUB / 2) * 16 + r16;
    else n = n0 + s * 16 + r16;
    brow[s] = wbase + static_cast<size_t>(n) * K;
  }

  f32x4 acc[NSUB];
#pragma unroll
  for (int s = 0; s < NSUB; ++s) acc[s] = f32x4{};
  const int kper = K / 4;
  const int kbeg = wave * kper, kend = kbeg + kper;
  int k = kbeg + kg * 8;
  // main loop: UNROLL k-steps of 32 per iteration, all loads issued first
  for (; k + (UNROLL - 1) * 32 < kend; k += UNROLL * 32) {
    uint4 av[UNROLL], bv[UNROLL][NSUB];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
#pragma unroll
      for (int s = 0; s < NSUB; ++s) bv[u][s] = *reinterpret_cast<const uint4*>(brow[s] + k + u * 32);
      av[u] = *reinterpret_cast<const uint4*>(arow + k + u * 32);
    }
#pragma unroll
    for (int u = 0; u < UNROLL; ++u)
#pragma unroll
      for (int s = 0; s < NSUB; ++s) acc[s] = mfma16x16x32(as_bf16x8(av[u]), as_bf16x8(bv[u][s]), acc[s]);
  }
  for (; k < kend; k += 32) {
    const uint4 av = *reinterpret_cast<const uint4*>(arow + k);
#pragma unroll
    for (int s = 0; s < NSUB; ++s)
      acc[s] = mfma16x16x32(as_bf16x8(av), as_bf16x8(*reinterpret_cast<const uint4*>(brow[s] + k)), acc[s]);
  }

  if (wave > 0) {
#pragma unroll
    for (int s = 0; s < NSUB; ++s) red[wave - 1][s][lane] = acc[s];
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int s = 0; s < NSUB; ++s)
#pragma unroll
    for (int w = 0; w < 3; ++w) acc[s] += red[w][s][lane];

  // D element i of a 16x16 tile is (row 4*(lane/16) + i, col lane%16)
  if (GEMM1) {
#pragma unroll
    for (int s = 0; s < NSUB / 2; ++s)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = m0 + 4 * kg + i, col = n0 + s * 16 + r16;
        static_cast<uint16_t*>(g.inter)[static_cast<size_t>(row) * g.I + col] =
            f32_to_bf16(silu_mul(acc[s][i], acc[s + NSUB / 2][i]));
      }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = m0 + 4 * kg + i;
      if (g.sorted_ids[row] >= g.n_routed) continue;  // pad rows are never read
#pragma unroll
      for (int s = 0; s < NSUB; ++s)
        static_cast<float*>(g.y)[static_cast<size_t>(row) * g.H + n0 + s * 16 + r16] = acc[s][i];
    }
  }
}

// ----------------------------------------------------------------- dispatch
bool bf16_use_skinny(int T, int top_k, int E) {
  return static_cast<long>(T) * top_k <= 32L * E;  // <= 32 rows per expert on average
}

hipError_t launch_gemms_bf16(const GroupedGemm& g, hipStream_t s) {
  if (bf16_use_skinny(g.T, g.top_k, g.E)) {
    constexpr int BM = 16;
    const dim3 grid1(g.max_rows / BM, g.I / 32), grid2(g.max_rows / BM, g.H / 64);
    hipLaunchKernelGGL((gemm_bf16_skinny<4, 4, true>), grid1, dim3(256), 0, s, g);
    hipLaunchKernelGGL((gemm_bf16_skinny<4, 4, false>), grid2, dim3(256), 0, s, g);
  } else {
    constexpr int BM = 128;
    const dim3 grid1(g.max_rows / BM, g.I / 64), grid2(g.max_rows / BM, g.H / 128);
    hipLaunchKernelGGL((gemm_bf16_tiled<BM, 64, 2, 2, true>), grid1, dim3(256), 0, s, g);
    hipLaunchKernelGGL((gemm_bf16_tiled<BM, 128, 2, 2, false>), grid2, dim3(256), 0, s, g);
  }
  return hipGetLastError();
}

int gemm_block_m_bf16(int T, int top_k, int E) { return bf16_use_skinny(T, top_k, E) ? 16 : 128; }

}  // namespace moe
