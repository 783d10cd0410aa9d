// Grouped expert GEMMs, LDS-tiled, for the three weight formats (the "Fused
// MoE" node of the paper's skeleton, Fig. 1 / Fig. 3; the quantised formats
// carry the numeric semantics Sec. 6.2 asks of quantised routes):
//   GEMM1  a = SiLU(x W1[e,:I]^T) * (x W1[e,I:]^T)     (SiLU*up epilogue)
//   GEMM2  y = a W2[e]^T
//
//  bf16  A, B bf16; v_mfma_f32_32x32x16_bf16.
//  fp8   A (activations) and B (weights) OCP e4m3; v_mfma_f32_32x32x64_f8f6f4
//        over one 128-wide K block at a time into a fresh partial, then
//        acc += partial * s_row(A) * s_block(B) on the VALU.  The GEMM1
//        epilogue requantises the intermediate per (row, 128 columns): the
//        tile holds exactly one such group per row.
//  int4  A bf16; B signed int4 words decoded in registers (q * bf16 scale,
//        rounded to bf16) right before the bf16 MFMA, never materialised.
//
// Every format streams 128 bytes of each A row per K step through LDS (64
// bf16 / 128 fp8 elements), 16-byte chunks XOR-swizzled by row so that the
// fragment reads are bank-conflict free; B rows likewise (int4: 32 bytes).
//
// Scheduling is persistent and XCD-aware: the launch has a few workgroups per
// CU; workgroups that land on one XCD (block ids congruent mod 8) own one
// contiguous range of logical tiles, ordered in groups of GM row tiles x all
// column tiles, so the row tiles (gathered hidden rows) and weight slabs a
// group shares are served from that XCD's L2.  The number of real row tiles
// is read on the device from expert_offsets[E] (segments are padded to BM).
#include <algorithm>

#include "common.hpp"
#include "launch.hpp"

namespace moe {

constexpr int kXcds = 8;

template <int FMT>
struct FmtTraits;
template <>
struct FmtTraits<0> {  // bf16
  static constexpr int KE = 64, BB = 128;
};
template <>
struct FmtTraits<1> {  // fp8
  static constexpr int KE = 128, BB = 128;
};
template <>
struct FmtTraits<2> {  // int4 weights, bf16 activations
  static constexpr int KE = 64, BB = 32;
};

// 8 signed nibbles -> 8 bf16 values q * s (s an fp32 copy of a bf16 scale).
__device__ __forceinline__ bf16x8 dequant_int4x8(uint32_t w, float s) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int q = static_cast<int>(w << (28 - 4 * i)) >> 28;
    r[i] = static_cast<__bf16>(static_cast<float>(q) * s);
  }
  return r;
}

template <int FMT, bool GEMM1, int BM, int BNW, int WM, int WN, int GM>
__global__ __launch_bounds__(256) void moe_gemm_tiled(GroupedGemm g) {
  static_assert(WM * WN == 4, "four waves");
  constexpr int KE = FmtTraits<FMT>::KE;  // K elements per step
  constexpr int KB = 128;                 // A bytes per row per step
  constexpr int BB = FmtTraits<FMT>::BB;  // B bytes per row per step
  constexpr int WTM = BM / WM, WTN = BNW / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int NC = GEMM1 ? BNW / 2 : BNW;  // output columns per tile
  constexpr int A_CH = BM * KB / 16 / 256, B_CH = BNW * BB / 16 / 256;
  static_assert(A_CH >= 1 && B_CH >= 1 && A_CH * 4096 == BM * KB && B_CH * 4096 == BNW * BB, "");
  static_assert(!GEMM1 || TN % 2 == 0, "gate/up pairs");
  static_assert(FMT != 1 || !GEMM1 || NC == 128, "fp8 requant needs one 128-column group per tile");

  __shared__ __attribute__((aligned(16))) uint8_t lds_a[2][BM * KB];
  __shared__ __attribute__((aligned(16))) uint8_t lds_b[2][BNW * BB];
  __shared__ __attribute__((aligned(16))) float lds_sa[FMT == 1 ? 2 : 1][FMT == 1 ? BM : 1];
  __shared__ float lds_amax[FMT == 1 && GEMM1 ? WN : 1][FMT == 1 && GEMM1 ? BM : 1];

  const int tid = threadIdx.x, lane = lane_id(), wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int l32 = lane & 31, kg = lane >> 5;
  const int K = GEMM1 ? g.H : g.I;
  const int N = GEMM1 ? g.I : g.H;       // output columns of the product
  const int nk = K / KE;
  const int n_tiles_n = N / NC;
  const int n_tiles_m = g.offsets[g.E] / BM;
  const int total = n_tiles_m * n_tiles_n;

  // this workgroup's share of the logical tiles: a contiguous range per XCD
  const int xcd = blockIdx.x % kXcds, slot = blockIdx.x / kXcds;
  const int per_xcd = gridDim.x / kXcds;
  const int chunk = (total + kXcds - 1) / kXcds;
  const int t_end = min(total, (xcd + 1) * chunk);

  for (int t = xcd * chunk + slot; t < t_end; t += per_xcd) {
    const int grp = t / (GM * n_tiles_n), in = t % (GM * n_tiles_n);
    const int m_first = grp * GM, gm = min(GM, n_tiles_m - m_first);
    const int mt = m_first + in % gm, nt = in / gm;
    const int m0 = mt * BM, n0 = nt * NC;
    const int e = find_segment(g.offsets, g.E, m0);

    // ---- global source rows of this thread's chunks
    const uint8_t* a_src[A_CH];
    int a_dst[A_CH];
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
      const int q = tid + i * 256, r = q >> 3, c = q & 7;
      const uint8_t* row;
      if (GEMM1) {
        const int sid = g.sorted_ids[m0 + r];
        const int tok = sid < g.n_routed ? sid / g.top_k : 0;
        row = static_cast<const uint8_t*>(g.x) + static_cast<size_t>(tok) * g.H * (FMT == 1 ? 1 : 2);
      } else {
        row = static_cast<const uint8_t*>(g.inter) + static_cast<size_t>(m0 + r) * g.I * (FMT == 1 ? 1 : 2);
      }
      a_src[i] = row + c * 16;
      a_dst[i] = r * KB + ((c ^ (r & 7)) << 4);
    }
    const size_t w_row_bytes = FMT == 0 ? K * 2 : (FMT == 1 ? K : K / 2);
    const uint8_t* wbase = static_cast<const uint8_t*>(GEMM1 ? g.w1 : g.w2) +
                           static_cast<size_t>(e) * (GEMM1 ? 2 * g.I : g.H) * w_row_bytes;
    const uint8_t* b_src[B_CH];
    int b_dst[B_CH];
#pragma unroll
    for (int i = 0; i < B_CH; ++i) {
      const int q = tid + i * 256;
      const int r = FMT == 2 ? q >> 1 : q >> 3, c = FMT == 2 ? q & 1 : q & 7;
      int n;
      if (GEMM1) n = r < NC ? n0 + r : g.I + n0 + (r - NC);
      else n = n0 + r;
      b_src[i] = wbase + static_cast<size_t>(n) * w_row_bytes + c * 16;
      b_dst[i] = FMT == 2 ? r * BB + ((c ^ ((r >> 2) & 1)) << 4) : r * BB + ((c ^ (r & 7)) << 4);
    }
    // fp8 activation scales: thread r < BM owns row r's per-K-block scale
    const float* sa_src = nullptr;
    if (FMT == 1 && tid < BM) {
      if (GEMM1) {
        const int sid = g.sorted_ids[m0 + tid];
        const int tok = sid < g.n_routed ? sid / g.top_k : 0;
        sa_src = g.x_scale + static_cast<size_t>(tok) * (g.H / 128);
      } else {
        sa_src = g.inter_scale + static_cast<size_t>(m0 + tid) * (g.I / 128);
      }
    }

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = f32x16{};

    u32x4 ra[A_CH], rb[B_CH];
    float rsa = 0.f;
#define MOE_TILE_LOAD(kt_)                                                                    \
  do {                                                                                        \
    _Pragma("unroll") for (int i = 0; i < A_CH; ++i) ra[i] =                                  \
        ld16(a_src[i] + (kt_) * KB);                               \
    _Pragma("unroll") for (int i = 0; i < B_CH; ++i) rb[i] =                                  \
        ld16(b_src[i] + (kt_) * BB);                               \
    if constexpr (FMT == 1) {                                                                 \
      if (sa_src) rsa = sa_src[kt_];                                                          \
    }                                                                                         \
  } while (0)
#define MOE_TILE_STORE(buf_)                                                                  \
  do {                                                                                        \
    _Pragma("unroll") for (int i = 0; i < A_CH; ++i)                                          \
        st16(&lds_a[buf_][a_dst[i]], ra[i]);                            \
    _Pragma("unroll") for (int i = 0; i < B_CH; ++i)                                          \
        st16(&lds_b[buf_][b_dst[i]], rb[i]);                            \
    if constexpr (FMT == 1) {                                                                 \
      if (tid < BM) lds_sa[buf_][tid] = rsa;                                                  \
    }                                                                                         \
  } while (0)

    // B row (within the tile) of wave tile j
#define brow(j) (GEMM1 ? ((j) < TN / 2 ? wn * (WTN / 2) + (j) * 32 : NC + wn * (WTN / 2) + ((j) - TN / 2) * 32) \
                       : wn * WTN + (j) * 32)

    MOE_TILE_LOAD(0);
    MOE_TILE_STORE(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const int buf = kt & 1;
      if (kt + 1 < nk) MOE_TILE_LOAD(kt + 1);
      const uint8_t* As = lds_a[buf];
      const uint8_t* Bs = lds_b[buf];
      if constexpr (FMT == 0) {
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const int ch = 2 * kk + kg;
          bf16x8 a[TM], b[TN];
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            const int r = wm * WTM + i * 32 + l32;
            a[i] = as_bf16x8(ld16(As + r * KB + ((ch ^ (r & 7)) << 4)));
          }
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int r = brow(j) + l32;
            b[j] = as_bf16x8(ld16(Bs + r * BB + ((ch ^ (r & 7)) << 4)));
          }
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = mfma32x32x16(a[i], b[j], acc[i][j]);
        }
      } else if constexpr (FMT == 1) {
        f32x16 part[TM][TN];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          const int c0 = 4 * kk + 2 * kg;
          i32x8 a[TM], b[TN];
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            const int r = wm * WTM + i * 32 + l32;
            const u32x4 lo = ld16(As + r * KB + ((c0 ^ (r & 7)) << 4));
            const u32x4 hi = ld16(As + r * KB + (((c0 + 1) ^ (r & 7)) << 4));
            a[i] = i32x8{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
          }
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int r = brow(j) + l32;
            const u32x4 lo = ld16(Bs + r * BB + ((c0 ^ (r & 7)) << 4));
            const u32x4 hi = ld16(Bs + r * BB + (((c0 + 1) ^ (r & 7)) << 4));
            b[j] = i32x8{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
          }
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
              part[i][j] = mfma32x32x64_fp8(a[i], b[j], kk == 0 ? f32x16{} : part[i][j]);
        }
        // acc += part * s_row * s_block(B) for this K block
        const float* wsc = static_cast<const float*>(GEMM1 ? g.w1_scale : g.w2_scale) +
                           static_cast<size_t>(e) * ((GEMM1 ? 2 * g.I : g.H) / 128) * (K / 128);
        float sb[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int r = brow(j);
          const int n_glob = GEMM1 ? (r < NC ? n0 + r : g.I + n0 + (r - NC)) : n0 + r;
          sb[j] = wsc[static_cast<size_t>(n_glob / 128) * (K / 128) + kt];
        }
#pragma unroll
        for (int i = 0; i < TM; ++i) {
#pragma unroll
          for (int v4 = 0; v4 < 4; ++v4) {
            const float4 sr = *reinterpret_cast<const float4*>(&lds_sa[buf][wm * WTM + i * 32 + 8 * v4 + 4 * kg]);
            const float s4[4] = {sr.x, sr.y, sr.z, sr.w};
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
              for (int u = 0; u < 4; ++u)
                acc[i][j][4 * v4 + u] = fmaf(part[i][j][4 * v4 + u], s4[u] * sb[j], acc[i][j][4 * v4 + u]);
          }
        }
      } else {  // int4
        // this lane's B words for the four 16-wide K substeps, and its scales
        const uint16_t* wsc = static_cast<const uint16_t*>(GEMM1 ? g.w1_scale : g.w2_scale) +
                              static_cast<size_t>(e) * (GEMM1 ? 2 * g.I : g.H) * (K / 128);
        u32x4 bw[TN];
        float sb[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int r = brow(j) + l32;
          bw[j] = ld16(Bs + r * BB + ((kg ^ ((r >> 2) & 1)) << 4));
          const int n_glob = GEMM1 ? (r < NC ? n0 + r : g.I + n0 + (r - NC)) : n0 + r;
          sb[j] = bf16_to_f32(wsc[static_cast<size_t>(n_glob) * (K / 128) + (kt * KE) / 128]);
        }
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          // substep kk of lane group kg covers K elements [(4kg+kk)*8, +8) of the step
          const int ch = 4 * kg + kk;
          bf16x8 a[TM], b[TN];
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            const int r = wm * WTM + i * 32 + l32;
            a[i] = as_bf16x8(ld16(As + r * KB + ((ch ^ (r & 7)) << 4)));
          }
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const uint32_t wd = kk == 0 ? bw[j].x : (kk == 1 ? bw[j].y : (kk == 2 ? bw[j].z : bw[j].w));
            b[j] = dequant_int4x8(wd, sb[j]);
          }
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = mfma32x32x16(a[i], b[j], acc[i][j]);
        }
      }
      if (kt + 1 < nk) MOE_TILE_STORE(buf ^ 1);
      __syncthreads();
    }
#undef MOE_TILE_LOAD
#undef MOE_TILE_STORE
#undef brow

    // ---- epilogue.  D element v of a 32x32 tile: row 8*(v/4) + 4*kg + v%4, column l32.
    if constexpr (GEMM1) {
      constexpr int TH = TN / 2;  // gate tiles (paired with up tile j + TH)
      float av[TM][TH][16];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TH; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) av[i][j][v] = silu_mul(acc[i][j][v], acc[i][j + TH][v]);
      if constexpr (FMT == 1) {
        // per-row amax over the tile's 128 columns: lanes, then waves (LDS)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            float m = 0.f;
#pragma unroll
            for (int j = 0; j < TH; ++j) m = fmaxf(m, fabsf(av[i][j][v]));
#pragma unroll
            for (int off = 1; off < 32; off <<= 1) m = fmaxf(m, __shfl_xor(m, off));
            if (l32 == 0) lds_amax[wn][wm * WTM + i * 32 + 8 * (v >> 2) + 4 * kg + (v & 3)] = m;
          }
        __syncthreads();
        uint8_t* q = static_cast<uint8_t*>(g.inter);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int rl = wm * WTM + i * 32 + 8 * (v >> 2) + 4 * kg + (v & 3);
            float m = 0.f;
#pragma unroll
            for (int w = 0; w < WN; ++w) m = fmaxf(m, lds_amax[w][rl]);
            const float s = fmaxf(m, 1e-10f) / 448.0f;
            const int row = m0 + rl;
#pragma unroll
            for (int j = 0; j < TH; ++j) {
              const int col = n0 + wn * (WTN / 2) + j * 32 + l32;
              q[static_cast<size_t>(row) * g.I + col] =
                  static_cast<uint8_t>(f32x2_to_e4m3(sat_e4m3(av[i][j][v] / s), 0.f) & 0xFF);
            }
            if (wn == 0 && l32 == 0) g.inter_scale[static_cast<size_t>(row) * (g.I / 128) + n0 / 128] = s;
          }
        __syncthreads();  // lds_amax is reused by the next tile
      } else {
        uint16_t* o = static_cast<uint16_t*>(g.inter);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TH; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
              const int row = m0 + wm * WTM + i * 32 + 8 * (v >> 2) + 4 * kg + (v & 3);
              const int col = n0 + wn * (WTN / 2) + j * 32 + l32;
              o[static_cast<size_t>(row) * g.I + col] = f32_to_bf16(av[i][j][v]);
            }
      }
    } else {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int row = m0 + wm * WTM + i * 32 + 8 * (v >> 2) + 4 * kg + (v & 3);
          if (g.sorted_ids[row] >= g.n_routed) continue;  // pad rows are never read
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int col = n0 + wn * WTN + j * 32 + l32;
            if (y_is_f32(FMT))
              static_cast<float*>(g.y)[static_cast<size_t>(row) * g.H + col] = acc[i][j][v];
            else
              static_cast<uint16_t*>(g.y)[static_cast<size_t>(row) * g.H + col] = f32_to_bf16(acc[i][j][v]);
          }
        }
    }
  }
}

// ----------------------------------------------------------------- launchers
namespace {

int cu_count() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    n = 256;
  return n;
}

// Persistent grid: as many workgroups as fit on the device at once (a
// multiple of the XCD count), never more than the largest possible number of
// tiles.
template <class Kernel>
dim3 persistent_grid(Kernel k, long max_tiles) {
  int per_cu = 1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, 256, 0) != hipSuccess || per_cu < 1)
    per_cu = 1;
  long n = static_cast<long>(cu_count()) * per_cu;
  n = (n + kXcds - 1) / kXcds * kXcds;
  const long cap = (max_tiles + kXcds - 1) / kXcds * kXcds;
  return dim3(static_cast<unsigned>(std::max<long>(kXcds, std::min(n, cap))));
}

template <int FMT, bool GEMM1, int BM, int BNW, int WM, int WN, int GM>
hipError_t launch_tiled(const GroupedGemm& g, hipStream_t s) {
  constexpr int NC = GEMM1 ? BNW / 2 : BNW;
  const long mt = g.max_rows / BM, nt = (GEMM1 ? g.I : g.H) / NC;
  auto kern = moe_gemm_tiled<FMT, GEMM1, BM, BNW, WM, WN, GM>;
  hipLaunchKernelGGL(kern, persistent_grid(kern, mt * nt), dim3(256), 0, s, g);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm1_bf16_tiled(const GroupedGemm& g, hipStream_t s) {
  return launch_tiled<0, true, 128, 256, 2, 2, 4>(g, s);
}
hipError_t launch_gemm2_bf16_tiled(const GroupedGemm& g, hipStream_t s) {
  if (g.H % 256) return launch_tiled<0, false, 128, 128, 2, 2, 4>(g, s);
  return launch_tiled<0, false, 128, 256, 2, 2, 4>(g, s);
}

int gemm_block_m_fp8(int, int, int) { return 128; }
hipError_t launch_gemm1_fp8(const GroupedGemm& g, hipStream_t s) {
  return launch_tiled<1, true, 128, 256, 2, 2, 4>(g, s);
}
hipError_t launch_gemm2_fp8(const GroupedGemm& g, hipStream_t s) {
  if (g.H % 256) return launch_tiled<1, false, 128, 128, 2, 2, 4>(g, s);
  return launch_tiled<1, false, 128, 256, 2, 2, 4>(g, s);
}

int gemm_block_m_int4(int, int, int) { return 64; }
hipError_t launch_gemm1_int4(const GroupedGemm& g, hipStream_t s) {
  return launch_tiled<2, true, 64, 256, 1, 4, 4>(g, s);
}
hipError_t launch_gemm2_int4(const GroupedGemm& g, hipStream_t s) {
  if (g.H % 256) return launch_tiled<2, false, 64, 128, 1, 4, 4>(g, s);
  return launch_tiled<2, false, 64, 256, 1, 4, 4>(g, s);
}

}  // namespace moe
