// Grouped expert GEMMs for bf16 weights (the "Fused MoE" node, Fig. 1 /
// Fig. 3): per expert e, over the rows of its permuted segment,
//   GEMM1  a = SiLU(x W1[e,:I]^T) * (x W1[e,I:]^T)   (SiLU*up fused in the epilogue)
//   GEMM2  y = a W2[e]^T
// Weights are [N,K] with K contiguous, so both products read B rows along K.
//
// Two kernel families: the LDS-tiled persistent kernel shared with the other
// formats (gemm_tiled.hip) when experts hold many rows, and here
//  * skinny (decode: a few rows per expert): 16-row tile, the K range split
//    over the four waves on 128-byte line boundaries, weight fragments streamed from HBM straight into
//    registers (no reuse to stage for), v_mfma_f32_16x16x32_bf16, partial sums
//    reduced through LDS.
// Segments are padded to the row tile, so every tile belongs to one expert;
// tiles past the last segment exit at once.
#include "common.hpp"
#include "launch.hpp"
#include "lds_dma.hpp"

namespace moe {

// ----------------------------------------------------------------- skinny
// NSUB 16-column weight subtiles per workgroup (GEMM1: NSUB/2 gate + NSUB/2
// up subtiles covering the same act columns).
template <int NSUB, int UNROLL, bool GEMM1>
__global__ __launch_bounds__(256) void gemm_bf16_skinny(GroupedGemm g) {
  constexpr int BM = 16;
  constexpr int BN = GEMM1 ? NSUB / 2 * 16 : NSUB * 16;  // output columns
  __shared__ f32x4 red[3][NSUB][64];

  // column tiles vary fastest in dispatch order: the workgroups of one row
  // tile (one expert) run together, and the empty row tiles past the last
  // segment come last
  const int m0 = blockIdx.y * BM;
  if (m0 >= g.offsets[g.E]) return;
  const int e = find_segment(g.offsets, g.E, m0);
  const int n0 = blockIdx.x * BN;
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
  // K split over the four waves on 64-element (128-byte line) boundaries, so
  // no cache line is fetched by two waves: wave w takes nl/4 lines, plus one
  // of the nl%4 remainder lines for the first waves.
  const int nl = K / 64, lb = nl / 4, lr = nl % 4;
  const int kbeg = 64 * (wave * lb + min(wave, lr));
  const int kend = kbeg + 64 * (lb + (wave < lr ? 1 : 0));
  // Main loop, software pipelined: UNROLL k-steps of 32 form one stage; the
  // loads of stage i+1 are issued before the MFMAs of stage i, so every lane
  // keeps NSUB*UNROLL weight loads in flight while it computes.
  const int nst = (kend - kbeg) / (32 * UNROLL);
  int k = kbeg + kg * 8;
  u32x4 a0[UNROLL], b0[UNROLL][NSUB], a1[UNROLL], b1[UNROLL][NSUB];
#define MOE_SKINNY_LOAD(A, Bv, k_)                                                           \
  do {                                                                                       \
    _Pragma("unroll") for (int u = 0; u < UNROLL; ++u) {                                     \
      _Pragma("unroll") for (int s = 0; s < NSUB; ++s) Bv[u][s] = ld16(brow[s] + (k_) + u * 32); \
      A[u] = ld16(arow + (k_) + u * 32);                                                     \
    }                                                                                        \
  } while (0)
#define MOE_SKINNY_MMA(A, Bv)                                                                \
  do {                                                                                       \
    _Pragma("unroll") for (int u = 0; u < UNROLL; ++u)                                       \
        _Pragma("unroll") for (int s = 0; s < NSUB; ++s)                                     \
            acc[s] = mfma16x16x32(as_bf16x8(A[u]), as_bf16x8(Bv[u][s]), acc[s]);             \
  } while (0)
  if (nst > 0) MOE_SKINNY_LOAD(a0, b0, k);
  for (int i = 0; i < nst; i += 2) {
    if (i + 1 < nst) MOE_SKINNY_LOAD(a1, b1, k + 32 * UNROLL);
    MOE_SKINNY_MMA(a0, b0);
    if (i + 2 < nst) MOE_SKINNY_LOAD(a0, b0, k + 64 * UNROLL);
    if (i + 1 < nst) MOE_SKINNY_MMA(a1, b1);
    k += 64 * UNROLL;
  }
#undef MOE_SKINNY_LOAD
#undef MOE_SKINNY_MMA
  k = kbeg + kg * 8 + nst * 32 * UNROLL;
  for (; k < kend; k += 32) {
    const u32x4 av = ld16(arow + k);
#pragma unroll
    for (int s = 0; s < NSUB; ++s)
      acc[s] = mfma16x16x32(as_bf16x8(av), as_bf16x8(ld16(brow[s] + k)), acc[s]);
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

// ------------------------------------------------------ streamed (decode)
// The decode GEMMs read every weight byte once, so they are bound by how
// fast HBM delivers the weight slab.  The skinny kernel above walks 16 rows
// per load instruction (64 bytes of each, at the row stride); this one reads
// the slab the way HBM streams best: the four waves split K in quarters and
// the workgroup walks its weight rows in order, each row's quarters read
// together, with non-temporal direct-to-LDS copies of 512 bytes of one row
// per instruction (measured on the MI355X: 7.3 TB/s for this pattern,
// against 6.2 TB/s for loads that walk 16 rows at a time).  Stage (group gi,
// piece p) holds 16 rows x 512 bytes of the wave's quarter; two stages per
// wave are in flight, and two workgroups fit a CU.  The activation fragments
// of the wave's K quarter (NP pieces: K = 1024 NP) are loaded once and stay
// in registers.  Each stage row sits at a stride of 528 bytes, so the 16
// rows of a fragment read fall in distinct LDS bank groups.
// NG: 16-row weight groups per workgroup (GEMM1: NG/2 gate + NG/2 up).
template <int NG, int NP, bool GEMM1>
__global__ __launch_bounds__(256) void gemm_bf16_stream(GroupedGemm g) {
  constexpr int PC = 512;
  constexpr int ROWB = PC + 16, STAGE = 16 * ROWB;
  constexpr int JP = PC / 64;   // MFMAs (32 K elements each) per piece
  constexpr int NJ = NP * JP;   // MFMA slots over the quarter
  constexpr int NC = GEMM1 ? NG / 2 * 16 : NG * 16;
  constexpr int NST = NG * NP;  // stages per tile
  static_assert(4 * NG * 64 * 16 <= 4 * 2 * STAGE, "the reduction fits in the stage buffers");
  __shared__ __attribute__((aligned(1024))) uint8_t smem[4][2][STAGE];

  const int m0 = blockIdx.y * 16;
  if (m0 >= g.offsets[g.E]) return;
  const int e = find_segment(g.offsets, g.E, m0);
  const int n0 = blockIdx.x * NC;
  const int K = GEMM1 ? g.H : g.I;
  const int lane = lane_id(), wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  constexpr int qe = NP * PC / 2;  // this wave's K elements of each row (K = 4 qe)
  const int k0 = wave * qe;

  // A fragments: MFMA j covers K [k0 + 32 j, +32), lane group kg its
  // elements [8 kg, 8 kg + 8); the B fragments use the same K order.  All
  // of them have landed before the first weight copy is issued, so the
  // compiler's own wait counts never cover a copy.
  const uint16_t* arow;
  if (GEMM1) {
    const int sid = g.sorted_ids[m0 + r16];
    const int tok = sid < g.n_routed ? sid / g.top_k : 0;
    arow = static_cast<const uint16_t*>(g.x) + static_cast<size_t>(tok) * g.H;
  } else {
    arow = static_cast<const uint16_t*>(g.inter) + static_cast<size_t>(m0 + r16) * g.I;
  }
  arow += k0 + 8 * kg;
  u32x4 a[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) a[j] = ld16(arow + 32 * j);
  vm_wait<0>();

  const size_t rowbytes = static_cast<size_t>(K) * 2;
  const uint8_t* wq = static_cast<const uint8_t*>(GEMM1 ? g.w1 : g.w2) +
                      static_cast<size_t>(e) * (GEMM1 ? 2 * g.I : g.H) * rowbytes + 2 * static_cast<size_t>(k0) +
                      16 * lane;
  const uint32_t sbase = lds_addr(&smem[wave][0][0]);
  // stage s = gi * NP + p: rows of group gi, bytes [p*PC, (p+1)*PC) of the quarter
  auto issue = [&](int s) {
    const int gi = s / NP, p = s % NP;
    const int wr = GEMM1 ? (gi < NG / 2 ? n0 + gi * 16 : g.I + n0 + (gi - NG / 2) * 16) : n0 + gi * 16;
    const uint8_t* src = wq + static_cast<size_t>(wr) * rowbytes + p * PC;
    const uint32_t dst = sbase + (s & 1) * STAGE;
    if (16 * lane < PC) {  // 32 lanes x 16 bytes per row
#pragma unroll
      for (int i = 0; i < 16; ++i) dma16_nt(src + i * rowbytes, dst + i * ROWB);
    }
  };

  f32x4 acc[NG];
#pragma unroll
  for (int gi = 0; gi < NG; ++gi) acc[gi] = f32x4{};
  issue(0);
  if (NST > 1) issue(1);
#pragma unroll
  for (int s = 0; s < NST; ++s) {
    const int gi = s / NP, p = s % NP;
    if (s + 1 < NST) vm_wait<16>();  // stage s has landed
    else vm_wait<0>();
    const uint8_t* B = &smem[wave][s & 1][0] + r16 * ROWB + 16 * kg;
#pragma unroll
    for (int jj = 0; jj < JP; ++jj)
      acc[gi] = mfma16x16x32(as_bf16x8(a[p * JP + jj]), as_bf16x8(ld16(B + 64 * jj)), acc[gi]);
    lds_wait();  // buffer s & 1 is read out before stage s + 2 overwrites it
    if (s + 2 < NST) issue(s + 2);
  }

  // reduce the four K quarters through LDS; wave w finishes groups w, w+4, ...
  __syncthreads();
  f32x4* red = reinterpret_cast<f32x4*>(&smem[0][0][0]);  // [4 waves][NG][64 lanes]
#pragma unroll
  for (int gi = 0; gi < NG; ++gi) red[(wave * NG + gi) * 64 + lane] = acc[gi];
  __syncthreads();
  auto sum = [&](int gi) {
    f32x4 v = red[gi * 64 + lane];
#pragma unroll
    for (int w = 1; w < 4; ++w) v += red[(w * NG + gi) * 64 + lane];
    return v;
  };
  // D element i of a 16x16 tile is (row 4*(lane/16) + i, col lane%16)
  if (GEMM1) {
    for (int gi = wave; gi < NG / 2; gi += 4) {
      const f32x4 gt = sum(gi), up = sum(gi + NG / 2);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = m0 + 4 * kg + i, col = n0 + gi * 16 + r16;
        static_cast<uint16_t*>(g.inter)[static_cast<size_t>(row) * g.I + col] = f32_to_bf16(silu_mul(gt[i], up[i]));
      }
    }
  } else {
    for (int gi = wave; gi < NG; gi += 4) {
      const f32x4 v = sum(gi);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = m0 + 4 * kg + i;
        if (g.sorted_ids[row] >= g.n_routed) continue;  // pad rows are never read
        static_cast<float*>(g.y)[static_cast<size_t>(row) * g.H + n0 + gi * 16 + r16] = v[i];
      }
    }
  }
}

// ------------------------------------------------- skinny, weight-only fp8
// The decode kernel on fp8 weights with bf16 activations: the same 16-row
// tile and reduction, the K range split over the four waves in 128-wide
// blocks (the weight scale granule).  Per block a lane reads 64 contiguous
// bytes of its activation row and 32 bytes of each weight row: within the
// block, MFMA u takes K elements [32 kg + 8 u, +8) for lane group kg (one K
// permutation, applied to both operands).  The e4m3 codes decode exactly to
// bf16 (v_cvt_pk_f32_fp8); the block's partial is scaled by the block's
// fp32 scale and added to the accumulator.  The loads of block b+1 are in
// flight while block b computes.
__device__ __forceinline__ bf16x8 e4m3x8_to_bf16(uint32_t lo, uint32_t hi) {
  bf16x8 r;
  const auto f0 = __builtin_amdgcn_cvt_pk_f32_fp8(lo, false), f1 = __builtin_amdgcn_cvt_pk_f32_fp8(lo, true);
  const auto f2 = __builtin_amdgcn_cvt_pk_f32_fp8(hi, false), f3 = __builtin_amdgcn_cvt_pk_f32_fp8(hi, true);
  r[0] = static_cast<__bf16>(f0[0]); r[1] = static_cast<__bf16>(f0[1]);  // exact: e4m3 fits bf16
  r[2] = static_cast<__bf16>(f1[0]); r[3] = static_cast<__bf16>(f1[1]);
  r[4] = static_cast<__bf16>(f2[0]); r[5] = static_cast<__bf16>(f2[1]);
  r[6] = static_cast<__bf16>(f3[0]); r[7] = static_cast<__bf16>(f3[1]);
  return r;
}

template <int NSUB, bool GEMM1>
__global__ __launch_bounds__(256) void gemm_w8a16_skinny(GroupedGemm g) {
  constexpr int BM = 16;
  constexpr int BN = GEMM1 ? NSUB / 2 * 16 : NSUB * 16;
  __shared__ f32x4 red[3][NSUB][64];

  const int m0 = blockIdx.y * BM;
  if (m0 >= g.offsets[g.E]) return;
  const int e = find_segment(g.offsets, g.E, m0);
  const int n0 = blockIdx.x * BN;
  const int K = GEMM1 ? g.H : g.I;
  const int NR = GEMM1 ? 2 * g.I : g.H;  // weight rows of one expert
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
  arow += kg * 32;
  const uint8_t* wbase = static_cast<const uint8_t*>(GEMM1 ? g.w1 : g.w2) + static_cast<size_t>(e) * NR * K;
  const float* sbase = static_cast<const float*>(GEMM1 ? g.w1_scale : g.w2_scale) +
                       static_cast<size_t>(e) * (NR / 128) * (K / 128);
  const uint8_t* brow[NSUB];
  const float* srow[NSUB];  // the subtile's 16 weight rows share one 128-row scale block
#pragma unroll
  for (int s = 0; s < NSUB; ++s) {
    int nf;  // first weight row of subtile s
    if (GEMM1) nf = s < NSUB / 2 ? n0 + s * 16 : g.I + n0 + (s - NSUB / 2) * 16;
    else nf = n0 + s * 16;
    brow[s] = wbase + static_cast<size_t>(nf + r16) * K + kg * 32;
    srow[s] = sbase + static_cast<size_t>(nf / 128) * (K / 128);
  }

  f32x4 acc[NSUB];
#pragma unroll
  for (int s = 0; s < NSUB; ++s) acc[s] = f32x4{};
  const int nb = K / 128, lb = nb / 4, lr = nb % 4;
  const int bbeg = wave * lb + min(wave, lr);
  const int bend = bbeg + lb + (wave < lr ? 1 : 0);

  u32x4 a0[4], b0[NSUB][2], a1[4], b1[NSUB][2];
#define MOE_W8_LOAD(A, Bv, blk)                                                                   \
  do {                                                                                            \
    _Pragma("unroll") for (int u = 0; u < 4; ++u) A[u] = ld16(arow + (blk) * 128 + u * 8);       \
    _Pragma("unroll") for (int s = 0; s < NSUB; ++s) {                                          \
      Bv[s][0] = ld16(brow[s] + (blk) * 128);                                                    \
      Bv[s][1] = ld16(brow[s] + (blk) * 128 + 16);                                               \
    }                                                                                             \
  } while (0)
#define MOE_W8_MMA(A, Bv, blk)                                                                    \
  do {                                                                                            \
    _Pragma("unroll") for (int s = 0; s < NSUB; ++s) {                                          \
      f32x4 part = {};                                                                            \
      _Pragma("unroll") for (int u = 0; u < 4; ++u) {                                           \
        const u32x4& w = Bv[s][u >> 1];                                                           \
        const bf16x8 b = (u & 1) ? e4m3x8_to_bf16(w.z, w.w) : e4m3x8_to_bf16(w.x, w.y);          \
        part = mfma16x16x32(as_bf16x8(A[u]), b, part);                                           \
      }                                                                                           \
      acc[s] += part * srow[s][blk];                                                              \
    }                                                                                             \
  } while (0)
  int b = bbeg;
  if (b < bend) MOE_W8_LOAD(a0, b0, b);
  for (; b + 1 < bend; b += 2) {
    MOE_W8_LOAD(a1, b1, b + 1);
    MOE_W8_MMA(a0, b0, b);
    if (b + 2 < bend) MOE_W8_LOAD(a0, b0, b + 2);
    MOE_W8_MMA(a1, b1, b + 1);
  }
  if (b < bend) MOE_W8_MMA(a0, b0, b);
#undef MOE_W8_LOAD
#undef MOE_W8_MMA

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

// Decode tile knobs: weight subtiles of 16 rows per workgroup and k-steps of
// 32 loaded ahead per lane (NSUB * UNROLL 16-byte loads in flight per lane).
#ifndef MOE_SKINNY1_NSUB
#define MOE_SKINNY1_NSUB 4
#endif
#ifndef MOE_SKINNY1_UNROLL
#define MOE_SKINNY1_UNROLL 2
#endif
#ifndef MOE_SKINNY2_NSUB
#define MOE_SKINNY2_NSUB 4
#endif
#ifndef MOE_SKINNY2_UNROLL
#define MOE_SKINNY2_UNROLL 2
#endif

// Streamed decode kernel: 16-row weight groups per workgroup.
#ifndef MOE_STREAM_NG1
#define MOE_STREAM_NG1 4
#endif
#ifndef MOE_STREAM_NG2
#define MOE_STREAM_NG2 4
#endif
#ifndef MOE_STREAM
#define MOE_STREAM 1
#endif

template <int NG, bool GEMM1>
hipError_t launch_stream(const GroupedGemm& g, hipStream_t s) {
  constexpr int NC = GEMM1 ? NG / 2 * 16 : NG * 16;
  const dim3 grid((GEMM1 ? g.I : g.H) / NC, g.max_rows / 16);
  switch ((GEMM1 ? g.H : g.I) / 1024) {
    case 1: hipLaunchKernelGGL((gemm_bf16_stream<NG, 1, GEMM1>), grid, dim3(256), 0, s, g); break;
    case 2: hipLaunchKernelGGL((gemm_bf16_stream<NG, 2, GEMM1>), grid, dim3(256), 0, s, g); break;
    case 3: hipLaunchKernelGGL((gemm_bf16_stream<NG, 3, GEMM1>), grid, dim3(256), 0, s, g); break;
    default: hipLaunchKernelGGL((gemm_bf16_stream<NG, 4, GEMM1>), grid, dim3(256), 0, s, g); break;
  }
  return hipGetLastError();
}
// K = 1024 * NP, NP <= 4 (each wave's quarter of a row is whole 512-byte
// pieces); other decode shapes take the skinny kernel
bool stream_fits(int K, int N, int nc) { return MOE_STREAM && K % 1024 == 0 && K <= 4096 && N % nc == 0; }

hipError_t launch_gemm1_bf16(const GroupedGemm& g, hipStream_t s) {
  if (bf16_use_skinny(g.T, g.top_k, g.E) && stream_fits(g.H, g.I, MOE_STREAM_NG1 / 2 * 16))
    return launch_stream<MOE_STREAM_NG1, true>(g, s);
  if (bf16_use_skinny(g.T, g.top_k, g.E)) {
    constexpr int NS = MOE_SKINNY1_NSUB;
    const dim3 grid(g.I / (NS / 2 * 16), g.max_rows / 16);
    hipLaunchKernelGGL((gemm_bf16_skinny<NS, MOE_SKINNY1_UNROLL, true>), grid, dim3(256), 0, s, g);
    return hipGetLastError();
  }
  return launch_gemm1_bf16_tiled(g, s);
}

hipError_t launch_gemm2_bf16(const GroupedGemm& g, hipStream_t s) {
  if (bf16_use_skinny(g.T, g.top_k, g.E) && stream_fits(g.I, g.H, MOE_STREAM_NG2 * 16))
    return launch_stream<MOE_STREAM_NG2, false>(g, s);
  if (bf16_use_skinny(g.T, g.top_k, g.E)) {
    constexpr int NS = MOE_SKINNY2_NSUB;
    const dim3 grid(g.H / (NS * 16), g.max_rows / 16);
    hipLaunchKernelGGL((gemm_bf16_skinny<NS, MOE_SKINNY2_UNROLL, false>), grid, dim3(256), 0, s, g);
    return hipGetLastError();
  }
  return launch_gemm2_bf16_tiled(g, s);
}

// Weight-only fp8 (decode route; the host guarantees T*k <= 32*E).
#ifndef MOE_W8_NSUB
#define MOE_W8_NSUB 4
#endif
hipError_t launch_gemm1_w8a16(const GroupedGemm& g, hipStream_t s) {
  constexpr int NS = MOE_W8_NSUB;
  const dim3 grid(g.I / (NS / 2 * 16), g.max_rows / 16);
  hipLaunchKernelGGL((gemm_w8a16_skinny<NS, true>), grid, dim3(256), 0, s, g);
  return hipGetLastError();
}
hipError_t launch_gemm2_w8a16(const GroupedGemm& g, hipStream_t s) {
  constexpr int NS = MOE_W8_NSUB;
  const dim3 grid(g.H / (NS * 16), g.max_rows / 16);
  hipLaunchKernelGGL((gemm_w8a16_skinny<NS, false>), grid, dim3(256), 0, s, g);
  return hipGetLastError();
}

int gemm_block_m_bf16(int T, int top_k, int E) {
  return bf16_use_skinny(T, top_k, E) ? 16 : bf16_tiled_block_m();
}

}  // namespace moe
