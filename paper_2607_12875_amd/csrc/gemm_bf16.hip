// Grouped expert GEMMs with bf16 activations at decode sizes (the "Fused
// MoE" node, Fig. 1 / Fig. 3): per expert e, over the rows of its permuted
// segment,
//   GEMM1  a = SiLU(x W1[e,:I]^T) * (x W1[e,I:]^T)   (SiLU*up fused in the epilogue)
//   GEMM2  y = a W2[e]^T
// Weights are [N,K] with K contiguous, so both products read B rows along K.
//
// When experts hold many rows the LDS-tiled persistent kernel of
// gemm_tiled.hip runs; here are the 16-row kernels for a few rows per expert
// (no reuse to stage for), all on v_mfma_f32_16x16x32_bf16 with the weights
// decoded to bf16 in registers and partial sums reduced through LDS:
//  * streamed (gemm_bf16_stream): the weight slab copied straight into LDS
//    row by row in long pieces, for bf16, int4, weight-only fp8 and MXFP4
//    weights;
//  * skinny (gemm_bf16_skinny, gemm_w8a16_skinny, gemm_w4a16_skinny): the K
//    range split over the four waves, weight fragments loaded straight into
//    registers, for the K sizes the streamed kernel does not take.
// Segments are padded to the row tile, so every tile belongs to one expert;
// tiles past the last segment exit at once.
#include <algorithm>

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

// Two words of 8 signed nibbles each (element k of a word in bits
// [4k, 4k+4)) -> 2 x 8 bf16 values 136 + q, exact: bits 0x4300 | (q + 8),
// i.e. 128 + (q + 8) with the nibble in the low mantissa bits of 128, and
// q + 8 = n ^ 8 for the two's-complement nibble n.  In the order two
// operations per dword give: dword d takes nibbles d and d + 4 (bf16 slots
// 2d, 2d + 1), so slot s holds element {0,4,1,5,2,6,3,7}[s] of the word.
// Each half is (n & 0xF) ^ 0x4308, one v_bitop3 (truth table of
// (S0 & S1) ^ S2 over (0xF0, 0xCC, 0xAA): 0x6A) on the word shifted right by
// 4 d.  The shifted copies of both words come from 64-bit shifts of the pair
// (one v_lshrrev_b64 in place of two 32-bit shifts; the bits of w1 that move
// into the top of w0's copy are never selected), written as asm because the
// compiler splits a 64-bit shift into v_alignbit_b32 + v_lshrrev_b32.
__device__ __forceinline__ void int4x16_biased_bf16_strided(uint32_t w0, uint32_t w1, bf16x8& d0, bf16x8& d1) {
  const uint64_t pr = static_cast<uint64_t>(w1) << 32 | w0;
  uint64_t s4, s8, s12;
  asm("v_lshrrev_b64 %0, 4, %1" : "=v"(s4) : "v"(pr));
  asm("v_lshrrev_b64 %0, 8, %1" : "=v"(s8) : "v"(pr));
  asm("v_lshrrev_b64 %0, 12, %1" : "=v"(s12) : "v"(pr));
  auto dw = [](uint32_t v) { return static_cast<uint32_t>(__builtin_amdgcn_bitop3_b32(v, 0x000F000Fu, 0x43084308u, 0x6A)); };
  auto lo = [](uint64_t v) { return static_cast<uint32_t>(v); };
  auto hi = [](uint64_t v) { return static_cast<uint32_t>(v >> 32); };
  d0 = as_bf16x8(u32x4{dw(w0), dw(lo(s4)), dw(lo(s8)), dw(lo(s12))});
  d1 = as_bf16x8(u32x4{dw(w1), dw(hi(s4)), dw(hi(s8)), dw(hi(s12))});
}

// ------------------------------------------------------ streamed (decode)
#ifndef MOE_STREAM_NS
#define MOE_STREAM_NS 4
#endif
#ifndef MOE_STREAM_OCC
#define MOE_STREAM_OCC 1  // workgroups per CU the stage buffers are sized for
#endif
#ifndef MOE_STREAM_F4_HALF
#define MOE_STREAM_F4_HALF 1
#endif
// The decode GEMMs read every weight byte once, so they are bound by how
// fast HBM delivers the weight slab.  The skinny kernel above walks 16 rows
// per load instruction (64 bytes of each, at the row stride); this one reads
// the slab the way HBM streams best: the four waves split K in quarters and
// the workgroup walks its weight rows in order, each row's quarters read
// together, with non-temporal direct-to-LDS copies of one piece (up to 1 KB)
// of one row per instruction (measured on the MI355X: 7.1-7.3 TB/s for this
// pattern, against 6.2 TB/s for loads that walk 16 rows at a time).
//
// Persistent: one workgroup per CU takes an equal share of the (row tile,
// column block) units, in row-tile order, read from expert_offsets on the
// device.  A run of units of one row tile shares the activation fragments
// of the wave's K quarter (loaded once into registers), and the copy
// pipeline runs on across its blocks (NS stages of 16 rows x one piece per
// wave), so start-up costs are paid once per run and the per-block epilogue
// (cross-wave reduction through LDS, SiLU*up or the y store) overlaps the
// copies in flight.  A stage row sits at a stride of PC + 16 bytes, so the
// 16 rows of a fragment read fall in distinct LDS bank groups.
//
// FMT 0: bf16 weights.  FMT 3: e4m3 weights with fp32 scales per 128x128
// block (the weight-only fp8 route): each stage also copies its group's
// block scales for the piece (one 4-byte copy per 128-wide K block) next to
// the weights; inside a 128-wide block lane group kg takes bytes
// [32 kg, 32 kg + 32), the four MFMAs of the block decode them exactly to
// bf16 (the activation fragments use the same K order), and the block's
// partial is scaled into the accumulator.  FMT 2: int4 weights (eight
// signed nibbles per word along K) with a bf16 scale per row and 128-wide K
// group: the stage also copies each of its 16 rows' group scales for the
// piece (whole dwords), the codes enter the MFMA exactly as bf16 136 + q (the
// activation fragments permuted once per run to the decode's element
// order), each group's partial starts from the row's -136 * (sum of its
// activations over the group), formed once per run by the MFMA itself, and
// the lane's weight row scale multiplies it into the accumulator.
// NG: 16-row weight groups per block (GEMM1: NG/2 gate + NG/2 up); NP
// pieces of JP MFMAs (32 K elements each) per row and wave: K = NWV * 32 * NP * JP.

template <int FMT, int NWV, int NG, int NP, int JP, bool GEMM1>
__global__ __launch_bounds__(64 * NWV) void gemm_bf16_stream(GroupedGemm g) {
  constexpr bool F8 = FMT == 3, F4 = FMT == 4, I4 = FMT == 2;
  constexpr bool BLK = F8 || F4 || I4;              // K taken in 128-wide blocks
  constexpr int B32 = F8 ? 32 : ((F4 || I4) ? 16 : 64);  // weight bytes per 32 elements
  constexpr int PC = B32 * JP, ROWB = PC + 16;      // piece bytes, LDS row stride
  constexpr int NSI = F4 ? (JP + 15) / 16 : ((F8 || I4) ? 1 : 0);  // scale copy instructions per stage
  constexpr int STAGE = 16 * ROWB + (F8 ? 64 : 0) + (F4 ? ((16 * JP + 15) / 16) * 16 : 0) + (I4 ? 8 * JP : 0);
  constexpr int CPS = 16 + NSI;                     // copy instructions per stage
  static_assert(!BLK || JP % 4 == 0, "pieces are whole 128-wide blocks");
  static_assert(!I4 || (JP % 8 == 0 && JP <= 32), "int4: a row's group scales of a piece are whole dwords, one copy");
  // stage buffers per wave: as many as LDS holds beside the reduction, up to MOE_STREAM_NS
  constexpr int RED = (NWV - 1) * NG * 1024;  // bytes of the reduction buffer
  constexpr int NSO = (160 * 1024 / MOE_STREAM_OCC - RED) / (NWV * STAGE);
  constexpr int NSF = NSO >= 2 ? NSO : (160 * 1024 - RED) / (NWV * STAGE);
  constexpr int NS = NSF < MOE_STREAM_NS ? NSF : MOE_STREAM_NS;
  static_assert(NS >= 2, "two stage buffers per wave");
  constexpr int NJ = NP * JP;   // MFMAs over the quarter
  constexpr int NC = GEMM1 ? NG / 2 * 16 : NG * 16;
  constexpr int NST = NG * NP;  // stages per column block
  static_assert(PC <= 1024 && (PC / 16) % 2 == 0, "row stride an odd number of 16-byte slots");
  static_assert(STAGE % 16 == 0, "16-byte aligned stages");
  __shared__ __attribute__((aligned(1024))) uint8_t smem[NWV][NS][STAGE];
  __shared__ f32x4 red[NWV - 1][NG][64];  // partials of waves 1.. for wave 0

  const int N = GEMM1 ? g.I : g.H, K = GEMM1 ? g.H : g.I;
  const int nb = N / NC;                                           // column blocks per row tile
  const long units = static_cast<long>(g.offsets[g.E] / 16) * nb;  // (row tile, block) pairs
  const long u_end = units * (blockIdx.x + 1) / gridDim.x;
  const int lane = lane_id(), wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  constexpr int qe = NJ * 32;  // this wave's K elements of each row
  const int k0 = wave * qe;
  const size_t rowbytes = static_cast<size_t>(K) / 32 * B32;
  const uint32_t sbase = lds_addr(&smem[wave][0][0]);

  for (long u = units * blockIdx.x / gridDim.x; u < u_end;) {
    // one run: row tile rt, column blocks [cb0, cb1)
    const int rt = static_cast<int>(u / nb), cb0 = static_cast<int>(u % nb);
    const int cb1 = static_cast<int>(min(static_cast<long>(nb), cb0 + (u_end - u)));
    u += cb1 - cb0;
    const int m0 = rt * 16;
    const int e = find_segment(g.offsets, g.E, m0);

    // A fragments: MFMA j covers K [k0 + 32 j, +32), lane group kg its
    // elements [8 kg, 8 kg + 8) (the 128-wide block formats: MFMA 4 b + u
    // covers block b, lane group kg its elements [32 kg + 8 u, +8)); the B
    // fragments use the same K order.
    // They (and the pad flags of the rows this lane stores) have landed
    // before the run's first weight copy is issued, and the previous run
    // ended with every copy landed, so the compiler's own wait counts never
    // cover a copy.
    const uint16_t* arow;
    if (GEMM1) {
      const int sid = g.sorted_ids[m0 + r16];
      const int tok = sid < g.n_routed ? sid / g.top_k : 0;
      arow = static_cast<const uint16_t*>(g.x) + static_cast<size_t>(tok) * g.H;
    } else {
      arow = static_cast<const uint16_t*>(g.inter) + static_cast<size_t>(m0 + r16) * g.I;
    }
    arow += k0;
    u32x4 a[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      a[j] = ld16(arow + (BLK ? 128 * (j / 4) + 32 * kg + 8 * (j % 4) : 32 * j + 8 * kg));
    bool live[4];  // GEMM2: rows m0 + 4 kg + i that are routed rows (pads are never read)
#pragma unroll
    for (int i = 0; i < 4; ++i) live[i] = GEMM1 || g.sorted_ids[m0 + 4 * kg + i] < g.n_routed;
    vm_wait<0>();
    // int4: each fragment's elements put in the order the weight decode
    // gives (int4x16_biased_bf16_strided), and nbias[b] = -136 * (each row's
    // sum over the quarter's 128-group b), the start of that group's partial
    f32x4 nbias[I4 ? NJ / 4 : 1];
    if constexpr (I4) {
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const u32x4 v = a[j];
        a[j] = u32x4{__builtin_amdgcn_perm(v.z, v.x, 0x05040100u), __builtin_amdgcn_perm(v.z, v.x, 0x07060302u),
                     __builtin_amdgcn_perm(v.w, v.y, 0x05040100u), __builtin_amdgcn_perm(v.w, v.y, 0x07060302u)};
      }
      const u32x4 c = {0xC308C308u, 0xC308C308u, 0xC308C308u, 0xC308C308u};  // bf16 -136
#pragma unroll
      for (int b = 0; b < NJ / 4; ++b) {
        nbias[b] = f32x4{};
#pragma unroll
        for (int u = 0; u < 4; ++u) nbias[b] = mfma16x16x32(as_bf16x8(a[4 * b + u]), as_bf16x8(c), nbias[b]);
      }
    }

    const int NR = GEMM1 ? 2 * g.I : g.H;  // weight rows per expert
    const uint8_t* wq = static_cast<const uint8_t*>(GEMM1 ? g.w1 : g.w2) + static_cast<size_t>(e) * NR * rowbytes +
                        static_cast<size_t>(k0) / 32 * B32 + 16 * lane;
    // fp8: scale row of the 128-row block, at this wave's first K block
    const float* wsc = F8 ? static_cast<const float*>(GEMM1 ? g.w1_scale : g.w2_scale) +
                                static_cast<size_t>(e) * (NR / 128) * (K / 128) + k0 / 128 + lane
                          : nullptr;
    // MXFP4: the expert's E8M0 bytes [NR][K/32], at this wave's first 32-block
    const uint8_t* wsc4 = F4 ? static_cast<const uint8_t*>(GEMM1 ? g.w1_scale : g.w2_scale) +
                                   static_cast<size_t>(e) * NR * (K / 32) + k0 / 32
                             : nullptr;
    // int4: the expert's bf16 group scales [NR][K/128], at this wave's first group
    const uint16_t* wsc2 = I4 ? static_cast<const uint16_t*>(GEMM1 ? g.w1_scale : g.w2_scale) +
                                    static_cast<size_t>(e) * NR * (K / 128) + k0 / 128
                              : nullptr;
    const int nsg = (cb1 - cb0) * NST;  // stages of this run
    // stage q of the run: block cb0 + q / NST, group gi, piece p
    auto issue = [&](int q) {
      const int cb = cb0 + q / NST, r = q % NST, gi = r / NP, p = r % NP;
      const int n0 = cb * NC;
      const int wr = GEMM1 ? (gi < NG / 2 ? n0 + gi * 16 : g.I + n0 + (gi - NG / 2) * 16) : n0 + gi * 16;
      const uint8_t* src = wq + static_cast<size_t>(wr) * rowbytes + p * PC;
      const uint32_t dst = sbase + (q % NS) * STAGE;
      if (16 * lane < PC) {
#pragma unroll
        for (int i = 0; i < 16; ++i) dma16_nt(src + i * rowbytes, dst + i * ROWB);
      }
      if constexpr (F8) {  // the piece's JP / 4 block scales of the group's 128-row block
        if (lane < JP / 4) dma4(wsc + static_cast<size_t>(wr / 128) * (K / 128) + p * (PC / 128), dst + 16 * ROWB);
      }
      if constexpr (F4) {  // the piece's JP scale bytes of each of the 16 rows, [row][JP] in LDS
#pragma unroll
        for (int c = 0; c < NSI; ++c) {
          const int gi4 = 64 * c + lane, row = gi4 / (JP / 4), dw = gi4 % (JP / 4);
          if (row < 16)
            dma4(wsc4 + static_cast<size_t>(wr + row) * (K / 32) + p * JP + 4 * dw, dst + 16 * ROWB + 256 * c);
        }
      }
      if constexpr (I4) {  // the piece's JP / 4 group scales of each of the 16 rows, [row][JP / 4] in LDS
        constexpr int DW = JP / 8;  // dwords per row
        if (lane < 16 * DW)
          dma4(wsc2 + static_cast<size_t>(wr + lane / DW) * (K / 128) + p * (JP / 4) + 2 * (lane % DW),
               dst + 16 * ROWB);
      }
    };
#pragma unroll
    for (int q = 0; q < NS - 1; ++q)
      if (q < nsg) issue(q);

    for (int cb = cb0, q0 = 0; cb < cb1; ++cb, q0 += NST) {
      f32x4 acc[NG];
#pragma unroll
      for (int gi = 0; gi < NG; ++gi) acc[gi] = f32x4{};
#pragma unroll
      for (int r = 0; r < NST; ++r) {
        const int q = q0 + r, gi = r / NP, p = r % NP;
        // the copy NS-1 stages ahead goes into the buffer read out in stage q-1
        if (q + NS - 1 < nsg) issue(q + NS - 1);
        // stage q has landed once at most the later stages' CPS copies each fly
        if (NS >= 4 && q + 3 < nsg) vm_wait<3 * CPS>();
        else if (NS >= 3 && q + 2 < nsg) vm_wait<2 * CPS>();
        else if (q + 1 < nsg) vm_wait<CPS>();
        else vm_wait<0>();
        const uint8_t* St = &smem[wave][0][0] + (q % NS) * STAGE;
        if constexpr (F4) {
          const uint8_t* B = St + r16 * ROWB + 16 * kg;
          const uint8_t* sc = St + 16 * ROWB + r16 * JP + kg;  // E8M0 of (row, 32-block 4 b + kg)
#pragma unroll
          for (int b = 0; b < JP / 4; ++b) {
            const u32x4 wv = ld16(B + 64 * b);
            const float scf = __uint_as_float(static_cast<uint32_t>(sc[4 * b]) << 23);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const uint32_t w = u == 0 ? wv.x : (u == 1 ? wv.y : (u == 2 ? wv.z : wv.w));
              acc[gi] = mfma16x16x32(as_bf16x8(a[p * JP + 4 * b + u]), as_bf16x8(mxfp4x8_to_bf16(w, scf)), acc[gi]);
            }
          }
        } else if constexpr (I4) {
          const uint8_t* B = St + r16 * ROWB + 16 * kg;
          const uint16_t* sc = reinterpret_cast<const uint16_t*>(St + 16 * ROWB) + r16 * (JP / 4);
#pragma unroll
          for (int b = 0; b < JP / 4; ++b) {
            const u32x4 wv = ld16(B + 64 * b);
            f32x4 part = nbias[(p * JP) / 4 + b];
            bf16x8 dq[4];
            int4x16_biased_bf16_strided(wv.x, wv.y, dq[0], dq[1]);
            int4x16_biased_bf16_strided(wv.z, wv.w, dq[2], dq[3]);
#pragma unroll
            for (int u = 0; u < 4; ++u) part = mfma16x16x32(as_bf16x8(a[p * JP + 4 * b + u]), dq[u], part);
            const float sw = __uint_as_float(static_cast<uint32_t>(sc[b]) << 16);  // this lane's weight row
            acc[gi] += part * sw;
          }
        } else if constexpr (F8) {
          const uint8_t* B = St + r16 * ROWB + 32 * kg;
          const float* sc = reinterpret_cast<const float*>(St + 16 * ROWB);
#pragma unroll
          for (int b = 0; b < JP / 4; ++b) {
            const u32x4 w0 = ld16(B + 128 * b), w1 = ld16(B + 128 * b + 16);
            f32x4 part = {};
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const u32x4& wv = u < 2 ? w0 : w1;
              const bf16x8 bq = (u & 1) ? e4m3x8_to_bf16(wv.z, wv.w) : e4m3x8_to_bf16(wv.x, wv.y);
              part = mfma16x16x32(as_bf16x8(a[p * JP + 4 * b + u]), bq, part);
            }
            acc[gi] += part * sc[b];
          }
        } else {
          const uint8_t* B = St + r16 * ROWB + 16 * kg;
#pragma unroll
          for (int jj = 0; jj < JP; ++jj)
            acc[gi] = mfma16x16x32(as_bf16x8(a[p * JP + jj]), as_bf16x8(ld16(B + 64 * jj)), acc[gi]);
        }
        lds_wait();  // this stage's buffer is read out before a later copy lands in it
      }

      // reduce the K slices in wave order; wave 0 finishes every group (the
      // other waves go on with the next block's stages)
      if (wave > 0) {
#pragma unroll
        for (int gi = 0; gi < NG; ++gi) red[wave - 1][gi][lane] = acc[gi];
      }
      lds_wait();
      bar();
      const int n0 = cb * NC;
      auto sum = [&](int gi) {
        f32x4 v = acc[gi];
#pragma unroll
        for (int w = 1; w < NWV; ++w) v += red[w - 1][gi][lane];
        return v;
      };
      // D element i of a 16x16 tile is (row 4*(lane/16) + i, col lane%16)
      if (GEMM1) {
#pragma unroll
        for (int gi = 0; gi < NG / 2; ++gi) {
          if (wave != 0) break;
          const f32x4 gt = sum(gi), up = sum(gi + NG / 2);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int row = m0 + 4 * kg + i, col = n0 + gi * 16 + r16;
            static_cast<uint16_t*>(g.inter)[static_cast<size_t>(row) * g.I + col] =
                f32_to_bf16(silu_mul(gt[i], up[i]));
          }
        }
      } else {
#pragma unroll
        for (int gi = 0; gi < NG; ++gi) {
          if (wave != 0) break;
          const f32x4 v = sum(gi);
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (live[i]) static_cast<float*>(g.y)[static_cast<size_t>(m0 + 4 * kg + i) * g.H + n0 + gi * 16 + r16] = v[i];
        }
      }
      lds_wait();
      bar();  // red is read out before the next block writes it
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

// ------------------------------------------------ skinny, MXFP4 weights
// The decode kernel on MXFP4 weights (OCP MX: E2M1 codes, two per byte, low
// nibble first; one E8M0 scale byte per 32 along K) with bf16 activations:
// the weight-only fp8 kernel's structure (16-row tile, K split over the four
// waves in 128-wide blocks; inside a block lane group kg takes elements
// [32 kg, 32 kg + 32), 16 bytes of each weight row, and the matching 64
// bytes of its activation row).  Those 32 elements share one E8M0 scale, so
// v_cvt_scalef32_pk_bf16_fp4 decodes each code pair straight to bf16 with
// the scale applied (exact: a code times a power of two; the instruction
// takes the f32 scale's exponent field, which is the E8M0 byte itself).

template <int NSUB, int UB, bool GEMM1>
__global__ __launch_bounds__(256) void gemm_w4a16_skinny(GroupedGemm g) {
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
  const uint8_t* wbase = static_cast<const uint8_t*>(GEMM1 ? g.w1 : g.w2) + static_cast<size_t>(e) * NR * (K / 2);
  const uint8_t* sbase = static_cast<const uint8_t*>(GEMM1 ? g.w1_scale : g.w2_scale) +
                         static_cast<size_t>(e) * NR * (K / 32);
  const uint8_t* brow[NSUB];
  const uint32_t* srow[NSUB];  // the four scale bytes of each 128-wide block, one word
#pragma unroll
  for (int s = 0; s < NSUB; ++s) {
    int n;
    if (GEMM1) n = s < NSUB / 2 ? n0 + s * 16 + r16 : g.I + n0 + (s - NSUB / 2) * 16 + r16;
    else n = n0 + s * 16 + r16;
    brow[s] = wbase + static_cast<size_t>(n) * (K / 2) + kg * 16;
    srow[s] = reinterpret_cast<const uint32_t*>(sbase + static_cast<size_t>(n) * (K / 32));
  }

  f32x4 acc[NSUB];
#pragma unroll
  for (int s = 0; s < NSUB; ++s) acc[s] = f32x4{};
  const int nb = K / 128, lb = nb / 4, lr = nb % 4;
  const int bbeg = wave * lb + min(wave, lr);
  const int bend = bbeg + lb + (wave < lr ? 1 : 0);

  // UB blocks per pipeline stage: a block of MXFP4 is half the bytes of an
  // fp8 one, so two are loaded together to keep as many bytes in flight
  u32x4 a0[UB][4], b0[UB][NSUB], a1[UB][4], b1[UB][NSUB];
  uint32_t s0[UB][NSUB], s1[UB][NSUB];
#define MOE_W4_LOAD(A, Bv, Sv, blk)                                                               \
  do {                                                                                            \
    _Pragma("unroll") for (int v = 0; v < UB; ++v) {                                            \
      const int bb = min((blk) + v, bend - 1); /* a short last stage re-reads its last block */   \
      _Pragma("unroll") for (int u = 0; u < 4; ++u) A[v][u] = ld16(arow + bb * 128 + u * 8);     \
      _Pragma("unroll") for (int s = 0; s < NSUB; ++s) {                                        \
        Bv[v][s] = ld16(brow[s] + bb * 64);                                                      \
        Sv[v][s] = srow[s][bb];                                                                   \
      }                                                                                           \
    }                                                                                             \
  } while (0)
#define MOE_W4_MMA(A, Bv, Sv, blk)                                                                \
  do {                                                                                            \
    _Pragma("unroll") for (int v = 0; v < UB; ++v) {                                            \
      if ((blk) + v >= bend) break;                                                               \
      _Pragma("unroll") for (int s = 0; s < NSUB; ++s) {                                        \
        const float sc = __uint_as_float(((Sv[v][s] >> (8 * kg)) & 0xFFu) << 23);                 \
        _Pragma("unroll") for (int u = 0; u < 4; ++u) {                                         \
          const u32x4& bw = Bv[v][s];                                                             \
          const uint32_t w = u == 0 ? bw.x : (u == 1 ? bw.y : (u == 2 ? bw.z : bw.w));            \
          acc[s] = mfma16x16x32(as_bf16x8(A[v][u]), as_bf16x8(mxfp4x8_to_bf16(w, sc)), acc[s]);  \
        }                                                                                         \
      }                                                                                           \
    }                                                                                             \
  } while (0)
  int b = bbeg;
  if (b < bend) MOE_W4_LOAD(a0, b0, s0, b);
  for (; b + UB < bend; b += 2 * UB) {
    MOE_W4_LOAD(a1, b1, s1, b + UB);
    MOE_W4_MMA(a0, b0, s0, b);
    if (b + 2 * UB < bend) MOE_W4_LOAD(a0, b0, s0, b + 2 * UB);
    MOE_W4_MMA(a1, b1, s1, b + UB);
  }
  if (b < bend) MOE_W4_MMA(a0, b0, s0, b);
#undef MOE_W4_LOAD
#undef MOE_W4_MMA

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
// The 16-row decode kernels: at most 32 rows per expert on average, and H, I
// multiples of 128 (other bf16 shapes, multiples of 8, run the tiled kernels,
// which handle a ragged last K step and column tile).
bool bf16_use_skinny(int T, int top_k, int E, int H, int I) {
  return static_cast<long>(T) * top_k <= 32L * E && H % 128 == 0 && I % 128 == 0;
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

int stream_grid() {
  static const int cus = MOE_STREAM_OCC * [] {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    return n;
  }();
  return cus;
}
template <int NG, bool GEMM1>
hipError_t launch_stream(const GroupedGemm& g, hipStream_t s) {
  constexpr int NC = GEMM1 ? NG / 2 * 16 : NG * 16;
  const int K = GEMM1 ? g.H : g.I;
  // one workgroup per CU, at most one per (row tile, column block) unit
  const long units = static_cast<long>(g.max_rows / 16) * ((GEMM1 ? g.I : g.H) / NC);
  const dim3 grid(static_cast<unsigned>(std::max(1L, std::min<long>(stream_grid(), units))));
#define MOE_STREAM_CASE(NP, JP) \
  hipLaunchKernelGGL((gemm_bf16_stream<0, 4, NG, NP, JP, GEMM1>), grid, dim3(256), 0, s, g)
  const int qb = K / 2;  // bytes of a row per wave
  if (qb % 512 == 0) {   // 512-byte pieces
    switch (qb / 512) {
      case 1: MOE_STREAM_CASE(1, 8); break;
      case 2: MOE_STREAM_CASE(2, 8); break;
      case 3: MOE_STREAM_CASE(3, 8); break;
      default: MOE_STREAM_CASE(4, 8); break;
    }
  } else {  // one piece: the quarter is 64 * JP bytes
    switch (qb / 64) {
      case 1: MOE_STREAM_CASE(1, 1); break;
      case 2: MOE_STREAM_CASE(1, 2); break;
      case 3: MOE_STREAM_CASE(1, 3); break;
      case 4: MOE_STREAM_CASE(1, 4); break;
      case 5: MOE_STREAM_CASE(1, 5); break;
      case 6: MOE_STREAM_CASE(1, 6); break;
      case 7: MOE_STREAM_CASE(1, 7); break;
      case 9: MOE_STREAM_CASE(1, 9); break;
      case 10: MOE_STREAM_CASE(1, 10); break;
      case 11: MOE_STREAM_CASE(1, 11); break;
      case 12: MOE_STREAM_CASE(1, 12); break;
      case 13: MOE_STREAM_CASE(1, 13); break;
      case 14: MOE_STREAM_CASE(1, 14); break;
      default: MOE_STREAM_CASE(1, 15); break;
    }
  }
#undef MOE_STREAM_CASE
  return hipGetLastError();
}

// fp8 weights (one byte per element): the wave's quarter of a row, K/4
// bytes (whole 128-wide blocks), is one piece of up to 1 KB.  Above that
// (K = 7168: two pieces) the 56 activation fragments a wave would hold spill
// (measured 523 us against the skinny kernel's 385 us), so those shapes keep
// the skinny kernel.
template <int NG, bool GEMM1>
hipError_t launch_stream_f8(const GroupedGemm& g, hipStream_t s) {
  constexpr int NC = GEMM1 ? NG / 2 * 16 : NG * 16;
  const int K = GEMM1 ? g.H : g.I;
  const long units = static_cast<long>(g.max_rows / 16) * ((GEMM1 ? g.I : g.H) / NC);
  const dim3 grid(static_cast<unsigned>(std::max(1L, std::min<long>(stream_grid(), units))));
#define MOE_STREAM_CASE(JP) \
  hipLaunchKernelGGL((gemm_bf16_stream<3, 4, NG, 1, JP, GEMM1>), grid, dim3(256), 0, s, g)
  switch (K / 512) {
    case 1: MOE_STREAM_CASE(4); break;
    case 2: MOE_STREAM_CASE(8); break;
    case 3: MOE_STREAM_CASE(12); break;
    case 4: MOE_STREAM_CASE(16); break;
    case 5: MOE_STREAM_CASE(20); break;
    case 6: MOE_STREAM_CASE(24); break;
    case 7: MOE_STREAM_CASE(28); break;
    default: MOE_STREAM_CASE(32); break;
  }
#undef MOE_STREAM_CASE
  return hipGetLastError();
}
bool stream_fits_f8(int K, int N, int nc) { return MOE_STREAM && K % 512 == 0 && K <= 4096 && N % nc == 0; }

// MXFP4 weights (half a byte per element): one piece per wave and row, the
// wave's K range = K / NWV elements held as activation fragments (at most
// 32); four waves up to K = 4096, eight (K in eighths) up to 7168 (at 8192
// eight waves' two stage buffers no longer fit LDS beside the reduction).
template <int NG, bool GEMM1>
hipError_t launch_stream_f4(const GroupedGemm& g, hipStream_t s) {
  constexpr int NC = GEMM1 ? NG / 2 * 16 : NG * 16;
  const int K = GEMM1 ? g.H : g.I;
  const long units = static_cast<long>(g.max_rows / 16) * ((GEMM1 ? g.I : g.H) / NC);
  const dim3 grid(static_cast<unsigned>(std::max(1L, std::min<long>(stream_grid(), units))));
#define MOE_STREAM_CASE(NWV, JP) \
  hipLaunchKernelGGL((gemm_bf16_stream<4, NWV, NG, 1, JP, GEMM1>), grid, dim3(64 * NWV), 0, s, g)
  if (MOE_STREAM_F4_HALF && K <= 2048) {
    // two waves (K in halves): pieces twice as long, twice the workgroups
    const dim3 grid2(static_cast<unsigned>(std::max(1L, std::min<long>(2L * stream_grid(), units))));
#define MOE_STREAM_CASE2(JP) \
    hipLaunchKernelGGL((gemm_bf16_stream<4, 2, NG, 1, JP, GEMM1>), grid2, dim3(128), 0, s, g)
    switch (K / 512) {
      case 1: MOE_STREAM_CASE2(8); break;
      case 2: MOE_STREAM_CASE2(16); break;
      case 3: MOE_STREAM_CASE2(24); break;
      default: MOE_STREAM_CASE2(32); break;
    }
#undef MOE_STREAM_CASE2
    return hipGetLastError();
  }
  if (K <= 4096) {
    switch (K / 512) {
      case 1: MOE_STREAM_CASE(4, 4); break;
      case 2: MOE_STREAM_CASE(4, 8); break;
      case 3: MOE_STREAM_CASE(4, 12); break;
      case 4: MOE_STREAM_CASE(4, 16); break;
      case 5: MOE_STREAM_CASE(4, 20); break;
      case 6: MOE_STREAM_CASE(4, 24); break;
      case 7: MOE_STREAM_CASE(4, 28); break;
      default: MOE_STREAM_CASE(4, 32); break;
    }
  } else {
    switch (K / 1024) {
      case 5: MOE_STREAM_CASE(8, 20); break;
      case 6: MOE_STREAM_CASE(8, 24); break;
      default: MOE_STREAM_CASE(8, 28); break;
    }
  }
#undef MOE_STREAM_CASE
  return hipGetLastError();
}
bool stream_fits_f4(int K, int N, int nc) {
  return MOE_STREAM && K % 512 == 0 && K <= 7168 && (K <= 4096 || K % 1024 == 0) && N % nc == 0;
}

// int4 weights (half a byte per element, a bf16 scale per 128-wide group):
// one piece per wave and row, whose group scales must be whole dwords (JP a
// multiple of 8): two waves (K in halves, two workgroups per CU) up to
// K = 2048, four waves for K = 3072 and 4096.
template <int NG, bool GEMM1>
hipError_t launch_stream_i4(const GroupedGemm& g, hipStream_t s) {
  constexpr int NC = GEMM1 ? NG / 2 * 16 : NG * 16;
  const int K = GEMM1 ? g.H : g.I;
  const long units = static_cast<long>(g.max_rows / 16) * ((GEMM1 ? g.I : g.H) / NC);
#define MOE_STREAM_CASE(NWV, JP, GRID) \
  hipLaunchKernelGGL((gemm_bf16_stream<2, NWV, NG, 1, JP, GEMM1>), GRID, dim3(64 * NWV), 0, s, g)
  if (K <= 2048) {
    const dim3 grid2(static_cast<unsigned>(std::max(1L, std::min<long>(2L * stream_grid(), units))));
    switch (K / 512) {
      case 1: MOE_STREAM_CASE(2, 8, grid2); break;
      case 2: MOE_STREAM_CASE(2, 16, grid2); break;
      case 3: MOE_STREAM_CASE(2, 24, grid2); break;
      default: MOE_STREAM_CASE(2, 32, grid2); break;
    }
  } else {
    const dim3 grid(static_cast<unsigned>(std::max(1L, std::min<long>(stream_grid(), units))));
    if (K == 3072) MOE_STREAM_CASE(4, 24, grid);
    else MOE_STREAM_CASE(4, 32, grid);
  }
#undef MOE_STREAM_CASE
  return hipGetLastError();
}
bool stream_fits_i4(int K, int N, int nc) {
  return MOE_STREAM && K % 512 == 0 && (K <= 2048 || K == 3072 || K == 4096) && N % nc == 0;
}
// Both int4 products fit the streamed kernel (the 16-row decode route)
bool int4_stream_fits(int H, int I) {
  return stream_fits_i4(H, I, MOE_STREAM_NG1 / 2 * 16) && stream_fits_i4(I, H, MOE_STREAM_NG2 * 16);
}
hipError_t launch_gemm1_int4_stream(const GroupedGemm& g, hipStream_t s) {
  return launch_stream_i4<MOE_STREAM_NG1, true>(g, s);
}
hipError_t launch_gemm2_int4_stream(const GroupedGemm& g, hipStream_t s) {
  return launch_stream_i4<MOE_STREAM_NG2, false>(g, s);
}

// Streamed when each wave's quarter of a row is whole 512-byte pieces (K a
// multiple of 1024, up to 4096) or one piece under 1 KB (K < 2048)
bool stream_fits(int K, int N, int nc) {
  return MOE_STREAM && ((K % 1024 == 0 && K <= 4096) || K < 2048) && N % nc == 0;
}

hipError_t launch_gemm1_bf16(const GroupedGemm& g, hipStream_t s) {
  if (bf16_use_skinny(g.T, g.top_k, g.E, g.H, g.I) && stream_fits(g.H, g.I, MOE_STREAM_NG1 / 2 * 16))
    return launch_stream<MOE_STREAM_NG1, true>(g, s);
  if (bf16_use_skinny(g.T, g.top_k, g.E, g.H, g.I)) {
    constexpr int NS = MOE_SKINNY1_NSUB;
    const dim3 grid(g.I / (NS / 2 * 16), g.max_rows / 16);
    hipLaunchKernelGGL((gemm_bf16_skinny<NS, MOE_SKINNY1_UNROLL, true>), grid, dim3(256), 0, s, g);
    return hipGetLastError();
  }
  return launch_gemm1_bf16_tiled(g, s);
}

hipError_t launch_gemm2_bf16(const GroupedGemm& g, hipStream_t s) {
  if (bf16_use_skinny(g.T, g.top_k, g.E, g.H, g.I) && stream_fits(g.I, g.H, MOE_STREAM_NG2 * 16))
    return launch_stream<MOE_STREAM_NG2, false>(g, s);
  if (bf16_use_skinny(g.T, g.top_k, g.E, g.H, g.I)) {
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
  if (stream_fits_f8(g.H, g.I, MOE_STREAM_NG1 / 2 * 16)) return launch_stream_f8<MOE_STREAM_NG1, true>(g, s);
  constexpr int NS = MOE_W8_NSUB;
  const dim3 grid(g.I / (NS / 2 * 16), g.max_rows / 16);
  hipLaunchKernelGGL((gemm_w8a16_skinny<NS, true>), grid, dim3(256), 0, s, g);
  return hipGetLastError();
}
// MXFP4 weights (decode route; the host guarantees T*k <= 32*E)
#ifndef MOE_W4_NSUB
#define MOE_W4_NSUB 4
#endif
#ifndef MOE_W4_UB
#define MOE_W4_UB 2
#endif
hipError_t launch_gemm1_w4a16(const GroupedGemm& g, hipStream_t s) {
  if (stream_fits_f4(g.H, g.I, MOE_STREAM_NG1 / 2 * 16)) return launch_stream_f4<MOE_STREAM_NG1, true>(g, s);
  constexpr int NS = MOE_W4_NSUB;
  const dim3 grid(g.I / (NS / 2 * 16), g.max_rows / 16);
  hipLaunchKernelGGL((gemm_w4a16_skinny<NS, MOE_W4_UB, true>), grid, dim3(256), 0, s, g);
  return hipGetLastError();
}
hipError_t launch_gemm2_w4a16(const GroupedGemm& g, hipStream_t s) {
  if (stream_fits_f4(g.I, g.H, MOE_STREAM_NG2 * 16)) return launch_stream_f4<MOE_STREAM_NG2, false>(g, s);
  constexpr int NS = MOE_W4_NSUB;
  const dim3 grid(g.H / (NS * 16), g.max_rows / 16);
  hipLaunchKernelGGL((gemm_w4a16_skinny<NS, MOE_W4_UB, false>), grid, dim3(256), 0, s, g);
  return hipGetLastError();
}
hipError_t launch_gemm2_w8a16(const GroupedGemm& g, hipStream_t s) {
  if (stream_fits_f8(g.I, g.H, MOE_STREAM_NG2 * 16)) return launch_stream_f8<MOE_STREAM_NG2, false>(g, s);
  constexpr int NS = MOE_W8_NSUB;
  const dim3 grid(g.H / (NS * 16), g.max_rows / 16);
  hipLaunchKernelGGL((gemm_w8a16_skinny<NS, false>), grid, dim3(256), 0, s, g);
  return hipGetLastError();
}

int gemm_block_m_bf16(int T, int top_k, int E, int H, int I) {
  return bf16_use_skinny(T, top_k, E, H, I) ? 16 : bf16_tiled_block_m();
}

}  // namespace moe
