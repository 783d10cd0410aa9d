// Grouped expert GEMMs, LDS-tiled, for the three weight formats (the "Fused
// MoE" node of the paper's skeleton, Fig. 1 / Fig. 3; the quantised formats
// carry the numeric semantics Sec. 6.2 asks of quantised routes):
//   GEMM1  a = SiLU(x W1[e,:I]^T) * (x W1[e,I:]^T)     (SiLU*up epilogue)
//   GEMM2  y = a W2[e]^T
//
//  bf16  A, B bf16; v_mfma_f32_32x32x16_bf16.
//  fp8   A (activations) and B (weights) OCP e4m3; v_mfma_f32_32x32x64_f8f6f4
//        with W as the first operand (the product is formed transposed),
//        one 128-wide K block at a time into a fresh partial, then
//        acc += partial * s_row(A) * s_block(B) on the VALU, overlapped with
//        the next blocks' MFMAs.  The GEMM1 epilogue requantises the
//        intermediate per (row, 128 columns): the tile holds exactly one such
//        group per row.
//  int4  A bf16; B signed int4 words decoded in registers (q * bf16 scale,
//        rounded to bf16) right before the bf16 MFMA, never materialised.
//  mxfp4 A bf16; B OCP MX E2M1 codes with an E8M0 scale per 32 elements,
//        decoded by v_cvt_scalef32_pk_bf16_fp4 (exact: the bf16 result is the
//        code's value times a power of two) right before the bf16 MFMA.
// Every GEMM2 also forms its product transposed (four consecutive output
// columns per lane, so y goes out in 16-byte stores).
//
// Each K step streams KB bytes of every A row through LDS -- 128 (64 bf16 /
// 128 fp8 elements), or 256 for the 4-bit formats (128 elements, so each
// weight row gives 64 bytes, half a cache line) -- in 16-byte chunks XOR-swizzled by row
// so that the fragment reads are bank-conflict free; B rows likewise.
//
// Scheduling is persistent and XCD-aware: the launch has a few workgroups per
// CU; workgroups that land on one XCD (block ids congruent mod 8) own one
// contiguous range of logical tiles, ordered expert by expert in chunks of at
// most GM row tiles x all column tiles, so the weight slab and row tiles that
// concurrently running workgroups share are read from HBM about once.  The
// number of real row tiles is read on the device from expert_offsets[E]
// (segments are padded to BM).
#include <algorithm>

#include "common.hpp"
#include "launch.hpp"
#include "lds_dma.hpp"

namespace moe {

constexpr int kXcds = 8;
constexpr int MOE_MAX_EXPERTS_DEV = 1024;  // the ABI's expert limit

// Sixteen zero bytes: the source of every bf16 copy chunk that lies past the
// end of K (K a multiple of 8 but not of the 64-element step), so a ragged
// last step multiplies zeros and reads nothing beyond a row.
__device__ __align__(16) const uint8_t kZeroChunk[16] = {};

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

// 8 signed nibbles -> 8 bf16 values 136 + q, exact: the bits are 0x4300 | (q + 8)
// (128 + (q + 8), the nibble in the low mantissa bits of 128).  Element k of
// the word (bits [4k, 4k+4)) lands in half k % 2 of dword k / 2.  `keep` = 0
// turns every code into q = 0.  The v_bitop3 immediate is the truth table
// over (S0, S1, S2) = (0xF0, 0xCC, 0xAA): 0x6A = (S0 & S1) ^ S2.
__device__ __forceinline__ bf16x8 int4x8_biased_bf16(uint32_t w, uint32_t keep) {
  const uint32_t y = __builtin_amdgcn_bitop3_b32(w, keep, 0x88888888u, 0x6A);  // q + 8 per nibble
  const uint32_t y4 = y >> 4;                                                  // odd nibbles moved down
  u32x4 r;
  r.x = (__builtin_amdgcn_perm(y4, y, 0x0c040c00u) & 0x000F000Fu) | 0x43004300u;
  r.y = (__builtin_amdgcn_perm(y4, y, 0x0c050c01u) & 0x000F000Fu) | 0x43004300u;
  r.z = (__builtin_amdgcn_perm(y4, y, 0x0c060c02u) & 0x000F000Fu) | 0x43004300u;
  r.w = (__builtin_amdgcn_perm(y4, y, 0x0c070c03u) & 0x000F000Fu) | 0x43004300u;
  return as_bf16x8(r);
}

// XOR swizzle of the 16-byte chunks of a 128-byte LDS row: row r stores its
// chunk c in slot c ^ swz<KB>(r).  For the fragment reads (32 consecutive rows,
// lanes l and l+32 on neighbouring chunks of one row) (r >> 1) & 7 measured
// 1.6x the LDS read throughput of r & 7 on gfx950.
// With 64-byte rows (4 chunks) the analogous choice is (r >> 2) & 3; a
// 256-byte row spans all 64 banks, so there the slot alone must tell 16
// consecutive rows apart: r & 15.
template <int KB>
__device__ __forceinline__ int swz(int r) { return KB == 256 ? r & 15 : KB == 128 ? (r >> 1) & 7 : (r >> 2) & 3; }
// int4 B rows (32 or 64 bytes: 2 or 4 chunks)
// (128-byte 4-bit rows, 256-element MXFP8 steps: as swz<128>)
template <int BB>
__device__ __forceinline__ int swz_b(int r) { return BB == 32 ? (r >> 2) & 1 : BB == 64 ? (r >> 2) & 3 : (r >> 1) & 7; }

// NP > 0: NP extra waves only issue the global->LDS copies and the NW math
// waves never touch global memory in the main loop, so a stalled load queue
// (L1 waiting on L2) cannot hold up the MFMA stream behind an in-order copy
// instruction.  NP == 0: the math waves issue the copies themselves.
template <int FMT, bool GEMM1, int BM, int BNW, int WM, int WN, int GM, int KBT = 128, int STAGES = 3, int NP = 0>
// The 64-row 4-bit GEMMs with copy waves are held to 128 registers, which keeps two workgroups per CU.
__global__ __launch_bounds__((WM * WN + NP) * 64) __attribute__((amdgpu_waves_per_eu((FMT == 2 || FMT == 4) && (GEMM1 || NP > 0) && BM == 64 ? 4 : 1)))
void moe_gemm_tiled(GroupedGemm g) {
  constexpr int NW = WM * WN, NT = (NW + NP) * 64;
  constexpr int LW = NP > 0 ? NP : NW;  // waves that issue the copies
  static_assert(NW == 4 || NW == 8, "four or eight math waves");
  static_assert(NP == 0 || NW % NP == 0, "scale slots split evenly over the copy waves");
  static_assert(NP == 0 || WM * WN == 4, "split launches have one math wave per SIMD");
  constexpr bool F4B = FMT == 2 || FMT == 4;  // 4-bit weights (int4, MXFP4), bf16 activations
  constexpr bool MX8 = FMT == 5;              // MXFP4 weights, MXFP8 activations
  constexpr bool A8 = FMT == 1 || MX8;        // one-byte (e4m3) activations
  constexpr bool B4 = F4B || MX8;             // 4-bit weight rows
  static_assert(KBT == 128 || (KBT == 64 && FMT == 0) || (KBT == 256 && (F4B || FMT == 5)),
                "64-byte steps are bf16 only, 256-byte steps 4-bit weights only");
  constexpr int KB = KBT;                                       // A bytes per row per step
  constexpr int KE = A8 ? KB : KB / 2;                                 // K elements per step
  constexpr int BB = B4 ? KE / 2 : KB;                                 // B bytes per row per step
  constexpr int LPB = BB / 16;                                         // lanes per 4-bit B row in a copy
  // bf16 and int4 GEMM2 form their product transposed, as fp8 does (16-byte
  // y stores, one pad check per row; bf16 prefill 4 % faster, GEMM1 was not)
  constexpr bool TRB = !A8 && !GEMM1;
  constexpr int RPI = 1024 / KB, LPR = KB / 16;  // rows per DMA instruction, lanes per row
  constexpr int WTM = BM / WM, WTN = BNW / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int NC = GEMM1 ? BNW / 2 : BNW;  // output columns per tile
  // 16-byte DMA instructions per copy wave per stage (each moves 1 KB)
  constexpr int A_CH = BM * KB / 1024 / LW, B_CH = BNW * BB / 1024 / LW;
  static_assert(A_CH >= 1 && B_CH >= 1 && A_CH * LW * 1024 == BM * KB && B_CH * LW * 1024 == BNW * BB, "");
  static_assert(!GEMM1 || TN % 2 == 0, "gate/up pairs");
  static_assert(FMT != 1 || !GEMM1 || NC == 128, "fp8 requant needs one 128-column group per tile");
  static_assert(!MX8 || (NP > 0 && WM * WN == 4), "MXFP8: four math waves beside copy waves");
  // per-stage scale block: NW slots of 256 bytes, one 4-byte DMA instruction
  // each (64 floats); fp8: slots [0, BM/64) the row scales of A, slot BM/64
  // the block scales of B; int4: slots [0, BNW/64) the bf16 pair holding each
  // B row's group scale, int4 GEMM1 also slots [BNW/64, BNW/64 + BM/64) the
  // rows' biased group sums (x_gsum).  Copy wave lw fills slots lw, lw + LW, ...
  // MXFP8: MXD E8M0 dwords per row per step (four 32-element blocks each);
  // slots [0, MXD BM/64) the A rows' dwords (slot d BM/64 + g: dword d of
  // row group g), then MXD BNW/64 slots of the B rows' likewise; slots past
  // those load a harmless dummy.
  constexpr bool GSUM = FMT == 2 && GEMM1;
  constexpr int MXD = MX8 ? KE / 128 : 1;
  constexpr int NSLOT = FMT == 0 ? 0 : (MX8 ? MXD * (BM + BNW) / 64 : (GSUM ? 2 : 1) * NW);
  constexpr int SC = (NSLOT + LW - 1) / LW;  // scale loads per copy wave per stage
  static_assert(FMT != 1 || BM / 64 < NW, "fp8 scale DMA layout");
  static_assert(!F4B || (NW == 4 && BNW / 64 <= NW), "4-bit scale DMA layout");
  static_assert(!GSUM || (BNW / 64 + BM / 64 <= 2 * NW && STAGES == 2), "int4 group-sum DMA layout");
  static_assert(STAGES >= 2 && (STAGES - 2) * (A_CH + B_CH + SC) < 64, "vmcnt range");
  constexpr int A_BYTES = BM * KB, B_BYTES = BNW * BB, S_BYTES = SC * LW * 256;
  constexpr int STAGE = A_BYTES + B_BYTES + S_BYTES;
  constexpr int N_DMA = A_CH + B_CH + SC;  // loads per copy wave per stage

  __shared__ __attribute__((aligned(1024))) uint8_t smem[STAGES][STAGE];
  __shared__ float lds_amax[FMT == 1 && GEMM1 ? WN : 1][FMT == 1 && GEMM1 ? BM : 1];
  __shared__ int lds_off[MOE_MAX_EXPERTS_DEV + 1];  // expert_offsets, read once per workgroup
  // copy waves: the next tile's row ids, one slot per copy wave
  __shared__ int lds_sid[NP > 0 ? NP : 1][NP > 0 ? BM : 1];

  const int tid = threadIdx.x, lane = lane_id(), wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const bool is_math = wave < NW;                       // uniform per wave
  const bool is_loader = NP == 0 || wave >= NW;
  // copy-wave index (math waves of a split launch take 0: their sources stay in range, unused)
  const int lw = NP > 0 ? (is_loader ? wave - NW : 0) : wave;
  const int l32 = lane & 31, kg = lane >> 5;
  const int K = GEMM1 ? g.H : g.I;
  const int N = GEMM1 ? g.I : g.H;       // output columns of the product
  // bf16 only: K and N multiples of 8 -- a ragged last K step (zero chunks)
  // and a ragged last column tile (weight rows clamped, stores masked); the
  // quantised formats have K and N multiples of 128
  const int nk = (K + KE - 1) / KE;
  const int n_tiles_n = (N + NC - 1) / NC;
  for (int i = tid; i <= g.E; i += NT) lds_off[i] = g.offsets[i];
  __syncthreads();
  const int n_tiles_m = lds_off[g.E] / BM;
  const int total = n_tiles_m * n_tiles_n;

  // this workgroup's share of the logical tiles: a contiguous range per XCD
  const int xcd = blockIdx.x % kXcds, slot = blockIdx.x / kXcds;
  const int per_xcd = gridDim.x / kXcds;
  const int chunk = (total + kXcds - 1) / kXcds;
  const int t_end = min(total, (xcd + 1) * chunk);
  const uint32_t smem0 = lds_addr(&smem[0][0]);

  // Logical tile order: expert by expert; inside expert e (row tiles
  // [base, base+cnt)) chunks of at most GM row tiles, each chunk swept
  // column tile by column tile with its row tiles adjacent.  Workgroups
  // running together then share one expert's weight slab and a few row tiles.
  auto coords = [&](int t, int& e, int& m0, int& n0) {
    e = find_segment(lds_off, g.E, (t / n_tiles_n) * BM);
    const int base = lds_off[e] / BM, cnt = (lds_off[e + 1] - lds_off[e]) / BM;
    const int local = t - base * n_tiles_n;
    const int c = local / (GM * n_tiles_n), within = local % (GM * n_tiles_n);
    const int sz = min(GM, cnt - c * GM);
    const int mt = base + c * GM + within % sz, nt = within / sz;
    m0 = mt * BM;
    n0 = nt * NC;
  };

  constexpr int NSL = SC > 0 ? SC : 1;
  struct Src {
    const uint8_t* a[A_CH];  // A rows
    int am[A_CH];            // A step-advance mask: -1, or 0 for a pad row (its source is the zero chunk)
    const uint8_t* b[B_CH];  // B rows
    const uint8_t* s[NSL];   // scale words
    int ss[NSL];             // scale advance per step
  };
  // staged: the tile's BM row ids are in this copy wave's lds_sid slot (else
  // they are read from sorted_ids)
  auto sources = [&](int e, int m0, int n0, Src& src, bool staged) {
    // per-lane DMA sources of the tile.  Instruction i of copy wave lw fills the 1 KB
    // block (i*LW + lw) of a stage: 1024/KB rows of A / of fp8-bf16 B (KB/16
    // lanes per row, one 16-byte slot each) or 64/LPB rows of int4 B (LPB
    // lanes per row).  Slot s of row r holds the row's chunk s ^ swz(r), the
    // XOR swizzle the fragment reads undo.
    // GEMM1 gathers its A rows by token: every row id this lane needs (A rows,
    // fp8 row scales) is requested before the first is used, so the tile
    // pays one memory round trip.  A pad row (id n_routed) of either product
    // copies the zero chunk at every step: one cache line per instruction
    // rather than a row's eight, and zeros in LDS; its products are never
    // read.  Scale sources of pad rows read the last token's.
    int sid[A_CH + NSL];
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
      const int r = (i * LW + lw) * RPI + lane / LPR;
      if constexpr (NP > 0) sid[i] = staged ? lds_sid[lw][r] : g.sorted_ids[m0 + r];
      else sid[i] = g.sorted_ids[m0 + r];
    }
    if constexpr (GEMM1) {
#pragma unroll
      for (int k = 0; k < NSL; ++k) {
        const int r = (lw + k * LW) * 64 + lane;
        int v = 0;
        if (A8 && lw + k * LW < MXD * (BM / 64)) {
          const int ra = ((lw + k * LW) % (BM / 64)) * 64 + lane;  // A row of the slot
          if constexpr (NP > 0) v = staged ? lds_sid[lw][ra] : g.sorted_ids[m0 + ra];
          else v = g.sorted_ids[m0 + ra];
        }
        const int rg = (lw + k * LW - BNW / 64) * 64 + lane;  // group-sum slot row
        if (GSUM && lw + k * LW >= BNW / 64 && lw + k * LW < BNW / 64 + BM / 64) {
          if constexpr (NP > 0) v = staged ? lds_sid[lw][rg] : g.sorted_ids[m0 + rg];
          else v = g.sorted_ids[m0 + rg];
        }
        sid[A_CH + k] = v;
      }
    }
    auto token = [&](int v) {
      return static_cast<size_t>(static_cast<unsigned>(min(v, g.n_routed - 1)) / static_cast<unsigned>(g.top_k));
    };
#pragma unroll
    for (int i = 0; i < A_CH; ++i) {
      const int r = (i * LW + lw) * RPI + lane / LPR;
      const uint8_t* row;
      if (GEMM1) {
        row = static_cast<const uint8_t*>(g.x) + token(sid[i]) * g.H * (A8 ? 1 : 2);
      } else {
        row = static_cast<const uint8_t*>(g.inter) + static_cast<size_t>(m0 + r) * g.I * (A8 ? 1 : 2);
      }
      const bool pad = sid[i] >= g.n_routed;
      src.a[i] = pad ? static_cast<const uint8_t*>(kZeroChunk) : row + (((lane % LPR) ^ swz<KB>(r)) << 4);
      src.am[i] = pad ? 0 : -1;
    }
    const size_t w_row_bytes = FMT == 0 ? K * 2 : (FMT == 1 ? K : K / 2);
    const uint8_t* wbase = static_cast<const uint8_t*>(GEMM1 ? g.w1 : g.w2) +
                           static_cast<size_t>(e) * (GEMM1 ? 2 * g.I : g.H) * w_row_bytes;
#pragma unroll
    for (int i = 0; i < B_CH; ++i) {
      const int blk = i * LW + lw;
      const int r = B4 ? blk * (64 / LPB) + lane / LPB : blk * RPI + lane / LPR;
      const int sl = B4 ? (lane % LPB) ^ swz_b<BB>(r) : (lane % LPR) ^ swz<KB>(r);
      // weight rows past N (a ragged last column tile) read the last row:
      // their columns are never stored
      int n;
      if (GEMM1) n = r < NC ? min(n0 + r, g.I - 1) : g.I + min(n0 + (r - NC), g.I - 1);
      else n = min(n0 + r, g.H - 1);
      src.b[i] = wbase + static_cast<size_t>(n) * w_row_bytes + (sl << 4);
    }
    // scale DMA sources of this lane, one per slot lw + k*LW (advanced by one
    // K block / half group per step); slots without a scale role load a
    // harmless dummy
#pragma unroll
    for (int k = 0; k < NSL; ++k) {
      const int sl = lw + k * LW;
      src.s[k] = src.a[0];
      src.ss[k] = 0;
      if constexpr (FMT == 1) {
        if (sl < BM / 64) {
          const int r = sl * 64 + lane;
          if (GEMM1) {
            src.s[k] = reinterpret_cast<const uint8_t*>(g.x_scale + token(sid[A_CH + k]) * (g.H / 128));
          } else {
            src.s[k] = reinterpret_cast<const uint8_t*>(g.inter_scale + static_cast<size_t>(m0 + r) * (g.I / 128));
          }
          src.ss[k] = 4;
        } else if (sl == BM / 64) {
          // lane l: block row of W (GEMM1: l odd -> up half, even -> gate half;
          // GEMM2: block row n0/128 + l % (BNW/128))
          const float* wsc = static_cast<const float*>(GEMM1 ? g.w1_scale : g.w2_scale) +
                             static_cast<size_t>(e) * ((GEMM1 ? 2 * g.I : g.H) / 128) * (K / 128);
          const int br = GEMM1 ? ((lane & 1) ? (g.I + n0) / 128 : n0 / 128) : n0 / 128 + lane % (BNW / 128);
          src.s[k] = reinterpret_cast<const uint8_t*>(wsc + static_cast<size_t>(br) * (K / 128));
          src.ss[k] = 4;
        }
      } else if constexpr (FMT == 2) {
        if (sl < BNW / 64) {
          const int r = sl * 64 + lane;
          const int n = GEMM1 ? (r < NC ? n0 + r : g.I + n0 + (r - NC)) : n0 + r;
          // bf16 scale [n][group] of K step kt sits at element n*(K/128) + kt/2;
          // the dword holding it starts at the even element below
          src.s[k] = reinterpret_cast<const uint8_t*>(static_cast<const uint16_t*>(GEMM1 ? g.w1_scale : g.w2_scale) +
                                                      (static_cast<size_t>(e) * (GEMM1 ? 2 * g.I : g.H) + n) * (K / 128));
          src.ss[k] = 1;  // advanced per step in elements below
        } else if (GSUM && sl < BNW / 64 + BM / 64) {
          // row (sl - BNW/64)*64 + lane: its token's sum over K step kt's group, one float per step
          src.s[k] = reinterpret_cast<const uint8_t*>(g.x_gsum + token(sid[A_CH + k]) * (g.H / 128));
          src.ss[k] = 4;
        }
      } else if constexpr (MX8) {
        if (sl < MXD * (BM / 64)) {
          // A row (sl % (BM/64))*64 + lane: its E8M0 bytes [K/32]; dword sl / (BM/64) of step kt
          const int r = (sl % (BM / 64)) * 64 + lane, d = sl / (BM / 64);
          if (GEMM1) src.s[k] = g.x_mx + token(sid[A_CH + k]) * (g.H / 32) + 4 * d;
          else src.s[k] = g.inter_mx + static_cast<size_t>(m0 + r) * (g.I / 32) + 4 * d;
          src.ss[k] = 4 * MXD;
        } else if (sl < MXD * (BM / 64 + BNW / 64)) {
          const int sb2 = sl - MXD * (BM / 64);
          const int r = (sb2 % (BNW / 64)) * 64 + lane, d = sb2 / (BNW / 64);
          const int n = GEMM1 ? (r < NC ? n0 + r : g.I + n0 + (r - NC)) : n0 + r;
          src.s[k] = static_cast<const uint8_t*>(GEMM1 ? g.w1_scale : g.w2_scale) +
                     (static_cast<size_t>(e) * (GEMM1 ? 2 * g.I : g.H) + n) * (K / 32) + 4 * d;
          src.ss[k] = 4 * MXD;
        }
      } else if constexpr (FMT == 4) {
        if (sl < BNW / 64) {
          // E8M0 bytes [n][K/32]: the four of K step kt are one dword at byte 4 kt
          const int r = sl * 64 + lane;
          const int n = GEMM1 ? (r < NC ? n0 + r : g.I + n0 + (r - NC)) : n0 + r;
          src.s[k] = static_cast<const uint8_t*>(GEMM1 ? g.w1_scale : g.w2_scale) +
                     (static_cast<size_t>(e) * (GEMM1 ? 2 * g.I : g.H) + n) * (K / 32);
          src.ss[k] = 4;
        }
      }
    }
  };

  // issue step kt of the tile `src` describes (DMA q in [q0, q1) of this copy
  // wave's A_CH + B_CH tile loads, plus the scale loads with q1 == N_DMA)
  // into LDS buffer `buf`
  // bf16 ragged K: in the last step a lane whose 8-element chunk starts at
  // or past K copies the zero chunk instead (A row chunk (lane % LPR) ^ swz(r),
  // r the row the instruction's lane covers; the bf16 B rows likewise)
  const bool k_ragged = FMT == 0 && K % KE != 0;
  auto tail_src = [&](const uint8_t* p, int blk, int kt) {
    const int r = blk * RPI + lane / LPR;
    const int c = (lane % LPR) ^ swz<KB>(r);
    return kt * KE + 8 * c >= K ? static_cast<const uint8_t*>(kZeroChunk) : p;
  };
  auto issue_part = [&](const Src& src, int kt, int buf, int q0, int q1) {
    const uint32_t base = smem0 + buf * STAGE;
    if (FMT == 0 && k_ragged && kt == nk - 1) {  // uniform: only the last step of a ragged K
#pragma unroll
      for (int i = 0; i < A_CH; ++i)
        if (i >= q0 && i < q1) dma16(tail_src(src.a[i] + (kt * KB & src.am[i]), i * LW + lw, kt), base + (i * LW + lw) * 1024);
#pragma unroll
      for (int i = 0; i < B_CH; ++i)
        if (A_CH + i >= q0 && A_CH + i < q1)
          dma16(tail_src(src.b[i] + kt * BB, i * LW + lw, kt), base + A_BYTES + (i * LW + lw) * 1024);
    } else {
#pragma unroll
      for (int i = 0; i < A_CH; ++i)
        if (i >= q0 && i < q1) dma16(src.a[i] + (kt * KB & src.am[i]), base + (i * LW + lw) * 1024);
#pragma unroll
      for (int i = 0; i < B_CH; ++i)
        if (A_CH + i >= q0 && A_CH + i < q1) dma16(src.b[i] + kt * BB, base + A_BYTES + (i * LW + lw) * 1024);
    }
    if (q1 < N_DMA) return;
#pragma unroll
    for (int k = 0; k < SC; ++k) {
      // int4 GEMM1 (two stages, so every wait drains all loads and the
      // per-wave load counts need not match) skips its empty slots
      if (GSUM && src.ss[k] == 0) continue;
      const uint32_t dst = base + A_BYTES + B_BYTES + (lw + k * LW) * 256;
      if constexpr (FMT == 1 || FMT == 4 || MX8) {
        dma4(src.s[k] + kt * src.ss[k], dst);
      } else if constexpr (FMT == 2) {
        // B scale words (ss 1): element kt*KE/128 of the row, rounded down to
        // an even element (4-byte aligned); group sums advance one float per
        // step (ss 4); dummies stay put (ss 0)
        const uint8_t* p = src.s[k] + kt * src.ss[k];
        if (src.ss[k] == 1) {
          const uintptr_t a = reinterpret_cast<uintptr_t>(src.s[k]) + ((kt * KE) / 128) * 2;
          p = reinterpret_cast<const uint8_t*>(a & ~static_cast<uintptr_t>(3));
        }
        dma4(p, dst);
      }
    }
  };
  auto issue = [&](const Src& src, int kt, int buf) { issue_part(src, kt, buf, 0, N_DMA); };
  // this copy wave's loads for a step have landed once at most `ahead`
  // later steps (N_DMA loads each) are still in flight
  auto wait_ahead = [&](int ahead) {
    if constexpr (STAGES >= 6) { if (ahead >= 4) { vm_wait<4 * N_DMA>(); return; } }
    if constexpr (STAGES >= 5) { if (ahead == 3) { vm_wait<3 * N_DMA>(); return; } }
    if constexpr (STAGES >= 4) { if (ahead == 2) { vm_wait<2 * N_DMA>(); return; } }
    if constexpr (STAGES >= 3) { if (ahead == 1) { vm_wait<N_DMA>(); return; } }
    vm_wait<0>();
  };

  // K steps are numbered across this workgroup's tiles, and step s of the
  // sequence lives in LDS buffer s % STAGES; `sb` is the buffer of a tile's
  // step 0.  STAGES-1 steps are loaded ahead: step s+STAGES-1 goes into the
  // buffer read in step s-1, issued once the barrier of step s shows every
  // wave is past it.  With copy waves the next tile's first STAGES-1 steps
  // are issued right after the barrier of the current tile's last step (their
  // buffers were read in earlier steps), so they load during that step and
  // the epilogue; without, each tile starts with a barrier and the math
  // waves load its first steps themselves.
  const int t0 = xcd * chunk + slot;
  Src cur;
  if constexpr (NP > 0) {
    if (!is_math) {
      // copy waves: one barrier per step, the same sequence as the math waves
      if (t0 < t_end) {
        int e, m0, n0;
        coords(t0, e, m0, n0);
        sources(e, m0, n0, cur, false);
#pragma unroll
        for (int q = 0; q < STAGES - 1; ++q)
          if (q < nk) issue(cur, q, q);
      }
      // the next tile's sources are computed in step kc; its row ids,
      // copied to this wave's LDS slot ahead of step STAGES-1's loads, have
      // landed by then: in-order completion, and the wait of step kt covers
      // every load issued before step kt+1 (all of them in the last step)
      const int kc = min(STAGES - 2, nk - 1);
      for (int t = t0, sb = 0; t < t_end; t += per_xcd, sb = (sb + nk) % STAGES) {
        const int tn = t + per_xcd;
        const bool next = tn < t_end;
        Src nxt;
        int en = 0, m0n = 0, n0n = 0;
        if (next) {
          coords(tn, en, m0n, n0n);
#pragma unroll
          for (int q = 0; q < BM / 64; ++q) dma4(g.sorted_ids + m0n + q * 64 + lane, lds_addr(&lds_sid[lw][q * 64]));
        }
        // Tiles of at most 32 steps (the second products here) run with
        // the next tile as one sequence of steps: step j of it is issued in
        // step j - (STAGES - 1), so the next tile's first steps load STAGES - 1
        // steps ahead like every other step, and the wait keeps them in
        // flight across the boundary (fp8 GEMM2 -2.4 %, prefill GEMM2 -2 %).
        // Longer tiles measured no gain, and tiles of fewer than 2 STAGES
        // steps may not have the next tile's sources ready in time: both
        // issue the next tile's first steps together in their last step.
        const bool flow = next && nk >= 2 * STAGES && nk <= 32;  // uniform
        for (int kt = 0; kt < nk; ++kt) {
          wait_ahead(flow ? STAGES - 2 : min(STAGES - 2, nk - 1 - kt));
          bar();
          if (next && kt == kc) sources(en, m0n, n0n, nxt, true);
          const int j = kt + STAGES - 1;
          if (j < nk) issue(cur, j, (sb + j) % STAGES);
          else if (flow) issue(nxt, j - nk, (sb + j) % STAGES);
          if (next && !flow && kt == nk - 1) {
#pragma unroll
            for (int q = 0; q < STAGES - 1; ++q)
              if (q < nk) issue(nxt, q, (sb + nk + q) % STAGES);
          }
        }
        if constexpr (FMT == 1 && GEMM1) {  // the two barriers of the requant epilogue
          bar();
          bar();
        }
        if (next) cur = nxt;
      }
      return;
    }
  }

  for (int t = t0, sb = 0; t < t_end; t += per_xcd, sb = (sb + nk) % STAGES) {
    int e, m0, n0;
    coords(t, e, m0, n0);
    if constexpr (NP == 0) {
      __syncthreads();  // the previous tile's buffers are no longer read
      sources(e, m0, n0, cur, false);
#pragma unroll
      for (int q = 0; q < STAGES - 1; ++q)
        if (q < nk) issue(cur, q, (sb + q) % STAGES);
    }

    // GEMM2: the ids of this lane's output rows, for the epilogue's pad-row
    // check, requested before the K loop (the math waves issue no other
    // global loads, so this one has landed long before it is used)
    int sid_ep[GEMM1 ? 1 : TM];
    if constexpr (!GEMM1) {
#pragma unroll
      for (int i = 0; i < TM; ++i) sid_ep[i] = g.sorted_ids[m0 + wm * WTM + i * 32 + l32];
    }
    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = f32x16{};
    float seff[TN];  // int4 GEMM1: the scale each column's accumulators are divided by (0: none yet)
#pragma unroll
    for (int j = 0; j < TN; ++j) seff[j] = 0.f;

    // B row (within the tile) of wave tile j
#define brow(j) (GEMM1 ? ((j) < TN / 2 ? wn * (WTN / 2) + (j) * 32 : NC + wn * (WTN / 2) + ((j) - TN / 2) * 32) \
                       : wn * WTN + (j) * 32)

    if constexpr (NP > 0 && FMT == 0) {
      // Math waves of a split bf16 launch: fragments are read one MFMA K
      // substep ahead into a double buffer.  The barrier for stage kt+1 sits
      // before the last substep's MFMAs of step kt (once this wave's reads of
      // stage kt are complete), so the next stage's first fragments load
      // while those MFMAs run; the barrier count is still one per step.
      constexpr int NKK = KE / 16;
      static_assert(NKK % 2 == 0, "substep parity");
      bf16x8 fa[2][TM], fb[2][TN];
      auto read_frags = [&](int kt, int kk, int buf) {
        const uint8_t* As = &smem[(sb + kt) % STAGES][0];
        const uint8_t* Bs = As + A_BYTES;
        const int ch = 2 * kk + kg;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int r = wm * WTM + i * 32 + l32;
          fa[buf][i] = as_bf16x8(ld16(As + r * KB + ((ch ^ swz<KB>(r)) << 4)));
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int r = brow(j) + l32;
          fb[buf][j] = as_bf16x8(ld16(Bs + r * BB + ((ch ^ swz<KB>(r)) << 4)));
        }
      };
      bar();  // stage 0 has landed
      read_frags(0, 0, 0);
      for (int kt = 0; kt < nk; ++kt) {
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
          if (kk + 1 < NKK) {
            read_frags(kt, kk + 1, (kk + 1) & 1);
          } else if (kt + 1 < nk) {
            __atomic_signal_fence(__ATOMIC_SEQ_CST);
            lds_wait();  // stage kt is in registers
            bar();                               // stage kt+1 has landed; buffer kt is free
            read_frags(kt + 1, 0, 0);
          }
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
              acc[i][j] = TRB ? mfma32x32x16(fb[kk & 1][j], fa[kk & 1][i], acc[i][j])
                              : mfma32x32x16(fa[kk & 1][i], fb[kk & 1][j], acc[i][j]);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    for (int kt = 0; kt < nk && !(NP > 0 && FMT == 0); ++kt) {
      if constexpr (NP == 0) wait_ahead(min(STAGES - 2, nk - 1 - kt));
      bar();  // every stage-kt copy of every copy wave has landed
      const bool pre = NP == 0 && kt + STAGES - 1 < nk;  // this wave starts a later stage
      if (FMT != 0 && pre) issue(cur, kt + STAGES - 1, (sb + kt + STAGES - 1) % STAGES);
      const uint8_t* As = &smem[(sb + kt) % STAGES][0];
      const uint8_t* Bs = As + A_BYTES;
      const uint8_t* Ss = Bs + B_BYTES;
      if constexpr (FMT == 0) {
        // every fragment of the K step is requested before the first MFMA
        constexpr int NKK = KE / 16;  // MFMA K substeps per step
        bf16x8 af[NKK][TM], bfr[NKK][TN];
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
          const int ch = 2 * kk + kg;
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            const int r = wm * WTM + i * 32 + l32;
            af[kk][i] = as_bf16x8(ld16(As + r * KB + ((ch ^ swz<KB>(r)) << 4)));
          }
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int r = brow(j) + l32;
            bfr[kk][j] = as_bf16x8(ld16(Bs + r * BB + ((ch ^ swz<KB>(r)) << 4)));
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        // the next stage's loads are issued between the MFMA groups, so the
        // matrix pipe keeps running while the address unit takes them
        constexpr int PER = (A_CH + B_CH + NKK - 1) / NKK;
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
              acc[i][j] = TRB ? mfma32x32x16(bfr[kk][j], af[kk][i], acc[i][j]) : mfma32x32x16(af[kk][i], bfr[kk][j], acc[i][j]);
          __builtin_amdgcn_sched_barrier(0);
          if (pre) issue_part(cur, kt + STAGES - 1, (sb + kt + STAGES - 1) % STAGES, kk * PER, min((kk + 1) * PER, A_CH + B_CH));
          __builtin_amdgcn_sched_barrier(0);
        }
      } else if constexpr (FMT == 1 && NP > 0) {
        // fp8 math waves of a split launch (two waves per SIMD, so at most 256
        // registers each): transposed product as below, but one 32x32 block
        // at a time -- its two K halves are MFMAs on one partial, and the
        // VALU folds the previous block's partial in between them -- with
        // the W fragments read per column block, one block ahead.
        i32x8 af[2][TM];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          const int c0 = 4 * kk + 2 * kg;
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            const int r = wm * WTM + i * 32 + l32;
            const i32x4 lo = __builtin_bit_cast(i32x4, ld16(As + r * KB + ((c0 ^ swz<KB>(r)) << 4)));
            const i32x4 hi = __builtin_bit_cast(i32x4, ld16(As + r * KB + (((c0 + 1) ^ swz<KB>(r)) << 4)));
            af[kk][i] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          }
        }
        i32x8 bq[2][2];  // [buffer][K half] of one column block
        auto read_b = [&](int j, int buf) {
          const int r = brow(j) + l32;
#pragma unroll
          for (int kk = 0; kk < 2; ++kk) {
            const int c0 = 4 * kk + 2 * kg;
            const i32x4 lo = __builtin_bit_cast(i32x4, ld16(Bs + r * BB + ((c0 ^ swz<KB>(r)) << 4)));
            const i32x4 hi = __builtin_bit_cast(i32x4, ld16(Bs + r * BB + (((c0 + 1) ^ swz<KB>(r)) << 4)));
            bq[buf][kk] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          }
        };
        read_b(0, 0);
        const float* sA = reinterpret_cast<const float*>(Ss);                    // [BM]
        const float* sB = reinterpret_cast<const float*>(Ss + (BM / 64) * 256);  // [64]
        float fa[TM], sb[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) fa[i] = sA[wm * WTM + i * 32 + l32];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int r = brow(j);
          sb[j] = GEMM1 ? sB[r < NC ? 0 : 1] : sB[(r / 128) % (BNW / 128)];
        }
        f32x16 part[2];
        // blocks column-major: b = j*TM + i
#pragma unroll
        for (int b = 0; b <= TM * TN; ++b) {
          const int i = b % TM, j = b / TM;
          const int ip = (b - 1) % TM, jp = (b - 1) / TM;  // the block folded in this iteration
          if (b < TM * TN && i == 0 && j + 1 < TN) read_b(j + 1, (j + 1) & 1);
          __builtin_amdgcn_sched_barrier(0);
          const float f = b > 0 ? fa[ip] * sb[jp] : 0.f;
          if (b < TM * TN) part[b & 1] = mfma32x32x64_fp8(bq[j & 1][0], af[0][i], f32x16{});
          if (b > 0) {
#pragma unroll
            for (int v = 0; v < 8; ++v) acc[ip][jp][v] = fmaf(part[(b - 1) & 1][v], f, acc[ip][jp][v]);
          }
          if (b < TM * TN) part[b & 1] = mfma32x32x64_fp8(bq[j & 1][1], af[1][i], part[b & 1]);
          if (b > 0) {
#pragma unroll
            for (int v = 8; v < 16; ++v) acc[ip][jp][v] = fmaf(part[(b - 1) & 1][v], f, acc[ip][jp][v]);
          }
          // keep the order written: each MFMA, then eight fmas that run on the
          // VALU while it executes (the compiler otherwise pairs the MFMAs and
          // stalls the fmas behind the second one)
          if (b > 0 && b < TM * TN) {
            __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);  // the scale product
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      } else if constexpr (FMT == 1) {
        // Transposed product: the MFMA's first operand is a 32-row block of
        // W (output columns n), the second a 32-row block of A (rows m), so
        // a lane's 16 values run down n for one row m.  Every value of a
        // lane then shares one A row scale and one W block scale: the K-block
        // rescale is one multiply per 32x32 block and one fma per value.
        i32x8 af[2][TM], bfr[2][TN];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          const int c0 = 4 * kk + 2 * kg;
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            const int r = wm * WTM + i * 32 + l32;
            const i32x4 lo = __builtin_bit_cast(i32x4, ld16(As + r * KB + ((c0 ^ swz<KB>(r)) << 4)));
            const i32x4 hi = __builtin_bit_cast(i32x4, ld16(As + r * KB + (((c0 + 1) ^ swz<KB>(r)) << 4)));
            af[kk][i] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          }
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int r = brow(j) + l32;
            const i32x4 lo = __builtin_bit_cast(i32x4, ld16(Bs + r * BB + ((c0 ^ swz<KB>(r)) << 4)));
            const i32x4 hi = __builtin_bit_cast(i32x4, ld16(Bs + r * BB + (((c0 + 1) ^ swz<KB>(r)) << 4)));
            bfr[kk][j] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          }
        }
        const float* sA = reinterpret_cast<const float*>(Ss);                    // [BM]
        const float* sB = reinterpret_cast<const float*>(Ss + (BM / 64) * 256);  // [64]
        float fa[TM], sb[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) fa[i] = sA[wm * WTM + i * 32 + l32];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int r = brow(j);
          sb[j] = GEMM1 ? sB[r < NC ? 0 : 1] : sB[(r / 128) % (BNW / 128)];
        }
        __builtin_amdgcn_sched_barrier(0);
        // Blocks in pairs: the two K halves of pair q go to the matrix pipe
        // (independent MFMAs back to back), then the VALU folds pair q-1 into
        // the accumulators while those run.  Four partial blocks are live.
        constexpr int NB = TM * TN;
        static_assert(NB % 2 == 0, "block pairs");
        f32x16 part[4];
#pragma unroll
        for (int q = 0; q <= NB / 2; ++q) {
          if (q < NB / 2) {
#pragma unroll
            for (int kk = 0; kk < 2; ++kk)
#pragma unroll
              for (int u = 0; u < 2; ++u) {
                const int bi = 2 * q + u, i = bi / TN, j = bi % TN;
                f32x16& pp = part[(q & 1) * 2 + u];
                pp = mfma32x32x64_fp8(bfr[kk][j], af[kk][i], kk == 0 ? f32x16{} : pp);
              }
          }
          if (q > 0) {
#pragma unroll
            for (int u = 0; u < 2; ++u) {
              const int bi = 2 * (q - 1) + u, i = bi / TN, j = bi % TN;
              const f32x16& pp = part[((q - 1) & 1) * 2 + u];
              const float f = fa[i] * sb[j];
#pragma unroll
              for (int v = 0; v < 16; ++v) acc[i][j][v] = fmaf(pp[v], f, acc[i][j][v]);
            }
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      } else if constexpr (GSUM) {
        // int4 GEMM1.  The codes enter the MFMA exactly, as bf16 136 + q, and
        // the group scale is applied in fp32: acc holds the tile's sum
        // divided by its column's current scale s, so each step first takes
        // acc * (s_prev / s) - 136 * (the row's sum over the group) and the
        // step's MFMAs then add sum(a * (136 + q)).  A zero scale keeps the
        // previous one and turns the group's codes into q = 0.
        constexpr int NKK = KE / 16, NBW = NKK / 4;
        const uint32_t* sW = reinterpret_cast<const uint32_t*>(Ss);  // one dword per tile row
        const float* sR = reinterpret_cast<const float*>(Ss + (BNW / 64) * 256);  // [BM] biased group sums
        float ratio[TN];
        uint32_t keep[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int r = brow(j) + l32;
          const int n_glob = r < NC ? n0 + r : g.I + n0 + (r - NC);
          // element index of the scale; only its parity (which half of the dword) is
          // used, so unsigned wrap-around for the largest weight tensors is harmless
          const unsigned idx = (static_cast<unsigned>(e) * 2u * g.I + n_glob) * (K / 128) + (kt * KE) / 128;
          const uint32_t d = sW[r];
          const float sc = __uint_as_float((idx & 1) ? (d & 0xFFFF0000u) : (d << 16));
          const bool z = sc == 0.f;
          const float se = z ? seff[j] : sc;
          ratio[j] = seff[j] == 0.f ? 0.f : seff[j] * __builtin_amdgcn_rcpf(se);  // 1-ulp reciprocal
          seff[j] = se;
          keep[j] = z ? 0u : ~0u;
        }
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int r0 = wm * WTM + i * 32 + 4 * kg;  // value v: row r0 + 8*(v/4) + v%4
          f32x16 rs;
#pragma unroll
          for (int b4 = 0; b4 < 4; ++b4) {
            const u32x4 q = ld16(sR + r0 + 8 * b4);
#pragma unroll
            for (int c = 0; c < 4; ++c) rs[4 * b4 + c] = __uint_as_float(q[c]);
          }
#pragma unroll
          for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = fmaf(acc[i][j][v], ratio[j], rs[v]);
        }
#pragma unroll
        for (int h = 0; h < NBW; ++h) {
          u32x4 bw[TN];
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int r = brow(j) + l32;
            bw[j] = ld16(Bs + r * BB + (((NBW * kg + h) ^ swz_b<BB>(r)) << 4));
          }
#pragma unroll
          for (int k4 = 0; k4 < 4; ++k4) {
            // substep kk of lane group kg covers K elements [(NKK*kg+kk)*8, +8) of the step
            const int kk = 4 * h + k4, ch = NKK * kg + kk;
            bf16x8 a[TM], b[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
              const int r = wm * WTM + i * 32 + l32;
              a[i] = as_bf16x8(ld16(As + r * KB + ((ch ^ swz<KB>(r)) << 4)));
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) b[j] = int4x8_biased_bf16(bw[j][k4], keep[j]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
              for (int j = 0; j < TN; ++j) acc[i][j] = mfma32x32x16(a[i], b[j], acc[i][j]);
          }
        }
      } else if constexpr (FMT == 2) {
        // int4 GEMM2: each code is decoded to bf16 q * s before the MFMA;
        // this lane's scales, then per 64-element half of the step its B words
        // (one word of eight nibbles per 16-wide K substep; a lane group
        // covers KE/2 elements of the step)
        constexpr int NKK = KE / 16, NBW = NKK / 4;
        const uint32_t* sW = reinterpret_cast<const uint32_t*>(Ss);  // one dword per tile row
        float sb[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int r = brow(j) + l32;
          const int n_glob = GEMM1 ? (r < NC ? n0 + r : g.I + n0 + (r - NC)) : n0 + r;
          const unsigned idx = (static_cast<unsigned>(e) * (GEMM1 ? 2 * g.I : g.H) + n_glob) * (K / 128) + (kt * KE) / 128;
          const uint32_t d = sW[r];
          sb[j] = __uint_as_float((idx & 1) ? (d & 0xFFFF0000u) : (d << 16));
        }
#pragma unroll
        for (int h = 0; h < NBW; ++h) {
          u32x4 bw[TN];
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int r = brow(j) + l32;
            bw[j] = ld16(Bs + r * BB + (((NBW * kg + h) ^ swz_b<BB>(r)) << 4));
          }
#pragma unroll
          for (int k4 = 0; k4 < 4; ++k4) {
            // substep kk of lane group kg covers K elements [(NKK*kg+kk)*8, +8) of the step
            const int kk = 4 * h + k4, ch = NKK * kg + kk;
            bf16x8 a[TM], b[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
              const int r = wm * WTM + i * 32 + l32;
              a[i] = as_bf16x8(ld16(As + r * KB + ((ch ^ swz<KB>(r)) << 4)));
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
              const uint32_t wd = k4 == 0 ? bw[j].x : (k4 == 1 ? bw[j].y : (k4 == 2 ? bw[j].z : bw[j].w));
              b[j] = dequant_int4x8(wd, sb[j]);
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
              for (int j = 0; j < TN; ++j) acc[i][j] = TRB ? mfma32x32x16(b[j], a[i], acc[i][j]) : mfma32x32x16(a[i], b[j], acc[i][j]);
          }
        }
      } else if constexpr (MX8) {
        // MXFP4 weights x MXFP8 activations, formed transposed like fp8 (the
        // weight fragment is the first operand).  MFMA kk of the step covers
        // K [64 kk, 64 kk + 64) in two 32-element scale blocks, and lane
        // group kg supplies block kg's E8M0 byte for both operands (byte
        // 2 (kk % 2) + kg of the row's dword kk / 2 for the step; the
        // instruction applies the scales itself, so the products accumulate
        // in place: no rescale on the VALU).  Weights: lane group kg holds
        // block kg, 16 bytes (chunk 2 kk + kg of the row's KE/2 bytes).
        // Activations: the e4m3 operand interleaves the blocks in 16-element
        // halves -- lane group kg holds elements [16 kg, +16) of block 0,
        // then of block 1, i.e. chunks 4 kk + kg and 4 kk + 2 + kg of the
        // row's KE bytes.
        const uint32_t* sA = reinterpret_cast<const uint32_t*>(Ss);                          // [MXD][BM]
        const uint32_t* sB = reinterpret_cast<const uint32_t*>(Ss + MXD * (BM / 64) * 256);  // [MXD][BNW]
        // per 128 K elements (one E8M0 dword per row): MFMAs 2 d and 2 d + 1
#pragma unroll
        for (int d = 0; d < MXD; ++d) {
          i32x8 af[2][TM], bq[2][TN];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int kk = 2 * d + h;
#pragma unroll
            for (int i = 0; i < TM; ++i) {
              const int r = wm * WTM + i * 32 + l32;
              const i32x4 lo = __builtin_bit_cast(i32x4, ld16(As + r * KB + (((4 * kk + kg) ^ swz<KB>(r)) << 4)));
              const i32x4 hi = __builtin_bit_cast(i32x4, ld16(As + r * KB + (((4 * kk + 2 + kg) ^ swz<KB>(r)) << 4)));
              af[h][i] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
              const int r = brow(j) + l32;
              const i32x4 q = __builtin_bit_cast(i32x4, ld16(Bs + r * BB + (((2 * kk + kg) ^ swz_b<BB>(r)) << 4)));
              bq[h][j] = __builtin_shufflevector(q, q, 0, 1, 2, 3, 0, 1, 2, 3);  // upper half unused
            }
          }
          int da[TM], db[TN];  // the row's dword d moved down by kg bytes: byte 2 h is block 2 h + kg
#pragma unroll
          for (int i = 0; i < TM; ++i) da[i] = static_cast<int>(sA[d * BM + wm * WTM + i * 32 + l32] >> (8 * kg));
#pragma unroll
          for (int j = 0; j < TN; ++j) db[j] = static_cast<int>(sB[d * BNW + brow(j) + l32] >> (8 * kg));
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = mfma32x32x64_f4f8<0>(bq[0][j], af[0][i], db[j], da[i], acc[i][j]);
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = mfma32x32x64_f4f8<2>(bq[1][j], af[1][i], db[j], da[i], acc[i][j]);
        }
      } else {  // MXFP4
        // lane group kg covers elements [64 kg, 64 kg + 64) of the step, the
        // 32-element blocks 2 kg and 2 kg + 1: their E8M0 bytes are bytes
        // 2 kg and 2 kg + 1 of the row's scale dword, passed as float(s << 23)
        constexpr int NKK = KE / 16, NBW = NKK / 4;
        static_assert(NBW == 2, "one 16-byte chunk per 32-element block");
        const uint32_t* sW = reinterpret_cast<const uint32_t*>(Ss);  // one dword per tile row
        float sc[TN][NBW];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const uint32_t d = sW[brow(j) + l32];
#pragma unroll
          for (int h = 0; h < NBW; ++h) sc[j][h] = __uint_as_float(((d >> (8 * (NBW * kg + h))) & 0xFFu) << 23);
        }
#pragma unroll
        for (int h = 0; h < NBW; ++h) {
          u32x4 bw[TN];
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int r = brow(j) + l32;
            bw[j] = ld16(Bs + r * BB + (((NBW * kg + h) ^ swz_b<BB>(r)) << 4));
          }
#pragma unroll
          for (int k4 = 0; k4 < 4; ++k4) {
            const int kk = 4 * h + k4, ch = NKK * kg + kk;
            bf16x8 a[TM], b[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
              const int r = wm * WTM + i * 32 + l32;
              a[i] = as_bf16x8(ld16(As + r * KB + ((ch ^ swz<KB>(r)) << 4)));
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
              const uint32_t wd = k4 == 0 ? bw[j].x : (k4 == 1 ? bw[j].y : (k4 == 2 ? bw[j].z : bw[j].w));
              b[j] = as_bf16x8(mxfp4x8_to_bf16(wd, sc[j][h]));
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
              for (int j = 0; j < TN; ++j) acc[i][j] = TRB ? mfma32x32x16(b[j], a[i], acc[i][j]) : mfma32x32x16(a[i], b[j], acc[i][j]);
          }
        }
      }
    }
#undef brow

    // ---- epilogue.  D element v of a 32x32 tile (bf16 / 4-bit GEMM1): row
    // 8*(v/4) + 4*kg + v%4, column l32.  fp8 and every GEMM2 form the product
    // transposed (W is the MFMA's first operand): lane (kg, l32) of row
    // block i holds row wm*WTM + i*32 + l32 at columns 8*(v/4) + 4*kg + v%4
    // of each column block, so four consecutive columns per store.
    if constexpr (GEMM1) {
      constexpr int TH = TN / 2;  // gate tiles (paired with up tile j + TH)
      if constexpr (GSUM) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] *= seff[j];
      }
      float av[TM][TH][16];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TH; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) av[i][j][v] = silu_mul(acc[i][j][v], acc[i][j + TH][v]);
      if constexpr (FMT == 1) {
        // transposed layout: lane (kg, l32) of row block i holds row
        // wm*WTM + i*32 + l32 at columns 8*(v/4) + 4*kg + v%4 of each gate
        // block.  Row amax over the tile's 128 columns: the lane's values,
        // the other k-group lane, then the WN waves (LDS).
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          float m = 0.f;
#pragma unroll
          for (int j = 0; j < TH; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) m = fmaxf(m, fabsf(av[i][j][v]));
          m = fmaxf(m, __shfl_xor(m, 32));
          if (kg == 0) lds_amax[wn][wm * WTM + i * 32 + l32] = m;
        }
        __syncthreads();
        uint8_t* q = static_cast<uint8_t*>(g.inter);
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int rl = wm * WTM + i * 32 + l32;
          float m = 0.f;
#pragma unroll
          for (int w = 0; w < WN; ++w) m = fmaxf(m, lds_amax[w][rl]);
          const float sc = fmaxf(m, 1e-10f) / 448.0f;
          const size_t row = static_cast<size_t>(m0 + rl);
          // a / sc as one IEEE reciprocal per row and a residual step per
          // value: q0 = a r, then q0 + (a - q0 sc) r, the residual exact by
          // fma, the sign restored for a = -0.  On the fp8 workload its codes
          // equal those of the IEEE quotient for all 134M intermediate values
          // (GEMM1 0.7 % faster than a divide per value).
          const float r = 1.0f / sc;
          auto qdiv = [&](float a) {
            const float q0 = a * r;
            return sat_e4m3(__builtin_copysignf(fmaf(fmaf(-q0, sc, a), r, q0), a));
          };
#pragma unroll
          for (int j = 0; j < TH; ++j)
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4) {
              const int col = n0 + wn * (WTN / 2) + j * 32 + 8 * v4 + 4 * kg;
              const float* a4 = &av[i][j][4 * v4];
              const uint32_t codes = f32x2_to_e4m3(qdiv(a4[0]), qdiv(a4[1])) |
                                     (f32x2_to_e4m3(qdiv(a4[2]), qdiv(a4[3])) << 16);
              *reinterpret_cast<uint32_t*>(q + row * g.I + col) = codes;
            }
          if (wn == 0 && kg == 0) g.inter_scale[row * (g.I / 128) + n0 / 128] = sc;
        }
        __syncthreads();  // lds_amax is reused by the next tile
      } else if constexpr (MX8) {
        // transposed layout as fp8; the OCP MX block is one 32-column gate
        // block j of the row: amax over the lane's 16 values and the other
        // k-group lane's, then the E8M0 byte and the exact power-of-two scaling
        uint8_t* q = static_cast<uint8_t*>(g.inter);
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const size_t row = static_cast<size_t>(m0 + wm * WTM + i * 32 + l32);
#pragma unroll
          for (int j = 0; j < TH; ++j) {
            float m = 0.f;
#pragma unroll
            for (int v = 0; v < 16; ++v) m = fmaxf(m, fabsf(av[i][j][v]));
            m = fmaxf(m, __shfl_xor(m, 32));
            const uint32_t byte = mx_e8m0_of_amax(m);
            const float mul = __uint_as_float((254u - byte) << 23);
            const int cb = n0 + wn * (WTN / 2) + j * 32;  // the block's first column
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4) {
              const float* a4 = &av[i][j][4 * v4];
              const uint32_t codes = f32x2_to_e4m3(sat_e4m3(a4[0] * mul), sat_e4m3(a4[1] * mul)) |
                                     (f32x2_to_e4m3(sat_e4m3(a4[2] * mul), sat_e4m3(a4[3] * mul)) << 16);
              *reinterpret_cast<uint32_t*>(q + row * g.I + cb + 8 * v4 + 4 * kg) = codes;
            }
            if (kg == 0) g.inter_mx[row * (g.I / 32) + cb / 32] = static_cast<uint8_t>(byte);
          }
        }
      } else {
        uint16_t* o = static_cast<uint16_t*>(g.inter);
        auto store = [&](bool masked) {
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TH; ++j)
#pragma unroll
              for (int v = 0; v < 16; ++v) {
                const int row = m0 + wm * WTM + i * 32 + 8 * (v >> 2) + 4 * kg + (v & 3);
                const int col = n0 + wn * (WTN / 2) + j * 32 + l32;
                if (!masked || col < g.I) o[static_cast<size_t>(row) * g.I + col] = f32_to_bf16(av[i][j][v]);
              }
        };
        if (n0 + NC <= g.I) store(false);  // uniform: only a ragged last column tile masks
        else store(true);
      }
    } else if constexpr (A8) {
      // transposed layout: a lane holds four consecutive output columns per
      // group and the lane 32 away the next four of the same row, so one
      // exchange makes eight consecutive columns per 16-byte store (half the
      // store instructions of 8-byte stores: GEMM2 of the fp8 workload
      // 1608 -> 1502 us)
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int row = m0 + wm * WTM + i * 32 + l32;
        if (sid_ep[i] >= g.n_routed) continue;  // pad rows are never read
        uint16_t* yr = static_cast<uint16_t*>(g.y) + static_cast<size_t>(row) * g.H;
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int p = 0; p < 2; ++p) {
            // groups 2p and 2p+1 (columns 16p + [0,16) of the block): lane kg
            // keeps its own four columns of group 2p+kg and takes the other
            // lane's four of that group, then stores eight columns at once
            const f32x16& c = acc[i][j];
            const int ga = 2 * p, gb = 2 * p + 1;
            const uint32_t a0 = pack_bf16x2(c[4 * ga], c[4 * ga + 1]), a1 = pack_bf16x2(c[4 * ga + 2], c[4 * ga + 3]);
            const uint32_t b0 = pack_bf16x2(c[4 * gb], c[4 * gb + 1]), b1 = pack_bf16x2(c[4 * gb + 2], c[4 * gb + 3]);
            const uint32_t s0 = kg ? a0 : b0, s1 = kg ? a1 : b1;
            const uint32_t r0 = __shfl_xor(s0, 32), r1 = __shfl_xor(s1, 32);
            const u32x4 o = kg ? u32x4{r0, r1, b0, b1} : u32x4{a0, a1, r0, r1};
            const int col = n0 + wn * WTN + j * 32 + 16 * p + 8 * kg;
            *reinterpret_cast<u32x4*>(yr + col) = o;
          }
      }
    } else {
      // transposed layout, fp32 y: four consecutive output columns per 16-byte store
      static_assert(TRB && y_is_f32(FMT), "bf16 and int4 routes keep y in fp32");
      const bool masked = n0 + NC > g.H;  // uniform: only a ragged last column tile masks
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int row = m0 + wm * WTM + i * 32 + l32;
        if (sid_ep[i] >= g.n_routed) continue;  // pad rows are never read
        float* yr = static_cast<float*>(g.y) + static_cast<size_t>(row) * g.H;
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int v4 = 0; v4 < 4; ++v4) {
            const int col = n0 + wn * WTN + j * 32 + 8 * v4 + 4 * kg;
            const f32x16& c = acc[i][j];
            if (!masked || col < g.H)  // four columns, all in or all out (H % 4 == 0)
              *reinterpret_cast<f32x4*>(yr + col) = f32x4{c[4 * v4], c[4 * v4 + 1], c[4 * v4 + 2], c[4 * v4 + 3]};
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

template <class Kernel>
int occupancy_per_cu(Kernel k, int threads) {
  int per_cu = 1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, threads, 0) != hipSuccess || per_cu < 1)
    per_cu = 1;
  return per_cu;
}

// Persistent grid: as many workgroups as fit on the device at once (per_cu
// per CU, a multiple of the XCD count), never more than the largest possible
// number of tiles.
dim3 persistent_grid(int per_cu, long max_tiles) {
  long n = static_cast<long>(cu_count()) * per_cu;
  n = (n + kXcds - 1) / kXcds * kXcds;
  const long cap = (max_tiles + kXcds - 1) / kXcds * kXcds;
  return dim3(static_cast<unsigned>(std::max<long>(kXcds, std::min(n, cap))));
}

template <int FMT, bool GEMM1, int BM, int BNW, int WM, int WN, int GM, int KBT = 128, int STAGES = 3, int NP = 0>
hipError_t launch_tiled(const GroupedGemm& g, hipStream_t s) {
  constexpr int NC = GEMM1 ? BNW / 2 : BNW;
  constexpr int NT = (WM * WN + NP) * 64;
  // only bf16 handles a ragged last K step; every other format's steps must
  // tile K exactly (a step past K would read beyond its rows)
  constexpr int KE = (FMT == 1 || FMT == 5) ? KBT : KBT / 2;
  if (FMT != 0 && (GEMM1 ? g.H : g.I) % KE != 0) return hipErrorInvalidValue;
  const long mt = g.max_rows / BM, nt = ((GEMM1 ? g.I : g.H) + NC - 1) / NC;
  auto kern = moe_gemm_tiled<FMT, GEMM1, BM, BNW, WM, WN, GM, KBT, STAGES, NP>;
  // workgroups per CU depend on the kernel's registers and LDS only: queried
  // once per instantiation (thread-safe static initialisation)
  static const int per_cu = occupancy_per_cu(kern, NT);
  hipLaunchKernelGGL(kern, persistent_grid(per_cu, mt * nt), dim3(NT), 0, s, g);
  return hipGetLastError();
}

}  // namespace

// bf16 tile shapes: rows x weight rows per workgroup, waves as WM x WN.
#ifndef MOE_T1_BNW
#define MOE_T1_BNW 256
#define MOE_T1_WM 2
#define MOE_T1_WN 2
#endif
#ifndef MOE_T2_BNW
#define MOE_T2_BNW 256
#define MOE_T2_WM 2
#define MOE_T2_WN 2
#endif
#ifndef MOE_TBF_BM
#define MOE_TBF_BM 128
#endif
#ifndef MOE_TBF_KB
#define MOE_TBF_KB 128
#endif
#ifndef MOE_TBF_STAGES
#define MOE_TBF_STAGES 3
#endif
// Copy waves beside the math waves (0: the math waves copy).  Every tiled
// launch uses four; the 64-row int4 kernels are held to 128 registers so two
// workgroups of eight waves still fit per CU.
#ifndef MOE_TBF_NP1
#define MOE_TBF_NP1 4
#endif
#ifndef MOE_TBF_NP2
#define MOE_TBF_NP2 4
#endif
#ifndef MOE_TI4_NP1
#define MOE_TI4_NP1 4
#endif
#ifndef MOE_TI4_NP2
#define MOE_TI4_NP2 4
#endif
// most row tiles of one expert swept together per column tile
#ifndef MOE_TGM
#define MOE_TGM 8
#endif
#ifndef MOE_TGM_INT4
#define MOE_TGM_INT4 16
#endif
int bf16_tiled_block_m() { return MOE_TBF_BM; }
hipError_t launch_gemm1_bf16_tiled(const GroupedGemm& g, hipStream_t s) {
  return launch_tiled<0, true, MOE_TBF_BM, MOE_T1_BNW, MOE_T1_WM, MOE_T1_WN, MOE_TGM, MOE_TBF_KB, MOE_TBF_STAGES, MOE_TBF_NP1>(g, s);
}
hipError_t launch_gemm2_bf16_tiled(const GroupedGemm& g, hipStream_t s) {
  if (g.H % MOE_T2_BNW) return launch_tiled<0, false, MOE_TBF_BM, 128, MOE_T2_WM, MOE_T2_WN, MOE_TGM, MOE_TBF_KB, MOE_TBF_STAGES, MOE_TBF_NP2>(g, s);
  return launch_tiled<0, false, MOE_TBF_BM, MOE_T2_BNW, MOE_T2_WM, MOE_T2_WN, MOE_TGM, MOE_TBF_KB, MOE_TBF_STAGES, MOE_TBF_NP2>(g, s);
}

// fp8 over the 128 x 256 tile: with copy waves (NP > 0) four math waves
// (2 x 2), else eight (MOE_F8_WM x MOE_F8_WN) that copy for themselves
#ifndef MOE_F8_WM
#define MOE_F8_WM 2
#define MOE_F8_WN 4
#endif
#ifndef MOE_F8_NP1
#define MOE_F8_NP1 4
#endif
#ifndef MOE_F8_NP2
#define MOE_F8_NP2 4
#endif
int gemm_block_m_fp8(int, int, int) { return 128; }
template <bool GEMM1, int BNW, int NP>
hipError_t launch_fp8(const GroupedGemm& g, hipStream_t s) {
  if constexpr (NP > 0) return launch_tiled<1, GEMM1, 128, BNW, 2, 2, MOE_TGM, 128, 3, NP>(g, s);
  else return launch_tiled<1, GEMM1, 128, BNW, MOE_F8_WM, MOE_F8_WN, MOE_TGM>(g, s);
}
hipError_t launch_gemm1_fp8(const GroupedGemm& g, hipStream_t s) {
  return launch_fp8<true, 256, MOE_F8_NP1>(g, s);
}
hipError_t launch_gemm2_fp8(const GroupedGemm& g, hipStream_t s) {
  if (g.H % 256) return launch_fp8<false, 128, MOE_F8_NP2>(g, s);
  return launch_fp8<false, 256, MOE_F8_NP2>(g, s);
}

// int4 row tile: one math wave per 64 columns covers all MOE_TI4_BM rows, so
// each decoded weight fragment feeds MOE_TI4_BM / 32 MFMAs
#ifndef MOE_TI4_BM
#define MOE_TI4_BM 64
#endif
// 128 K elements per step: 64 bytes of each int4 weight row (half a cache
// line, where 64 elements took a quarter), 256 bytes of each activation row;
// two stages keep two workgroups per CU
#ifndef MOE_TI4_KB
#define MOE_TI4_KB 256
#define MOE_TI4_STAGES 2
#endif
int gemm_block_m_int4(int, int, int) { return MOE_TI4_BM; }
hipError_t launch_gemm1_int4(const GroupedGemm& g, hipStream_t s) {
  return launch_tiled<2, true, MOE_TI4_BM, 256, 1, 4, MOE_TGM_INT4, MOE_TI4_KB, MOE_TI4_STAGES, MOE_TI4_NP1>(g, s);
}
// MXFP4 weights (same 4-bit packing as int4, E8M0 scales per 32)
#ifndef MOE_TMX_BM
#define MOE_TMX_BM 128
#endif
int gemm_block_m_mxfp4() { return MOE_TMX_BM; }
hipError_t launch_gemm1_mxfp4_tiled(const GroupedGemm& g, hipStream_t s) {
  if constexpr (MOE_TMX_BM == 64)
    return launch_tiled<4, true, 64, 256, 1, 4, MOE_TGM_INT4, MOE_TI4_KB, MOE_TI4_STAGES, MOE_TI4_NP1>(g, s);
  else
    return launch_tiled<4, true, 128, 256, 2, 2, MOE_TGM, 256, 3, 4>(g, s);
}
hipError_t launch_gemm2_mxfp4_tiled(const GroupedGemm& g, hipStream_t s) {
  if constexpr (MOE_TMX_BM == 64) {
    if (g.H % 256) return launch_tiled<4, false, 64, 128, 1, 4, MOE_TGM_INT4, MOE_TI4_KB, MOE_TI4_STAGES, MOE_TI4_NP2>(g, s);
    return launch_tiled<4, false, 64, 256, 1, 4, MOE_TGM_INT4, MOE_TI4_KB, MOE_TI4_STAGES, MOE_TI4_NP2>(g, s);
  } else {
    if (g.H % 256) return launch_tiled<4, false, 128, 128, 2, 2, MOE_TGM, 256, 3, 4>(g, s);
    return launch_tiled<4, false, 128, 256, 2, 2, MOE_TGM, 256, 3, 4>(g, s);
  }
}
// MXFP4 weights x MXFP8 activations: the fp8 tile (128 x 256, four math
// waves beside four copy waves).  When K is a multiple of 256, 256-element K
// steps, so each weight row gives a whole 128-byte line per step (256 bytes
// of each activation row, two E8M0 dwords per row of either), two stages;
// otherwise (K a multiple of 128) 128-element steps (half a line of each
// weight row) with four stages.  A step never reaches past K.
template <bool GEMM1, int BNW>
hipError_t launch_mx8(const GroupedGemm& g, hipStream_t s) {
  const int K = GEMM1 ? g.H : g.I;
  if (K % 256 == 0) return launch_tiled<5, GEMM1, 128, BNW, 2, 2, MOE_TGM, 256, 2, 4>(g, s);
  return launch_tiled<5, GEMM1, 128, BNW, 2, 2, MOE_TGM, 128, 4, 4>(g, s);
}
hipError_t launch_gemm1_mx8(const GroupedGemm& g, hipStream_t s) { return launch_mx8<true, 256>(g, s); }
hipError_t launch_gemm2_mx8(const GroupedGemm& g, hipStream_t s) {
  if (g.H % 256) return launch_mx8<false, 128>(g, s);
  return launch_mx8<false, 256>(g, s);
}
hipError_t launch_gemm2_int4(const GroupedGemm& g, hipStream_t s) {
  if (g.H % 256) return launch_tiled<2, false, MOE_TI4_BM, 128, 1, 4, MOE_TGM_INT4, MOE_TI4_KB, MOE_TI4_STAGES, MOE_TI4_NP2>(g, s);
  return launch_tiled<2, false, MOE_TI4_BM, 256, 1, 4, MOE_TGM_INT4, MOE_TI4_KB, MOE_TI4_STAGES, MOE_TI4_NP2>(g, s);
}

}  // namespace moe
