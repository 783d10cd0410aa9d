// Internal launchers of the MoE kernels (host side).  Shapes are validated by
// the C ABI layer (moe_api.hip) before any of these is called.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace moe {

hipError_t launch_gate_topk(const float* logits, const float* bias, int T, int E, int k, int mode,
                            int renorm, float scale, int32_t* ids, float* w, int32_t* ids2,
                            float* w2, hipStream_t s);

// Router GEMM (bf16 hidden [T,H] x w_router [E,H]^T, fp32) then the gate
// selection; logits_out (fp32 [T,E]) optional.  H % 128 == 0.  ws holds the
// K-slice partial logits: router_workspace_bytes(T, H, E) bytes.
size_t router_workspace_bytes(int T, int H, int E);
hipError_t launch_router_gate(const uint16_t* hidden, const uint16_t* wr, int T, int H, int E, int k, int mode,
                              int renorm, float scale, const float* bias, float* logits_out, int32_t* ids,
                              float* w, int32_t* ids2, float* w2, void* ws, hipStream_t s);

int permute_chunk(int E);
size_t permute_workspace_bytes(int T, int k, int E);
hipError_t launch_permute(const int32_t* ids, int T, int k, int E, int block_m, int32_t* offsets,
                          int32_t* sorted_ids, int32_t* inv_pos, int cap, void* ws,
                          hipStream_t s);

// y: [cap, H] rows in sorted order, fp32 (y_f32) or bf16.
hipError_t launch_combine(const void* y, bool y_f32, const float* w, const int32_t* inv_pos, int T,
                          int H, int k, bool out_bf16, void* out, hipStream_t s);

hipError_t launch_act_quant(const uint16_t* x, int M, int K, uint8_t* q, float* s, hipStream_t st);
// OCP MX e4m3 per (row, 32 columns): codes q [M,K] and E8M0 bytes sx [M,K/32]
hipError_t launch_act_quant_mx(const uint16_t* x, int M, int K, uint8_t* q, uint8_t* sx, hipStream_t st);
// out[m][g] = -136 * sum of x[m][128g, 128g + 128) in fp32 (int4 GEMM1's bias term)
hipError_t launch_group_sum(const uint16_t* x, int M, int K, float* out, hipStream_t st);

// Grouped expert GEMMs.  Rows are the permuted routed rows (sorted order),
// grouped by expert in segments padded to a multiple of the kernel's row tile;
// `offsets` is the permute's expert_offsets[E+1], `max_rows` the capacity.
struct GroupedGemm {
  // first product: A rows are hidden[sorted_ids[p] / top_k] (pads read row 0)
  const void* x;              // bf16 hidden [T,H] (fp8, MXFP8: e4m3 codes [T,H])
  const float* x_scale;       // fp8 only: [T, H/128]
  const uint8_t* x_mx;        // MXFP8 only: E8M0 bytes [T, H/32]
  const float* x_gsum;        // int4 only: [T, H/128], -136 * the sum of each 128-group of a hidden row
  const int32_t* sorted_ids;  // [cap]
  const int32_t* offsets;     // [E+1]
  int T, H, E, I, top_k, n_routed, max_rows;
  const void* w1;             // [E, 2I, H] in storage format
  const void* w1_scale;
  const void* w2;             // [E, H, I]
  const void* w2_scale;
  void* inter;                // [cap, I] bf16 (fp8, MXFP8: e4m3 codes)
  float* inter_scale;         // fp8 only: [cap, I/128]
  uint8_t* inter_mx;          // MXFP8 only: E8M0 bytes [cap, I/32]
  void* y;                    // [cap, H]: fp32 for bf16 weights, bf16 otherwise
};

// y is kept in fp32 for bf16-activation routes (a bf16 rounding of every
// routed row would take most of the bf16 2e-2 output tolerance) and in bf16
// for the fp8-activation ones (fp8, MXFP4 x MXFP8), whose 1.9 GB fp32 round
// trip at 8192 tokens would cost more than the error budget it buys back.
__host__ __device__ constexpr bool y_is_f32(int wfmt) { return wfmt != 1 && wfmt != 5; }

// Row tile (padding granule) the kernels for this format/shape use.
int gemm_block_m(int wfmt, int T, int top_k, int E, int H, int I);
// int4 weights on the 16-row streamed kernels, which need no group sums of x
bool int4_decode(int T, int top_k, int E, int H, int I);
int bf16_tiled_block_m();
hipError_t launch_gemm1_bf16_tiled(const GroupedGemm& g, hipStream_t s);
hipError_t launch_gemm2_bf16_tiled(const GroupedGemm& g, hipStream_t s);
hipError_t launch_gemm1(int wfmt, const GroupedGemm& g, hipStream_t s);  // + SiLU*up epilogue
hipError_t launch_gemm2(int wfmt, const GroupedGemm& g, hipStream_t s);

}  // namespace moe
