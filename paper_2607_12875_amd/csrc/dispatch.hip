// Per-format dispatch of the grouped expert GEMMs.
#include "launch.hpp"

namespace moe {

int gemm_block_m_bf16(int T, int top_k, int E, int H, int I);
hipError_t launch_gemm1_bf16(const GroupedGemm& g, hipStream_t s);
hipError_t launch_gemm2_bf16(const GroupedGemm& g, hipStream_t s);
int gemm_block_m_fp8(int T, int top_k, int E);
hipError_t launch_gemm1_fp8(const GroupedGemm& g, hipStream_t s);
hipError_t launch_gemm2_fp8(const GroupedGemm& g, hipStream_t s);
int gemm_block_m_int4(int T, int top_k, int E);
hipError_t launch_gemm1_int4(const GroupedGemm& g, hipStream_t s);
hipError_t launch_gemm2_int4(const GroupedGemm& g, hipStream_t s);
hipError_t launch_gemm1_w8a16(const GroupedGemm& g, hipStream_t s);
hipError_t launch_gemm1_w4a16(const GroupedGemm& g, hipStream_t s);
hipError_t launch_gemm2_w4a16(const GroupedGemm& g, hipStream_t s);
hipError_t launch_gemm2_w8a16(const GroupedGemm& g, hipStream_t s);
int gemm_block_m_mxfp4();
hipError_t launch_gemm1_mxfp4_tiled(const GroupedGemm& g, hipStream_t s);
hipError_t launch_gemm2_mxfp4_tiled(const GroupedGemm& g, hipStream_t s);
hipError_t launch_gemm1_mx8(const GroupedGemm& g, hipStream_t s);
hipError_t launch_gemm2_mx8(const GroupedGemm& g, hipStream_t s);
bool int4_stream_fits(int H, int I);
hipError_t launch_gemm1_int4_stream(const GroupedGemm& g, hipStream_t s);
hipError_t launch_gemm2_int4_stream(const GroupedGemm& g, hipStream_t s);

// MXFP4 takes the 16-row decode kernels up to 32 routed rows per expert on
// average, the tiled kernels above (the row tile is the permute's padding)
static bool mxfp4_decode(int T, int top_k, int E) { return static_cast<long>(T) * top_k <= 32L * E; }
// int4 takes the 16-row streamed kernels up to MOE_I4_DECODE_ROWS routed rows
// per expert on average (where both products' K fit them), the 64-row tiled
// kernels above
#ifndef MOE_I4_DECODE_ROWS
#define MOE_I4_DECODE_ROWS 8
#endif
bool int4_decode(int T, int top_k, int E, int H, int I) {
  return static_cast<long>(T) * top_k <= static_cast<long>(MOE_I4_DECODE_ROWS) * E && int4_stream_fits(H, I);
}

int gemm_block_m(int wfmt, int T, int top_k, int E, int H, int I) {
  switch (wfmt) {
    case 1: return gemm_block_m_fp8(T, top_k, E);
    case 2: return int4_decode(T, top_k, E, H, I) ? 16 : gemm_block_m_int4(T, top_k, E);
    case 3: return 16;  // the weight-only fp8 route runs the 16-row decode kernels only
    case 4: return mxfp4_decode(T, top_k, E) ? 16 : gemm_block_m_mxfp4();
    case 5: return 128;  // MXFP4 x MXFP8: the tiled kernels at every batch size
    default: return gemm_block_m_bf16(T, top_k, E, H, I);
  }
}

hipError_t launch_gemm1(int wfmt, const GroupedGemm& g, hipStream_t s) {
  switch (wfmt) {
    case 1: return launch_gemm1_fp8(g, s);
    case 2: return int4_decode(g.T, g.top_k, g.E, g.H, g.I) ? launch_gemm1_int4_stream(g, s) : launch_gemm1_int4(g, s);
    case 3: return launch_gemm1_w8a16(g, s);
    case 4: return mxfp4_decode(g.T, g.top_k, g.E) ? launch_gemm1_w4a16(g, s) : launch_gemm1_mxfp4_tiled(g, s);
    case 5: return launch_gemm1_mx8(g, s);
    default: return launch_gemm1_bf16(g, s);
  }
}

hipError_t launch_gemm2(int wfmt, const GroupedGemm& g, hipStream_t s) {
  switch (wfmt) {
    case 1: return launch_gemm2_fp8(g, s);
    case 2: return int4_decode(g.T, g.top_k, g.E, g.H, g.I) ? launch_gemm2_int4_stream(g, s) : launch_gemm2_int4(g, s);
    case 3: return launch_gemm2_w8a16(g, s);
    case 4: return mxfp4_decode(g.T, g.top_k, g.E) ? launch_gemm2_w4a16(g, s) : launch_gemm2_mxfp4_tiled(g, s);
    case 5: return launch_gemm2_mx8(g, s);
    default: return launch_gemm2_bf16(g, s);
  }
}

}  // namespace moe
