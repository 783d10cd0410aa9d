// Host-side driver of the C ABI (include/moe.h) for the sanitizer build:
// every entry point's argument validation, the workspace size and layout
// functions over many shapes and formats, and the T == 0 no-ops.  Built with
// the host code of every source under AddressSanitizer and
// UndefinedBehaviorSanitizer; no GPU is needed (nothing here reaches a launch
// except calls that then report MOE_ERR_HIP without a device).
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "moe.h"

static int fails = 0;
#define EXPECT(cond)                                                   \
  do {                                                                 \
    if (!(cond)) {                                                     \
      fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__, __LINE__, #cond); \
      ++fails;                                                         \
    }                                                                  \
  } while (0)

static void* const FAKE = reinterpret_cast<void*>(0x10000);  // aligned, never dereferenced

static moe_args make(int T, int H, int E, int I, int k, int wfmt) {
  moe_args a;
  memset(&a, 0, sizeof a);
  a.T = T; a.H = H; a.E = E; a.I = I; a.top_k = k;
  a.score_mode = MOE_SCORE_SOFTMAX; a.renormalize = 1; a.routed_scale = 1.f;
  a.wfmt = wfmt; a.ofmt = MOE_OUT_F32;
  a.hidden = static_cast<const uint16_t*>(FAKE); a.logits = static_cast<const float*>(FAKE);
  a.w1 = FAKE; a.w2 = FAKE; a.out = FAKE;
  if (wfmt != MOE_W_BF16) { a.w1_scale = FAKE; a.w2_scale = FAKE; }
  return a;
}

int main() {
  for (int s = 0; s <= 7; ++s) EXPECT(moe_status_str(s) != nullptr && strlen(moe_status_str(s)) > 0);
  EXPECT(moe_permute_capacity(10, 2, 8, 16) == 10 * 2 + 8 * 15);
  EXPECT(moe_permute_capacity(-1, 2, 8, 16) == 0);
  EXPECT(moe_permute_workspace_bytes(100000, 8, 256) > 0);
  EXPECT(moe_router_workspace_bytes(16, 4096, 64) > 0);
  EXPECT(moe_router_workspace_bytes(16, 100, 64) == 0);

  // workspace sizes and layouts: every format, decode and prefill batches,
  // odd expert counts, the ABI limits, bf16 shapes that are multiples of 8
  const int fmts[] = {MOE_W_BF16, MOE_W_FP8E4M3_B128, MOE_W_INT4_G128, MOE_W_FP8E4M3_B128_A16,
                      MOE_W_MXFP4_A16, MOE_W_MXFP4_MXFP8};
  const int shapes[][5] = {{0, 256, 8, 128, 2},     {1, 128, 1, 128, 1},   {16, 4096, 64, 1408, 6},
                           {4096, 4096, 64, 1408, 6}, {77, 384, 300, 256, 8}, {20, 256, 1024, 128, 32},
                           {8, 65536, 4, 256, 2}};
  for (int f : fmts)
    for (const auto& sh : shapes) {
      moe_args a = make(sh[0], sh[1], sh[2], sh[3], sh[4], f);
      const size_t n = moe_workspace_bytes(&a);
      moe_ws_layout L;
      EXPECT(moe_workspace_layout(&a, &L) == MOE_OK);
      EXPECT(n == static_cast<size_t>(L.total));
      EXPECT(L.block_m >= 1 && L.cap >= sh[0] * sh[4]);
      EXPECT(L.sorted_ids >= 0 && L.y >= 0 && L.y < L.total);
      a.w_router = static_cast<const uint16_t*>(FAKE);
      EXPECT(moe_workspace_layout(&a, &L) == MOE_OK && L.router_ws >= 0);
    }
  {
    moe_args a = make(300, 392, 6, 200, 2, MOE_W_BF16);  // bf16, multiples of 8
    EXPECT(moe_workspace_bytes(&a) > 0);
    a.wfmt = MOE_W_FP8E4M3_B128;
    EXPECT(moe_workspace_bytes(&a) == 0);
  }

  // validation: each error before any launch
  moe_args a = make(64, 256, 8, 128, 2, MOE_W_BF16);
  const size_t BIG = static_cast<size_t>(1) << 40;
  EXPECT(moe_forward(nullptr, FAKE, BIG, nullptr) == MOE_ERR_NULL);
  { moe_args b = a; b.top_k = 9; EXPECT(moe_forward(&b, FAKE, BIG, nullptr) == MOE_ERR_SHAPE); }
  { moe_args b = a; b.H = 196; EXPECT(moe_forward(&b, FAKE, BIG, nullptr) == MOE_ERR_SHAPE); }
  { moe_args b = a; b.E = 2000; EXPECT(moe_forward(&b, FAKE, BIG, nullptr) == MOE_ERR_SHAPE); }
  { moe_args b = a; b.wfmt = 17; EXPECT(moe_forward(&b, FAKE, BIG, nullptr) == MOE_ERR_UNSUPPORTED); }
  { moe_args b = a; b.score_mode = 5; EXPECT(moe_forward(&b, FAKE, BIG, nullptr) == MOE_ERR_UNSUPPORTED); }
  { moe_args b = a; b.hidden = nullptr; EXPECT(moe_forward(&b, FAKE, BIG, nullptr) == MOE_ERR_NULL); }
  { moe_args b = a; b.out = reinterpret_cast<char*>(FAKE) + 4; EXPECT(moe_forward(&b, FAKE, BIG, nullptr) == MOE_ERR_ALIGN); }
  { moe_args b = a; EXPECT(moe_forward(&b, FAKE, 16, nullptr) == MOE_ERR_WORKSPACE); }
  { moe_args b = a; b.wfmt = MOE_W_INT4_G128; b.w1_scale = nullptr; EXPECT(moe_forward(&b, FAKE, BIG, nullptr) == MOE_ERR_NULL); }
  { moe_args b = a; b.T = 0; EXPECT(moe_forward(&b, nullptr, 0, nullptr) == MOE_OK); }
  { moe_args b = a; b.T = 0; EXPECT(moe_forward_static_ws(&b, nullptr) == MOE_OK); }
  { moe_args b = make(4096, 4096, 64, 1408, 6, MOE_W_BF16); EXPECT(moe_forward_static_ws(&b, nullptr) == MOE_ERR_WORKSPACE); }
  EXPECT(moe_forward_profiled(&a, FAKE, BIG, nullptr, nullptr) == MOE_ERR_NULL);
  EXPECT(moe_gate_topk(static_cast<const float*>(FAKE), nullptr, 4, 8, 9, 0, 1, 1.f, static_cast<int32_t*>(FAKE),
                       static_cast<float*>(FAKE), nullptr) == MOE_ERR_SHAPE);
  EXPECT(moe_gate_topk(nullptr, nullptr, 0, 8, 2, 0, 1, 1.f, nullptr, nullptr, nullptr) == MOE_OK);
  EXPECT(moe_router_gate_topk(static_cast<const uint16_t*>(FAKE), static_cast<const uint16_t*>(FAKE), 4, 200, 8, 2,
                              0, 1, 1.f, nullptr, nullptr, static_cast<int32_t*>(FAKE), static_cast<float*>(FAKE),
                              FAKE, BIG, nullptr) == MOE_ERR_SHAPE);
  EXPECT(moe_permute(static_cast<const int32_t*>(FAKE), 10, 2, 8, 0, static_cast<int32_t*>(FAKE),
                     static_cast<int32_t*>(FAKE), static_cast<int32_t*>(FAKE), 200, nullptr, 0, nullptr) == MOE_ERR_SHAPE);
  EXPECT(moe_act_quant_fp8(static_cast<const uint16_t*>(FAKE), 4, 100, static_cast<uint8_t*>(FAKE),
                           static_cast<float*>(FAKE), nullptr) == MOE_ERR_SHAPE);

  if (fails) {
    fprintf(stderr, "%d expectation(s) failed\n", fails);
    return 1;
  }
  printf("abi driver ok\n");
  return 0;
}
