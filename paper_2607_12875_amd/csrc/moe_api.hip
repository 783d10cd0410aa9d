// C ABI of the fused MoE layer (declared in include/moe.h): host-side argument
// validation, workspace carving and the launch sequence
//   gate -> permute -> [fp8 activation quantisation] -> GEMM1(+SiLU*up) ->
//   GEMM2 -> combine
// for the MoE Gate -> Fused MoE -> Weight Sum skeleton (Fig. 1, Fig. 3).
// Every check runs before the first launch (quantised dispatch fails early on
// an incompatible request, the guard rule of Sec. 6.2 / Table 3); nothing here
// allocates or synchronises.  The only state is the per-device address of the
// static workspace moe_forward_static_ws runs in.
#include <atomic>
#include <mutex>

#include "../../include/moe.h"
#include "launch.hpp"

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

moe_status check_topk_shape(long T, int E, int top_k) {
  if (T < 0 || E < 1 || E > MOE_MAX_EXPERTS) return MOE_ERR_SHAPE;
  if (top_k < 1 || top_k > E || top_k > MOE_MAX_TOPK) return MOE_ERR_SHAPE;
  if (T * top_k > (1L << 28)) return MOE_ERR_SHAPE;
  return MOE_OK;
}

// H and I: multiples of 8 for bf16 weights, of 128 for the quantised formats
// (their scale blocks and groups are 128 wide along K, 128 rows for fp8),
// at most 65536.
moe_status check_hi(const moe_args* a) {
  const int q = a->wfmt == MOE_W_BF16 ? 8 : 128;
  if (a->H < q || a->I < q || a->H % q || a->I % q) return MOE_ERR_SHAPE;
  if (a->H > (1 << 16) || a->I > (1 << 16)) return MOE_ERR_SHAPE;
  return MOE_OK;
}

moe_status check_args(const moe_args* a) {
  if (!a) return MOE_ERR_NULL;
  moe_status st = check_topk_shape(a->T, a->E, a->top_k);
  if (st != MOE_OK) return st;
  if (check_hi(a) != MOE_OK) return MOE_ERR_SHAPE;
  if (a->score_mode != MOE_SCORE_SOFTMAX && a->score_mode != MOE_SCORE_SIGMOID) return MOE_ERR_UNSUPPORTED;
  if (a->renormalize != 0 && a->renormalize != 1) return MOE_ERR_UNSUPPORTED;
  if (a->wfmt != MOE_W_BF16 && a->wfmt != MOE_W_FP8E4M3_B128 && a->wfmt != MOE_W_INT4_G128 &&
      a->wfmt != MOE_W_FP8E4M3_B128_A16 && a->wfmt != MOE_W_MXFP4_A16 && a->wfmt != MOE_W_MXFP4_MXFP8)
    return MOE_ERR_UNSUPPORTED;
  // the weight-only fp8 route is a decode route (16-row kernels only)
  if (a->wfmt == MOE_W_FP8E4M3_B128_A16 && static_cast<long>(a->T) * a->top_k > 32L * a->E)
    return MOE_ERR_UNSUPPORTED;
  if (a->ofmt != MOE_OUT_F32 && a->ofmt != MOE_OUT_BF16) return MOE_ERR_UNSUPPORTED;
  // the router GEMM steps through H in K slices of 128-element multiples
  if (a->w_router && a->H % 128) return MOE_ERR_UNSUPPORTED;
  if (a->T == 0) return MOE_OK;
  if (!a->hidden || (!a->logits && !a->w_router) || !a->w1 || !a->w2 || !a->out) return MOE_ERR_NULL;
  if (a->wfmt != MOE_W_BF16 && (!a->w1_scale || !a->w2_scale)) return MOE_ERR_NULL;
  if (!aligned16(a->hidden) || !aligned16(a->w1) || !aligned16(a->w2) || !aligned16(a->out))
    return MOE_ERR_ALIGN;
  if (a->wfmt != MOE_W_BF16 && (!aligned16(a->w1_scale) || !aligned16(a->w2_scale)))
    return MOE_ERR_ALIGN;
  if (!aligned16(a->w_router) || !aligned4(a->logits_out)) return MOE_ERR_ALIGN;
  if (!aligned4(a->logits) || !aligned4(a->sel_bias) || !aligned4(a->topk_ids_out) ||
      !aligned4(a->topk_w_out))
    return MOE_ERR_ALIGN;
  return MOE_OK;
}

// Workspace layout for validated sizes (T may be 0).
moe_ws_layout make_layout(const moe_args* a) {
  moe_ws_layout L;
  const long n = static_cast<long>(a->T) * a->top_k;
  const int bm = moe::gemm_block_m(a->wfmt, a->T, a->top_k, a->E, a->H, a->I);
  const long cap = n + static_cast<long>(a->E) * (bm - 1);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes);
    return static_cast<int64_t>(o);
  };
  L.block_m = bm;
  L.cap = static_cast<int32_t>(cap);
  L.topk_ids = take(n * 4);
  L.topk_w = take(n * 4);
  L.expert_offsets = take((a->E + 1) * 4);
  L.sorted_ids = take(cap * 4);
  L.inv_pos = take(n * 4);
  if (a->wfmt == MOE_W_FP8E4M3_B128) {
    L.act_q = take(static_cast<size_t>(a->T) * a->H);
    L.act_s = take(static_cast<size_t>(a->T) * (a->H / 128) * 4);
    L.inter = take(static_cast<size_t>(cap) * a->I);
    L.inter_s = take(static_cast<size_t>(cap) * (a->I / 128) * 4);
  } else if (a->wfmt == MOE_W_MXFP4_MXFP8) {
    L.act_q = take(static_cast<size_t>(a->T) * a->H);
    L.act_s = take(static_cast<size_t>(a->T) * (a->H / 32));
    L.inter = take(static_cast<size_t>(cap) * a->I);
    L.inter_s = take(static_cast<size_t>(cap) * (a->I / 32));
  } else {
    L.act_q = -1;
    L.act_s = a->wfmt == MOE_W_INT4_G128 ? take(static_cast<size_t>(a->T) * (a->H / 128) * 4) : -1;
    L.inter = take(static_cast<size_t>(cap) * a->I * 2);
    L.inter_s = -1;
  }
  L.y = take(static_cast<size_t>(cap) * a->H * (moe::y_is_f32(a->wfmt) ? 4 : 2));
  L.permute_ws = take(moe::permute_workspace_bytes(a->T, a->top_k, a->E));
  L.router_ws = a->w_router ? take(moe::router_workspace_bytes(a->T, a->H, a->E)) : -1;
  L.total = static_cast<int64_t>(off);
  return L;
}

template <class T>
T* at(void* ws, int64_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

}  // namespace

extern "C" {

const char* moe_status_str(int s) {
  switch (s) {
    case MOE_OK: return "MOE_OK";
    case MOE_ERR_NULL: return "MOE_ERR_NULL";
    case MOE_ERR_SHAPE: return "MOE_ERR_SHAPE";
    case MOE_ERR_UNSUPPORTED: return "MOE_ERR_UNSUPPORTED";
    case MOE_ERR_ALIGN: return "MOE_ERR_ALIGN";
    case MOE_ERR_WORKSPACE: return "MOE_ERR_WORKSPACE";
    case MOE_ERR_HIP: return "MOE_ERR_HIP";
    default: return "MOE_ERR_UNKNOWN";
  }
}

size_t moe_permute_capacity(int T, int top_k, int E, int block_m) {
  if (T < 0 || top_k < 1 || E < 1 || block_m < 1) return 0;
  return static_cast<size_t>(T) * top_k + static_cast<size_t>(E) * (block_m - 1);
}

size_t moe_permute_workspace_bytes(int T, int top_k, int E) {
  if (check_topk_shape(T, E, top_k) != MOE_OK) return 0;
  return moe::permute_workspace_bytes(T, top_k, E);
}

moe_status moe_gate_topk(const float* logits, const float* sel_bias, int T, int E, int top_k,
                         int mode, int renormalize, float routed_scale, int32_t* topk_ids,
                         float* topk_w, hipStream_t stream) {
  moe_status st = check_topk_shape(T, E, top_k);
  if (st != MOE_OK) return st;
  if (mode != MOE_SCORE_SOFTMAX && mode != MOE_SCORE_SIGMOID) return MOE_ERR_UNSUPPORTED;
  if (renormalize != 0 && renormalize != 1) return MOE_ERR_UNSUPPORTED;
  if (T == 0) return MOE_OK;
  if (!logits || !topk_ids || !topk_w) return MOE_ERR_NULL;
  if (!aligned4(logits) || !aligned4(sel_bias) || !aligned4(topk_ids) || !aligned4(topk_w))
    return MOE_ERR_ALIGN;
  if (moe::launch_gate_topk(logits, sel_bias, T, E, top_k, mode, renormalize, routed_scale,
                            topk_ids, topk_w, nullptr, nullptr, stream) != hipSuccess)
    return MOE_ERR_HIP;
  return MOE_OK;
}

size_t moe_router_workspace_bytes(int T, int H, int E) {
  if (T < 0 || E < 1 || E > MOE_MAX_EXPERTS || H < 128 || H % 128 || H > (1 << 16)) return 0;
  return moe::router_workspace_bytes(T, H, E);
}

moe_status moe_router_gate_topk(const uint16_t* hidden, const uint16_t* w_router, int T, int H, int E,
                                int top_k, int mode, int renormalize, float routed_scale,
                                const float* sel_bias, float* logits, int32_t* topk_ids, float* topk_w,
                                void* ws, size_t ws_bytes, hipStream_t stream) {
  moe_status st = check_topk_shape(T, E, top_k);
  if (st != MOE_OK) return st;
  if (H < 128 || H % 128 || H > (1 << 16)) return MOE_ERR_SHAPE;
  if (mode != MOE_SCORE_SOFTMAX && mode != MOE_SCORE_SIGMOID) return MOE_ERR_UNSUPPORTED;
  if (renormalize != 0 && renormalize != 1) return MOE_ERR_UNSUPPORTED;
  if (T == 0) return MOE_OK;
  if (!hidden || !w_router || !topk_ids || !topk_w) return MOE_ERR_NULL;
  const size_t need = moe::router_workspace_bytes(T, H, E);
  if (need > 0 && (!ws || ws_bytes < need)) return MOE_ERR_WORKSPACE;
  if (!aligned16(hidden) || !aligned16(w_router) || !aligned16(ws)) return MOE_ERR_ALIGN;
  if (!aligned4(logits) || !aligned4(sel_bias) || !aligned4(topk_ids) || !aligned4(topk_w))
    return MOE_ERR_ALIGN;
  if (moe::launch_router_gate(hidden, w_router, T, H, E, top_k, mode, renormalize, routed_scale, sel_bias,
                              logits, topk_ids, topk_w, nullptr, nullptr, ws, stream) != hipSuccess)
    return MOE_ERR_HIP;
  return MOE_OK;
}

moe_status moe_permute(const int32_t* topk_ids, int T, int top_k, int E, int block_m,
                       int32_t* expert_offsets, int32_t* sorted_ids, int32_t* inv_pos, int cap,
                       void* ws, size_t ws_bytes, hipStream_t stream) {
  moe_status st = check_topk_shape(T, E, top_k);
  if (st != MOE_OK) return st;
  if (block_m < 1 || block_m > 1024) return MOE_ERR_SHAPE;
  if (cap < 0 || static_cast<size_t>(cap) < moe_permute_capacity(T, top_k, E, block_m))
    return MOE_ERR_SHAPE;
  if (!expert_offsets || !sorted_ids) return MOE_ERR_NULL;
  if (T > 0 && (!topk_ids || !inv_pos)) return MOE_ERR_NULL;
  if (!aligned4(topk_ids) || !aligned4(expert_offsets) || !aligned4(sorted_ids) || !aligned4(inv_pos))
    return MOE_ERR_ALIGN;
  const size_t need = moe::permute_workspace_bytes(T, top_k, E);
  if (need > 0 && (!ws || ws_bytes < need)) return MOE_ERR_WORKSPACE;
  if (need > 0 && !aligned16(ws)) return MOE_ERR_ALIGN;
  if (moe::launch_permute(topk_ids, T, top_k, E, block_m, expert_offsets, sorted_ids, inv_pos, cap,
                          ws, stream) != hipSuccess)
    return MOE_ERR_HIP;
  return MOE_OK;
}

moe_status moe_act_quant_fp8(const uint16_t* x, int M, int K, uint8_t* q, float* s,
                             hipStream_t stream) {
  if (M < 0 || K < 128 || K % 128) return MOE_ERR_SHAPE;
  if (M == 0) return MOE_OK;
  if (!x || !q || !s) return MOE_ERR_NULL;
  if (!aligned16(x) || !aligned16(q) || !aligned4(s)) return MOE_ERR_ALIGN;
  if (moe::launch_act_quant(x, M, K, q, s, stream) != hipSuccess) return MOE_ERR_HIP;
  return MOE_OK;
}

size_t moe_workspace_bytes(const moe_args* a) {
  if (!a || check_topk_shape(a->T, a->E, a->top_k) != MOE_OK) return 0;
  if (check_hi(a) != MOE_OK) return 0;
  return static_cast<size_t>(make_layout(a).total);
}

moe_status moe_workspace_layout(const moe_args* a, moe_ws_layout* layout) {
  if (!a || !layout) return MOE_ERR_NULL;
  moe_status st = check_topk_shape(a->T, a->E, a->top_k);
  if (st != MOE_OK) return st;
  if (check_hi(a) != MOE_OK) return MOE_ERR_SHAPE;
  *layout = make_layout(a);
  return MOE_OK;
}

}  // extern "C"

namespace {

// The launch sequence.  With `events` non-null, events[i] is recorded on the
// stream before stage i (gate, permute, activation quantisation, GEMM1, GEMM2,
// combine) and events[MOE_NUM_STAGES] after the last; the work is the same.
moe_status run_layer(const moe_args* a, void* ws, size_t ws_bytes, hipEvent_t* events,
                     hipStream_t stream) {
  moe_status st = check_args(a);
  if (st != MOE_OK) return st;
  if (a->T == 0) return MOE_OK;
  const moe_ws_layout L = make_layout(a);
  if (!ws || ws_bytes < static_cast<size_t>(L.total)) return MOE_ERR_WORKSPACE;
  if (!aligned16(ws)) return MOE_ERR_ALIGN;
  auto mark = [&](int i) {
    return events && events[i] ? hipEventRecord(events[i], stream) == hipSuccess : true;
  };

  int32_t* ids = at<int32_t>(ws, L.topk_ids);
  float* wts = at<float>(ws, L.topk_w);
  int32_t* offs = at<int32_t>(ws, L.expert_offsets);
  int32_t* sorted = at<int32_t>(ws, L.sorted_ids);
  int32_t* inv = at<int32_t>(ws, L.inv_pos);

  if (!mark(0)) return MOE_ERR_HIP;
  const hipError_t gate_err =
      a->w_router
          ? moe::launch_router_gate(a->hidden, a->w_router, a->T, a->H, a->E, a->top_k, a->score_mode,
                                    a->renormalize, a->routed_scale, a->sel_bias, a->logits_out, ids, wts,
                                    a->topk_ids_out, a->topk_w_out, at<void>(ws, L.router_ws), stream)
          : moe::launch_gate_topk(a->logits, a->sel_bias, a->T, a->E, a->top_k, a->score_mode, a->renormalize,
                                  a->routed_scale, ids, wts, a->topk_ids_out, a->topk_w_out, stream);
  if (gate_err != hipSuccess) return MOE_ERR_HIP;
  if (!mark(1)) return MOE_ERR_HIP;
  if (moe::launch_permute(ids, a->T, a->top_k, a->E, L.block_m, offs, sorted, inv, L.cap,
                          at<void>(ws, L.permute_ws), stream) != hipSuccess)
    return MOE_ERR_HIP;

  moe::GroupedGemm g;
  g.x = a->hidden;
  g.x_scale = nullptr;
  g.x_mx = nullptr;
  g.x_gsum = nullptr;
  if (!mark(2)) return MOE_ERR_HIP;
  if (a->wfmt == MOE_W_INT4_G128 && !moe::int4_decode(a->T, a->top_k, a->E, a->H, a->I)) {
    float* gs = at<float>(ws, L.act_s);
    if (moe::launch_group_sum(a->hidden, a->T, a->H, gs, stream) != hipSuccess) return MOE_ERR_HIP;
    g.x_gsum = gs;
  }
  if (a->wfmt == MOE_W_FP8E4M3_B128) {
    uint8_t* q = at<uint8_t>(ws, L.act_q);
    float* s = at<float>(ws, L.act_s);
    if (moe::launch_act_quant(a->hidden, a->T, a->H, q, s, stream) != hipSuccess) return MOE_ERR_HIP;
    g.x = q;
    g.x_scale = s;
  }
  if (a->wfmt == MOE_W_MXFP4_MXFP8) {
    uint8_t* q = at<uint8_t>(ws, L.act_q);
    uint8_t* sx = at<uint8_t>(ws, L.act_s);
    if (moe::launch_act_quant_mx(a->hidden, a->T, a->H, q, sx, stream) != hipSuccess) return MOE_ERR_HIP;
    g.x = q;
    g.x_mx = sx;
  }
  g.sorted_ids = sorted;
  g.offsets = offs;
  g.T = a->T;
  g.H = a->H;
  g.E = a->E;
  g.I = a->I;
  g.top_k = a->top_k;
  g.n_routed = a->T * a->top_k;
  g.max_rows = L.cap;
  g.w1 = a->w1;
  g.w1_scale = a->w1_scale;
  g.w2 = a->w2;
  g.w2_scale = a->w2_scale;
  g.inter = at<void>(ws, L.inter);
  g.inter_scale = L.inter_s >= 0 && a->wfmt == MOE_W_FP8E4M3_B128 ? at<float>(ws, L.inter_s) : nullptr;
  g.inter_mx = L.inter_s >= 0 && a->wfmt == MOE_W_MXFP4_MXFP8 ? at<uint8_t>(ws, L.inter_s) : nullptr;
  g.y = at<void>(ws, L.y);
  if (!mark(3)) return MOE_ERR_HIP;
  if (moe::launch_gemm1(a->wfmt, g, stream) != hipSuccess) return MOE_ERR_HIP;
  if (!mark(4)) return MOE_ERR_HIP;
  if (moe::launch_gemm2(a->wfmt, g, stream) != hipSuccess) return MOE_ERR_HIP;
  if (!mark(5)) return MOE_ERR_HIP;
  if (moe::launch_combine(g.y, moe::y_is_f32(a->wfmt), wts, inv, a->T, a->H, a->top_k,
                          a->ofmt == MOE_OUT_BF16, a->out, stream) != hipSuccess)
    return MOE_ERR_HIP;
  if (!mark(6)) return MOE_ERR_HIP;
  return MOE_OK;
}

}  // namespace

// The library's own workspace for moe_forward_static_ws: one array per GPU,
// created when the code object is loaded on that GPU and held until the
// process ends.  In host code `scratch` names a host-side stand-in, never the
// device memory: its device address is looked up once per device and only
// that address is used.
static __device__ __align__(256) uint8_t scratch[MOE_STATIC_WS_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of this device's `scratch` (nullptr on failure).
void* scratch_on_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p) return p;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
  if (!p) {
    void* q = nullptr;
    if (hipGetSymbolAddress(&q, HIP_SYMBOL(scratch)) != hipSuccess || !q) return nullptr;
    p = q;
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  return p;
}

}  // namespace

extern "C" {

moe_status moe_forward(const moe_args* a, void* ws, size_t ws_bytes, hipStream_t stream) {
  return run_layer(a, ws, ws_bytes, nullptr, stream);
}

moe_status moe_forward_static_ws(const moe_args* a, hipStream_t stream) {
  moe_status st = check_args(a);
  if (st != MOE_OK) return st;
  if (a->T == 0) return MOE_OK;
  if (static_cast<size_t>(make_layout(a).total) > MOE_STATIC_WS_BYTES) return MOE_ERR_WORKSPACE;
  void* ws = scratch_on_current_device();
  if (!ws) return MOE_ERR_HIP;
  return run_layer(a, ws, MOE_STATIC_WS_BYTES, nullptr, stream);
}

moe_status moe_forward_profiled(const moe_args* a, void* ws, size_t ws_bytes,
                                hipEvent_t* events, hipStream_t stream) {
  if (!events) return MOE_ERR_NULL;
  return run_layer(a, ws, ws_bytes, events, stream);
}

}  // extern "C"
