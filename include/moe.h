/*
 * moe.h -- C ABI of the fused Mixture-of-Experts layer for AMD MI355X (gfx950).
 *
 * The layer is the paper's MoE skeleton, MoE Gate -> Fused MoE -> Weight Sum
 * (Fig. 1; Fig. 3 and Sec. 5.1), for one GPU:
 *
 *   gate     router logits [T,E] -> top-k expert ids and weights per token
 *   permute  token -> expert grouping (histogram, padded prefix scan, stable
 *            scatter)
 *   experts  per expert e and routed row x:  a = SiLU(x W1[e,:I]^T) * (x W1[e,I:]^T),
 *            y = a W2[e]^T, SiLU(g) = g / (1 + exp(-g))
 *   combine  out[t] = sum_j w[t,j] * y[t,j]            ("Weight Sum")
 *
 * Quantised weight formats carry their full numeric semantics in the format
 * tag (e4m3 flavour, scale granularity, zero point, layout), as Sec. 6.2 and
 * the "FP8 representation" row of Table 3 ask of quantisation dispatch.
 *
 * Conventions for every entry point:
 *   - Pointers marked "device" are HIP device (or managed) memory owned by the
 *     caller; the library never allocates, frees or retains them, and keeps no
 *     state between calls.  All arrays are dense, row-major, contiguous.
 *   - bf16 values are passed as their uint16_t bit patterns.
 *   - Work is enqueued on `stream` and never synchronised; results are
 *     available when the stream has drained.  Nothing is copied to the host.
 *   - Arguments are validated on the host before anything is enqueued; on any
 *     error nothing is enqueued and outputs are untouched.
 *   - Calls on one stream are ordered; concurrent calls that share output or
 *     workspace buffers race.
 *   - Inputs must be finite, with one exception: a router logit or a
 *     selection bias of -inf masks that expert (it is chosen only when a
 *     token has fewer than top_k other experts, lowest index first, and a
 *     masked softmax logit gets weight 0).  NaN and +inf give unspecified
 *     results.
 */
#ifndef MOE_H
#define MOE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MOE_OK = 0,
  MOE_ERR_NULL = 1,        /* a required pointer is NULL                         */
  MOE_ERR_SHAPE = 2,       /* a size is out of range or inconsistent             */
  MOE_ERR_UNSUPPORTED = 3, /* valid request this library does not implement      */
  MOE_ERR_ALIGN = 4,       /* a device pointer is not 16-byte aligned            */
  MOE_ERR_WORKSPACE = 5,   /* workspace smaller than moe_workspace_bytes()       */
  MOE_ERR_HIP = 6          /* a kernel launch failed (hipGetLastError)           */
} moe_status;

/* Router scoring (MoE Gate, Fig. 1). */
typedef enum {
  /* key_e = logit_e (+ sel_bias_e); weights = softmax over the selected
     logits (renormalize=1) or the softmax over all E logits (renormalize=0). */
  MOE_SCORE_SOFTMAX = 0,
  /* s_e = 1/(1+exp(-logit_e)); key_e = s_e + sel_bias_e (selection only);
     weights = s_j / sum_selected s (renormalize=1) or s_j (renormalize=0). */
  MOE_SCORE_SIGMOID = 1
} moe_score;

/* Expert weight storage.  N x K below is [2I x H] for W1 and [H x I] for W2. */
typedef enum {
  /* bf16 bits, w[e][n][k] (uint16_t).  H and I multiples of 8 (rows stay
     16-byte aligned); when either is not a multiple of 128 every batch runs
     the tiled kernels (segments padded to 128 rows). */
  MOE_W_BF16 = 0,
  /* OCP fp8 e4m3fn codes (bias 7, max 448, no Inf, S.1111.111 = NaN),
     w[e][n][k] (uint8_t); fp32 scale per 128x128 block of [N,K]:
     scale[e][n/128][k/128]; value = decode(q) * scale.  Activations are then
     quantised in-layer to e4m3 with an fp32 scale per (row, 128 columns):
     s = max(amax, 1e-10) / 448 (IEEE fp32 divide), q = RNE(x / s) saturated
     to +-448; the SwiGLU intermediate is quantised the same way. */
  MOE_W_FP8E4M3_B128 = 1,
  /* signed two's-complement int4, zero point 0, 8 per int32 along K: element
     k = 8w+j sits in bits [4j,4j+4) of word w (low nibble first):
     w[e][n][K/8] (int32_t); bf16 scale per 128 along K: scale[e][n][k/128];
     value = q * scale.  Hidden rows enter as bf16 and the SwiGLU
     intermediate is rounded to bf16.  The first product sums each 128-group
     of codes exactly and applies the group's scale in fp32; the second
     rounds q * scale to bf16 before its products, except at decode sizes
     (T * top_k <= 8 * E, H and I in {512, 1024, 1536, 2048, 3072, 4096}),
     where both products take the first one's exact form.  A scale may be zero;
     the nonzero scales must be normal numbers within a factor 2^64 of each
     other along a weight row (other scales are unspecified): above the
     decode sizes the first product carries its running sums divided by the
     current group's scale, so a ratio r between groups multiplies them by r,
     and 2^64 keeps them inside the fp32 range with about 2^30 to spare for
     the sums themselves (the decode sizes scale each group's own partial
     and have no such limit).
     Scales from a per-group amax quantiser of real weight rows differ by a
     few powers of two. */
  MOE_W_INT4_G128 = 2,
  /* Weight-only fp8 (a decode route): the MOE_W_FP8E4M3_B128 storage and
     scales, but the hidden rows enter unquantised (bf16) and the SwiGLU
     intermediate is rounded to bf16 as with MOE_W_BF16; the weights are
     decoded to bf16 in registers (exact) and each 128-wide K block's partial
     sum is scaled by its block scale.  Requires T * top_k <= 32 * E (at most
     32 routed rows per expert on average), else MOE_ERR_UNSUPPORTED: larger
     batches take MOE_W_FP8E4M3_B128. */
  MOE_W_FP8E4M3_B128_A16 = 3,
  /* MXFP4 weights (OCP Microscaling v1.0), weight-only: E2M1 codes (S.EE.M, bias 1; magnitudes 0, 0.5,
     1, 1.5, 2, 3, 4, 6), two per byte, element k = 2b+j in bits [4j,4j+4) of
     byte b (low nibble first): w[e][n][K/2] (uint8_t); one E8M0 scale byte
     per 32 along K: scale[e][n][K/32], value 2^(s-127) (s = 255, NaN, and
     products beyond the bf16 range are unspecified); value = e2m1(q) *
     2^(s-127), decoded exactly to bf16.  Hidden rows enter as bf16, the
     SwiGLU intermediate is rounded to bf16.  Any batch: up to 32 routed rows
     per expert on average the 16-row decode kernels run, above that the
     tiled ones (segments padded to 128 rows). */
  MOE_W_MXFP4_A16 = 4,
  /* MXFP4 weights with MXFP8 activations (OCP Microscaling v1.0 on both
     sides of each product): the MOE_W_MXFP4_A16 weight storage and scales;
     the hidden rows are quantised in-layer per (row, 32 columns) to e4m3
     elements with a shared E8M0 scale X = 2^(floor(log2 amax) - 8) (8: the
     exponent of e4m3's largest power of two; the E8M0 byte is clamped to
     [0, 254], an all-zero block takes 2^-127), elements RNE(x / X) saturated
     to +-448; the SwiGLU intermediate (fp32) is quantised the same way per
     (row, 32 of I).  Both products run on the block-scaled matrix
     instruction, which applies the E8M0 scales itself.  Any batch size
     (segments padded to 128 rows). */
  MOE_W_MXFP4_MXFP8 = 5
} moe_wfmt;

typedef enum { MOE_OUT_F32 = 0, MOE_OUT_BF16 = 1 } moe_ofmt;

/* Limits checked on the host. */
#define MOE_MAX_EXPERTS 1024
#define MOE_MAX_TOPK 32

/*
 * MoE Gate (Fig. 1): top-k expert selection per token.
 *   logits    device fp32 [T,E]
 *   sel_bias  device fp32 [E] or NULL (= zeros); enters the selection key only
 *   T >= 0, 1 <= E <= MOE_MAX_EXPERTS, 1 <= top_k <= min(E, MOE_MAX_TOPK)
 *   mode      moe_score; renormalize 0/1; routed_scale multiplies every weight
 *   topk_ids  device int32 [T,top_k]: experts in descending key order; equal
 *             keys -> lower expert index first.  Keys are compared in fp64
 *             (the fp32 logit, or fp64 sigmoid + bias).
 *   topk_w    device fp32 [T,top_k]: weights, computed in fp64, rounded once.
 * Errors: MOE_ERR_NULL, MOE_ERR_SHAPE, MOE_ERR_ALIGN (logits/outputs need
 * 4-byte alignment only), MOE_ERR_HIP.  T == 0 is a no-op.
 */
moe_status moe_gate_topk(const float* logits, const float* sel_bias, int T, int E, int top_k,
                         int mode, int renormalize, float routed_scale, int32_t* topk_ids,
                         float* topk_w, hipStream_t stream);

/*
 * Router GEMM in front of the gate (the step before the MoE Gate node,
 * Fig. 1): logits[t,e] = sum_h hidden[t,h] * w_router[e,h], bf16 products
 * accumulated in fp32, then exactly the selection and weights of
 * moe_gate_topk on those fp32 logits.  Where T * E >= 2^20 (E % 8 == 0
 * and T > 64): the logits as a plain GEMM over 128-token tiles (row ids,
 * offsets and logits in ws), then the gate.  Otherwise up to 1024 tokens two
 * launches: the logits GEMM in K slices over many workgroups (partial
 * logits in ws; 16-token tiles up to 64 tokens, 64-token tiles above), then
 * one wavefront per token that sums the slices in slice order and selects;
 * above 1024 tokens one kernel per 16-token tile, and no scratch.
 *   hidden    device bf16 bits [T,H], 16-byte aligned; H % 128 == 0, H <= 65536
 *   w_router  device bf16 bits [E,H], 16-byte aligned
 *   logits    device fp32 [T,E] or NULL: receives the logits the selection used
 *   ws        device scratch of >= moe_router_workspace_bytes(T, H, E) bytes,
 *             16-byte aligned (contents on entry do not matter); may be NULL
 *             when that size is 0
 *   other arguments and the outputs as moe_gate_topk.
 * The fp32 accumulation order is the kernel's own and the same on every run:
 * logits agree with the exact sums to within a few fp32 roundings of
 * sum_h |hidden * w_router|.
 * Errors: MOE_ERR_NULL, MOE_ERR_SHAPE, MOE_ERR_UNSUPPORTED, MOE_ERR_ALIGN,
 * MOE_ERR_WORKSPACE, MOE_ERR_HIP.  T == 0 is a no-op.
 */
moe_status moe_router_gate_topk(const uint16_t* hidden, const uint16_t* w_router, int T, int H, int E,
                                int top_k, int mode, int renormalize, float routed_scale,
                                const float* sel_bias, float* logits, int32_t* topk_ids, float* topk_w,
                                void* ws, size_t ws_bytes, hipStream_t stream);

/* Scratch moe_router_gate_topk needs (bytes); 0 for invalid sizes.  Host-only, pure. */
size_t moe_router_workspace_bytes(int T, int H, int E);

/* Rows needed by moe_permute's sorted_ids: T*top_k + E*(block_m-1).  Host-only. */
size_t moe_permute_capacity(int T, int top_k, int E, int block_m);

/* Device scratch moe_permute needs (bytes).  Host-only, pure. */
size_t moe_permute_workspace_bytes(int T, int top_k, int E);

/*
 * Permute / align: groups the T*top_k routed rows by expert -- the hand-over
 * from the MoE Gate node to the Fused MoE node of Fig. 1 (and Fig. 3): the
 * fused expert products consume each expert's routed rows as one contiguous
 * segment (the paper names the nodes, not this step's algorithm).
 *   topk_ids        device int32 [T,top_k], each in [0,E)
 *   block_m         1..1024: every expert segment is padded to a multiple
 *   expert_offsets  device int32 [E+1]: off[0]=0,
 *                   off[e+1] = off[e] + roundup(count_e, block_m)
 *   sorted_ids      device int32 [cap], cap >= moe_permute_capacity(): inside
 *                   segment e the flat ids t*top_k+j of rows routed to e in
 *                   ascending order, then pads; every slot from the pads of
 *                   each segment up to cap holds the pad id T*top_k
 *   inv_pos         device int32 [T*top_k]: position of flat id f in sorted_ids
 *   ws, ws_bytes    device scratch of >= moe_permute_workspace_bytes()
 * Deterministic: bit-identical on every run.
 * Errors: MOE_ERR_NULL, MOE_ERR_SHAPE (cap too small, block_m out of range),
 * MOE_ERR_WORKSPACE, MOE_ERR_HIP.  T == 0 writes offsets (all 0) and pads.
 */
moe_status moe_permute(const int32_t* topk_ids, int T, int top_k, int E, int block_m,
                       int32_t* expert_offsets, int32_t* sorted_ids, int32_t* inv_pos, int cap,
                       void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Activation quantisation for the fp8 format (done inside moe_forward; exposed
 * for unit checks): per (row, 128-column group) of bf16 x [M,K]:
 *   s = max(amax, 1e-10) / 448 (fp32, IEEE divide), q = e4m3fn(RNE(x / s))
 *   saturated to +-448.
 *   x  device bf16 bits [M,K]; q device uint8 [M,K]; s device fp32 [M,K/128]
 * Needs K % 128 == 0 and 16-byte aligned pointers.
 */
moe_status moe_act_quant_fp8(const uint16_t* x, int M, int K, uint8_t* q, float* s,
                             hipStream_t stream);

/* The whole layer. */
typedef struct moe_args {
  int32_t T, H, E, I, top_k;
  int32_t score_mode;       /* moe_score                                     */
  int32_t renormalize;      /* 0 / 1                                          */
  float routed_scale;       /* multiplies every routing weight               */
  int32_t wfmt;             /* moe_wfmt                                       */
  int32_t ofmt;             /* moe_ofmt                                       */
  const float* sel_bias;    /* device fp32 [E] or NULL                        */
  const uint16_t* hidden;   /* device bf16 [T,H]                              */
  const float* logits;      /* device fp32 [T,E]; NULL when w_router is set    */
  const void* w1;           /* device, [E,2I,H] in the wfmt storage (gate rows [0,I), up rows [I,2I)) */
  const void* w2;           /* device, [E,H,I] in the wfmt storage            */
  const void* w1_scale;     /* device, per wfmt (NULL for bf16)               */
  const void* w2_scale;     /* device, per wfmt (NULL for bf16)               */
  void* out;                /* device [T,H], fp32 or bf16 per ofmt            */
  int32_t* topk_ids_out;    /* optional device int32 [T,top_k] copy, or NULL  */
  float* topk_w_out;        /* optional device fp32 [T,top_k] copy, or NULL   */
  const uint16_t* w_router; /* device bf16 [E,H] or NULL: if set, the layer computes its
                               logits from hidden (moe_router_gate_topk) and ignores `logits` */
  float* logits_out;        /* optional device fp32 [T,E]: those logits, or NULL */
} moe_args;

/* Workspace bytes moe_forward needs for these sizes/format.  Host-only, pure. */
size_t moe_workspace_bytes(const moe_args* a);

/* Where moe_forward keeps its intermediates inside the workspace (byte
   offsets; for inspection by tests and profilers).  -1 = not used. */
typedef struct moe_ws_layout {
  int64_t topk_ids, topk_w;          /* int32 / fp32 [T*top_k]                   */
  int64_t expert_offsets;            /* int32 [E+1]                              */
  int64_t sorted_ids, inv_pos;       /* int32 [cap], int32 [T*top_k]             */
  int64_t act_q, act_s;              /* fp8: uint8 [T,H], fp32 [T,H/128]; MXFP8:
                                        uint8 [T,H] e4m3, uint8 [T,H/32] E8M0;
                                        int4: act_s = fp32 [T,H/128] group sums
                                        of the hidden rows (times -136), not
                                        written at the decode sizes above     */
  int64_t inter, inter_s;            /* bf16 [cap,I] (fp8: uint8 [cap,I], fp32 [cap,I/128];
                                        MXFP8: uint8 [cap,I], uint8 [cap,I/32] E8M0) */
  int64_t y;                         /* [cap,H] rows in sorted order: bf16 for
                                        MOE_W_FP8E4M3_B128 and MOE_W_MXFP4_MXFP8,
                                        fp32 otherwise; pad rows unspecified */
  int64_t permute_ws;                /* moe_permute scratch                      */
  int64_t router_ws;                 /* router partial logits (w_router set), else -1 */
  int32_t block_m, cap;              /* padding granule and sorted_ids length   */
  int64_t total;                     /* == moe_workspace_bytes                  */
} moe_ws_layout;

moe_status moe_workspace_layout(const moe_args* a, moe_ws_layout* layout);

/*
 * Fused MoE layer: [router GEMM] gate -> permute -> [fp8 activation quantisation] ->
 * grouped GEMM1 with fused SiLU*up epilogue -> grouped GEMM2 -> combine, all
 * enqueued on `stream`; no host synchronisation, no allocation.
 * Requirements: T >= 0; 1 <= E <= MOE_MAX_EXPERTS; 1 <= top_k <= min(E,
 * MOE_MAX_TOPK); 8 <= H, I <= 65536, multiples of 8 for MOE_W_BF16 and of
 * 128 for the quantised formats (with w_router, H a multiple of 128 in every
 * format, else MOE_ERR_UNSUPPORTED); every device pointer 16-byte
 * aligned; ws_bytes >= moe_workspace_bytes(a); sel_bias only with a format
 * that reads it (both scoring modes do).  Padding rows of the intermediates
 * are unspecified.  T == 0 is a no-op.
 * MOE_W_FP8E4M3_B128_A16 additionally needs
 * T * top_k <= 32 * E.  With
 * w_router set the router GEMM and the gate run as moe_router_gate_topk
 * (its scratch inside the workspace) and `logits` may be NULL.
 * Errors: MOE_ERR_NULL, MOE_ERR_SHAPE, MOE_ERR_UNSUPPORTED, MOE_ERR_ALIGN,
 * MOE_ERR_WORKSPACE, MOE_ERR_HIP.
 */
moe_status moe_forward(const moe_args* a, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * moe_forward with per-stage timing: the same launches on the same stream,
 * with events[i] recorded before stage i and events[MOE_NUM_STAGES] after the
 * last stage.  Stages: 0 gate, 1 permute, 2 fp8 activation quantisation
 * (empty for bf16 / int4), 3 GEMM1 + SiLU*up, 4 GEMM2, 5 combine.
 *   events  host array of MOE_NUM_STAGES + 1 caller-created hipEvent_t; a
 *           NULL entry skips that mark (e.g. only GEMM1 bracketed: entries 3
 *           and 4 set)
 * Errors: those of moe_forward; MOE_ERR_NULL for a NULL array.
 */
#define MOE_NUM_STAGES 6
moe_status moe_forward_profiled(const moe_args* a, void* ws, size_t ws_bytes,
                                hipEvent_t* events, hipStream_t stream);

/*
 * moe_forward without a caller workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  The layer runs exactly as moe_forward, but its
 * intermediates live in the library's own device array of
 * MOE_STATIC_WS_BYTES, one per GPU, which exists from the first use of the
 * library on that GPU until the process ends.  The caller still passes
 * every input and output in `a`.  The call allocates nothing.
 *   a       as moe_forward; moe_workspace_bytes(a) must not exceed
 *           MOE_STATIC_WS_BYTES, else MOE_ERR_WORKSPACE (nothing enqueued).
 * Every call on one GPU shares that GPU's array and leaves its intermediates
 * there (nothing in it needs to start zeroed): calls that overlap on one GPU
 * (on different streams, or from several threads without ordering) race.
 * Errors: those of moe_forward; MOE_ERR_HIP if the array's device address
 * cannot be obtained.
 */
#define MOE_STATIC_WS_BYTES (256u << 20)
moe_status moe_forward_static_ws(const moe_args* a, hipStream_t stream);

/* Static, NUL-terminated name of a status code. */
const char* moe_status_str(int status);

#ifdef __cplusplus
}
#endif
#endif /* MOE_H */
