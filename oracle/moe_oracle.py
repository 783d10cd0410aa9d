"""fp64 CPU oracle of one fused MoE layer -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module.  The product path (the HIP library and
its Python binding) never imports, calls or links it, and it never imports the
product: the two sides share nothing but the seeded input data of
``synth.moe_inputs``.

What it computes is the paper's MoE skeleton, MoE Gate -> Fused MoE -> Weight
Sum (Fig. 1; Fig. 3 and Sec. 5.1), with the numeric semantics of every
quantised format spelled out (e4m3 format, scale granularity, zero point,
layout; Sec. 6.2 and the "FP8 representation" row of Table 3).  The paper
states no formula for the layer, so every step below is the plain definition
of the operation, written out in float64 with library primitives (sort,
bincount, matmul, exp) and no blocking or fusion:

  router    l[t,e] = sum_h x[t,h] Wr[e,h] on the exact bf16 values (the
            optional router GEMM in front of the gate; its kernel
            accumulates in fp32, so the tests run this gate on the
            kernel's own fp32 logits and bound the logits separately).
  gate      key_e = l_e (+ b_e)            softmax scoring
            key_e = sigmoid(l_e) + b_e      sigmoid scoring (b: selection only)
            top-k by key, descending, equal keys -> lower expert index first;
            weights: softmax over the selected logits (renormalised) or the
            full softmax; sigmoid scores over their selected sum
            (renormalised) or raw; all times routed_scale.
  permute   segment per expert (ascending e), each padded to a multiple of
            block_m, flat ids t*k+j ascending inside a segment, pads = T*k.
  experts   a = SiLU(x W1[e,:I]^T) * (x W1[e,I:]^T);  y = a W2[e]^T
            with SiLU(g) = g / (1 + exp(-g)).
  combine   out[t] = sum_j w[t,j] * y[t,j].

Quantisation points the kernels take are mirrored (``mirror=True``):
  * bf16 / int4 weights, fp8 weights with bf16 activations ("fp8a16",
    the weight-only fp8 route) and MXFP4 weights with bf16 activations
    ("mxfp4": OCP MX E2M1 elements, E8M0 scale per 32 along K, two elements
    per byte, low nibble first): the intermediate ``a`` is rounded to fp32,
    then to bf16 (round to nearest even) before the second product; the
    hidden rows enter exactly;
  * fp8: the hidden rows and the intermediate ``a`` are each quantised per
    (row, 128-column group): s = fp32(max(amax, 1e-10) / 448) with an IEEE
    fp32 divide, q = e4m3fn(RNE(fp32(x / s))) saturated to +-448, and the
    product then uses q * s;
  * MXFP4 weights with MXFP8 activations ("mxfp4x8"): the MXFP4 weight
    storage above, and the hidden rows and the intermediate ``a`` (rounded
    to fp32) quantised per (row, 32-column block) by the OCP MX rule: shared
    scale X = 2^(floor(log2 amax) - 8) kept as an E8M0 byte (8 is the
    exponent of e4m3's largest power of two, 256), elements e4m3(RNE(x / X))
    saturated to +-448; the products use q * X.
With ``mirror=False`` the layer is evaluated on the unquantised operands.

Every function here is pinned by the CPU tests (tests/test_oracle_*.py)
against closed forms, brute force, invariants and an independent library
implementation; nothing here is "parity unpinned".
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

E4M3_MAX = 448.0
QGROUP = 128  # quantisation group along K (activations, int4 weights, fp8 blocks)
MX_BLOCK = 32  # OCP MX block: elements sharing one E8M0 scale
E4M3_EMAX = 8  # exponent of the largest power of two an e4m3 element holds (256)


# ============================================================ storage decoding
def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exact float64 values."""
    b = np.asarray(bits).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def f32_to_bf16_rne(x: np.ndarray) -> np.ndarray:
    """fp32 values -> bf16 bit patterns, round to nearest, ties to even
    (finite inputs).  Integer arithmetic on the fp32 bit pattern."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def _e4m3_value(c: np.ndarray) -> np.ndarray:
    """Closed form of OCP fp8 e4m3fn: layout S.EEEE.MMM, exponent bias 7, no
    infinities, S.1111.111 is NaN, E=0 encodes subnormals M * 2^-9."""
    c = c.astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = c & 0x7
    val = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.ldexp(1.0, e - 7))
    val = np.where((e == 15) & (m == 7), np.nan, val)
    return sign * val


_E4M3_TABLE = _e4m3_value(np.arange(256))  # the closed form at every code


def e4m3_decode(codes: np.ndarray) -> np.ndarray:
    """OCP fp8 e4m3fn codes -> float64 (the closed form, tabulated per code)."""
    return _E4M3_TABLE[np.asarray(codes).astype(np.uint8)]


def e4m3_encode(x: np.ndarray) -> np.ndarray:
    """Finite values -> e4m3fn codes: magnitude saturated to 448, then rounded
    to the nearest representable value, ties to even mantissa."""
    x = np.asarray(x, dtype=np.float64)
    neg = np.signbit(x)
    a = np.minimum(np.abs(x), E4M3_MAX)
    _, ex = np.frexp(a)                      # a = f * 2^ex, f in [0.5, 1)
    e = np.maximum(ex - 1, -6)               # binade of a; subnormals share 2^-6's step
    step = np.ldexp(1.0, e - 3)              # 3 mantissa bits
    r = np.rint(a / step) * step             # exact scaling, ties to even
    # split r back into fields
    _, ex2 = np.frexp(r)
    e2 = ex2 - 1
    is_norm = r >= 2.0 ** -6
    exp_field = np.where(is_norm, e2 + 7, 0)
    mant = np.where(is_norm, np.rint((r / np.ldexp(1.0, e2) - 1.0) * 8.0), np.rint(r / 2.0 ** -9))
    exp_field = np.where(r == 0, 0, exp_field)
    mant = np.where(r == 0, 0, mant)
    code = (neg.astype(np.int64) << 7) | (exp_field.astype(np.int64) << 3) | mant.astype(np.int64)
    return code.astype(np.uint8)


def _nibble_pair(b: np.ndarray) -> np.ndarray:
    """Byte -> its (low, high) nibbles as two's complement int4 values."""
    lo, hi = b & 0xF, (b >> 4) & 0xF
    return np.stack([np.where(lo >= 8, lo - 16, lo), np.where(hi >= 8, hi - 16, hi)], axis=-1)


_NIBBLES = _nibble_pair(np.arange(256)).astype(np.int8)  # [256, 2]
_NIBBLES_LE16 = np.ascontiguousarray(_NIBBLES).view("<i2").reshape(256)  # (lo, hi) packed per byte value


def int4_unpack(words: np.ndarray) -> np.ndarray:
    """int32 words [..., K/8] -> signed nibbles int8 [..., K]; element 8w+j is
    bits [4j, 4j+4) of word w, two's complement.  Byte b of a (little-endian)
    word holds elements 2b (low nibble) and 2b+1 (high nibble)."""
    w = np.ascontiguousarray(words).astype("<u4", copy=False)
    by = w.view(np.uint8)                                   # [..., K/2]
    return _NIBBLES_LE16[by].view(np.int8).reshape(w.shape[:-1] + (w.shape[-1] * 8,))


def _e2m1_value(c: np.ndarray) -> np.ndarray:
    """Closed form of the OCP MX FP4 element E2M1: layout S.EE.M, exponent bias
    1, E=0 encodes the subnormal M * 0.5; no infinities or NaN.  Magnitudes
    0, 0.5, 1, 1.5, 2, 3, 4, 6."""
    c = np.asarray(c).astype(np.int64) & 0xF
    sign = np.where(c & 0x8, -1.0, 1.0)
    e = (c >> 1) & 0x3
    m = c & 0x1
    return sign * np.where(e == 0, m * 0.5, (1.0 + m / 2.0) * np.ldexp(1.0, e - 1))


_E2M1_TABLE = _e2m1_value(np.arange(16))


def e8m0_value(s: np.ndarray) -> np.ndarray:
    """OCP MX shared scale E8M0: 2^(s - 127) for s in [0, 254]; 255 is NaN."""
    s = np.asarray(s).astype(np.int64)
    return np.where(s == 255, np.nan, np.ldexp(1.0, s - 127))


def mxfp4_unpack(packed: np.ndarray) -> np.ndarray:
    """uint8 [..., K/2] -> E2M1 codes [..., K]: element 2b is the low nibble of
    byte b, element 2b+1 its high nibble."""
    b = np.asarray(packed).astype(np.uint8)
    return np.stack([b & 0xF, b >> 4], axis=-1).reshape(b.shape[:-1] + (b.shape[-1] * 2,))


def dequant_weight(wfmt: str, w: np.ndarray, scale) -> np.ndarray:
    """One expert's stored weight [N, K] (+ scales) -> exact float64 values."""
    if wfmt == "bf16":
        return bf16_to_f64(w)
    if wfmt in ("fp8", "fp8a16"):                       # same storage, same values
        q = e4m3_decode(w)                                  # [N, K]
        N, K = q.shape
        s = np.asarray(scale, dtype=np.float64)            # [N/128, K/128]
        return (q.reshape(N // QGROUP, QGROUP, K // QGROUP, QGROUP) * s[:, None, :, None]).reshape(N, K)
    if wfmt == "int4":
        q = int4_unpack(w).astype(np.float64)              # [N, K]
        N, K = q.shape
        s = bf16_to_f64(scale)                              # [N, K/128]
        return (q.reshape(N, K // QGROUP, QGROUP) * s[:, :, None]).reshape(N, K)
    if wfmt in ("mxfp4", "mxfp4x8"):                    # E2M1 x E8M0 per 32 along K
        q = _E2M1_TABLE[mxfp4_unpack(w)]                    # [N, K]
        N, K = q.shape
        s = e8m0_value(scale)                               # [N, K/32]
        return (q.reshape(N, K // 32, 32) * s[:, :, None]).reshape(N, K)
    raise ValueError(f"unknown weight format {wfmt!r}")


# ============================================================ the layer
def router_logits(hidden_bits, w_router_bits):
    """Router GEMM in front of the MoE Gate (the step that feeds Fig. 1's gate
    node): float64 [T,E] = x Wr^T on the exact values of bf16 hidden [T,H]
    and bf16 router weights [E,H]."""
    return bf16_to_f64(hidden_bits) @ bf16_to_f64(w_router_bits).T


def gate(logits, sel_bias, top_k, mode="softmax", renormalize=True, routed_scale=1.0):
    """MoE Gate (Fig. 1): returns expert ids int32 [T,k] in descending-key
    order (equal keys -> lower index first) and float64 weights [T,k]."""
    lg = np.asarray(logits, dtype=np.float32).astype(np.float64)
    T, E = lg.shape
    if not 1 <= top_k <= E:
        raise ValueError("top_k must be in [1, E]")
    bias = np.zeros(E) if sel_bias is None else np.asarray(sel_bias, np.float32).astype(np.float64)
    if mode == "softmax":
        key = lg + bias[None, :]
    elif mode == "sigmoid":
        score = 1.0 / (1.0 + np.exp(-lg))
        key = score + bias[None, :]
    else:
        raise ValueError(f"unknown scoring mode {mode!r}")
    order = np.argsort(-key, axis=1, kind="stable")         # stable: ties keep index order
    ids = order[:, :top_k].astype(np.int32)
    if mode == "softmax":
        sel = np.take_along_axis(lg, ids, axis=1)
        if renormalize:
            z = np.exp(sel - sel.max(axis=1, keepdims=True))
            w = z / z.sum(axis=1, keepdims=True)
        else:
            m = lg.max(axis=1, keepdims=True)
            w = np.exp(sel - m) / np.exp(lg - m).sum(axis=1, keepdims=True)
    else:
        sel = np.take_along_axis(score, ids, axis=1)
        w = sel / sel.sum(axis=1, keepdims=True) if renormalize else sel
    return ids, w * float(routed_scale)


def permute_capacity(T, top_k, E, block_m):
    return T * top_k + E * (block_m - 1)


def permute(ids, E, block_m=1):
    """Token -> expert permutation.  Returns expert_offsets [E+1],
    sorted_ids [cap] (flat ids t*k+j, pads = T*k) and inv_pos [T*k]."""
    flat = np.asarray(ids).reshape(-1).astype(np.int64)
    n = flat.size
    counts = np.bincount(flat, minlength=E)
    padded = (counts + block_m - 1) // block_m * block_m
    offsets = np.concatenate([[0], np.cumsum(padded)]).astype(np.int32)
    cap = n + E * (block_m - 1)
    sorted_ids = np.full(cap, n, dtype=np.int32)
    inv_pos = np.empty(n, dtype=np.int32)
    order = np.argsort(flat, kind="stable")                 # by expert, flat id ascending
    start = 0
    for e in range(E):
        seg = order[start:start + counts[e]]
        sorted_ids[offsets[e]:offsets[e] + counts[e]] = seg
        inv_pos[seg] = offsets[e] + np.arange(counts[e])
        start += counts[e]
    return offsets, sorted_ids, inv_pos


def act_quant_fp8(x32: np.ndarray):
    """Per (row, 128-column group) e4m3 quantisation of fp32 rows [M, K]:
    returns codes uint8 [M, K] and fp32 scales [M, K/128]."""
    x = np.ascontiguousarray(x32, dtype=np.float32)
    M, K = x.shape
    g = x.reshape(M, K // QGROUP, QGROUP)
    amax = np.abs(g).max(axis=2)
    s = (np.maximum(amax, np.float32(1e-10)) / np.float32(E4M3_MAX)).astype(np.float32)
    y = (g / s[:, :, None]).astype(np.float32)              # IEEE fp32 divide
    return e4m3_encode(y).reshape(M, K), s


def act_dequant_fp8(codes, scales):
    M, K = codes.shape
    s = np.asarray(scales, np.float64)
    return (e4m3_decode(codes).reshape(M, K // QGROUP, QGROUP) * s[:, :, None]).reshape(M, K)


def act_quant_mxfp8(x32: np.ndarray):
    """Per (row, 32-column block) OCP MX quantisation of fp32 rows [M, K] to
    e4m3 elements with a shared E8M0 scale: X = 2^(floor(log2 amax) - 8),
    its byte 127 + log2 X clamped to [0, 254] (an all-zero block: byte 0);
    q = e4m3(RNE(x / X)) saturated to +-448.  Returns codes uint8 [M, K] and
    scale bytes uint8 [M, K/32]."""
    x = np.ascontiguousarray(x32, dtype=np.float32).astype(np.float64)
    M, K = x.shape
    blk = x.reshape(M, K // MX_BLOCK, MX_BLOCK)
    amax = np.abs(blk).max(axis=2)
    _, ex = np.frexp(amax)                    # amax = f * 2^ex, f in [0.5, 1): floor(log2 amax) = ex - 1
    e = np.where(amax > 0, ex - 1 - E4M3_EMAX, -127)
    e = np.clip(e, -127, 127)
    q = e4m3_encode(blk / np.ldexp(1.0, e)[:, :, None])   # exact scaling, then RNE + saturation
    return q.reshape(M, K), (e + 127).astype(np.uint8)


def act_dequant_mxfp8(codes, scale_bytes):
    M, K = codes.shape
    s = e8m0_value(scale_bytes)
    return (e4m3_decode(codes).reshape(M, K // MX_BLOCK, MX_BLOCK) * s[:, :, None]).reshape(M, K)


def _round_intermediate(a: np.ndarray, wfmt: str) -> np.ndarray:
    a32 = a.astype(np.float32)
    if wfmt == "fp8":
        return act_dequant_fp8(*act_quant_fp8(a32))
    if wfmt == "mxfp4x8":
        return act_dequant_mxfp8(*act_quant_mxfp8(a32))
    return bf16_to_f64(f32_to_bf16_rne(a32))


def swiglu_expert(x, w1, w2, wfmt="bf16", mirror=True):
    """One expert on rows x [M,H]: returns (a [M,I], y [M,H]) in float64."""
    I = w1.shape[0] // 2
    g = x @ w1[:I].T
    u = x @ w1[I:].T
    with np.errstate(over="ignore"):
        a = g / (1.0 + np.exp(-g)) * u
    if mirror:
        a = _round_intermediate(a, wfmt)
    return a, a @ w2.T


def activation_operand(hidden_bits, wfmt="bf16", mirror=True):
    """The first product's left operand for hidden rows (bf16 bits [M,H])."""
    x = bf16_to_f64(hidden_bits)
    if wfmt == "fp8" and mirror:
        return act_dequant_fp8(*act_quant_fp8(x.astype(np.float32)))
    if wfmt == "mxfp4x8" and mirror:
        return act_dequant_mxfp8(*act_quant_mxfp8(x.astype(np.float32)))
    return x


def _blas_threads(n):
    """Context that holds the BLAS library to n threads (a no-op without
    threadpoolctl)."""
    try:
        from threadpoolctl import threadpool_limits
        return threadpool_limits(limits=n, user_api="blas")
    except ImportError:  # pragma: no cover
        import contextlib
        return contextlib.nullcontext()


def default_threads() -> int:
    """Experts the layer evaluates at once: OMP_NUM_THREADS if set, else the
    core count, at most 16 (each one holds its dequantised weights)."""
    env = os.environ.get("OMP_NUM_THREADS", "")
    n = int(env) if env.isdigit() and int(env) > 0 else (os.cpu_count() or 1)
    return max(1, min(n, 16))


def forward(cfg, inputs, mirror=True, tokens=None, want_rows=False, threads=None):
    """The whole layer.  ``tokens``: optional subset of token indices, in
    which case ``out`` has one row per listed token (gate and experts run for
    those tokens only).  Returns a dict with ids, w, out and, if
    ``want_rows``, the per-routed-row intermediates ``a`` and ``y`` indexed by
    (token slot, j).  ``threads``: experts evaluated at once (default: the
    host's core count)."""
    T, k = cfg.T, cfg.top_k
    tok = np.arange(T) if tokens is None else np.asarray(tokens, dtype=np.int64)
    ids, w = gate(inputs["logits"][tok], inputs.get("sel_bias"), k, cfg.mode,
                  cfg.renormalize, cfg.routed_scale)
    x = activation_operand(inputs["hidden"][tok], cfg.wfmt, mirror)
    n = tok.size
    y = np.zeros((n * k, cfg.H))
    a_rows = np.zeros((n * k, cfg.I)) if want_rows else None
    flat = ids.reshape(-1)

    def one_expert(e):
        rows = np.nonzero(flat == e)[0]                     # flat slots t*k+j, ascending
        w1 = dequant_weight(cfg.wfmt, inputs["w1"][e], None if inputs["w1_scale"] is None else inputs["w1_scale"][e])
        w2 = dequant_weight(cfg.wfmt, inputs["w2"][e], None if inputs["w2_scale"] is None else inputs["w2_scale"][e])
        a, ye = swiglu_expert(x[rows // k], w1, w2, cfg.wfmt, mirror)
        y[rows] = ye                                        # experts write disjoint rows
        if want_rows:
            a_rows[rows] = a

    # Experts are independent; running several at once changes no arithmetic
    # (each one's rows, weights and products are its own).
    experts = np.unique(flat)
    workers = max(1, min(threads or default_threads(), experts.size))
    if workers == 1:
        for e in experts:
            one_expert(e)
    else:
        # one BLAS thread per expert: the experts themselves fill the cores
        with _blas_threads(1), ThreadPoolExecutor(max_workers=workers) as pool:
            list(pool.map(one_expert, experts))
    out = (w[:, :, None] * y.reshape(n, k, cfg.H)).sum(axis=1)
    res = {"ids": ids, "w": w, "out": out}
    if want_rows:
        res["a"], res["y"] = a_rows, y
    return res
