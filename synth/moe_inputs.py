"""Seeded synthetic inputs for one fused MoE layer.

This module produces DATA only: router logits, hidden states and expert
weights in their storage encodings (bf16 bits, block-scaled OCP fp8 e4m3,
group-scaled signed int4).  It holds none of the layer's arithmetic (no
gating, routing, matmul, activation or combine).  The storage encoders here
use torch's CPU casts (``bfloat16``, ``float8_e4m3fn``) so that they share no
code with either the fp64 oracle or the HIP kernels.

The layer is the MoE Gate -> Fused MoE -> Weight Sum skeleton of the paper
(Fig. 1, Fig. 3 and Sec. 5.1); the storage formats carry their numeric
semantics explicitly (e4m3 format, scale granularity, zero points, layout),
as Sec. 6.2 and the "FP8 representation" row of Table 3 require.

Value recipe (the five workloads and their decode / format variants):
  * hidden  ~ N(0, 1) drawn in fp32, stored as bf16 (round-to-nearest-even).
  * logits  ~ N(0, 1) fp32, plus an optional per-expert bias:
      - "normal:<std>"  b_e ~ N(0, std^2), added to the logits (uneven loads);
      - "zipf:<s>"      b_e = -s * ln(rank_e), rank_e a seeded permutation
                        of 1..E, so exp(b_e) follows a Zipf(s) law (skew).
  * sel_bias (sigmoid scoring only) ~ N(0, std^2): used for selection only.
  * w_router (only for the fused router + gate) bf16 [E, H] ~ N(0, 1/H).
  (Weight spreads are variances, N(0, 1/fan_in) = LeCun init; the bias
  spreads are standard deviations.)
  * W1[E, 2I, H], W2[E, H, I] ~ N(0, 1/fan_in) in fp32 (fan_in = H for W1,
    I for W2), then stored as
      - bf16:  round-to-nearest-even bf16 bits (uint16);
      - fp8:   per 128x128 block of [N, K]: s = max(amax, 1e-10) / 448 (fp32),
               q = e4m3fn(clamp(w / s, -448, 448)) (uint8 codes), scales fp32
               [E, N/128, K/128];
      - mxfp4: per 32 along K (OCP MX): X = 2^(floor(log2 amax) - 2),
               E2M1 codes of w / X (nearest, ties to even, saturated to 6),
               two per byte low nibble first, uint8 [E, N, K/2]; E8M0 scale
               bytes (127 + log2 X) uint8 [E, N, K/32];
      - int4:  per 128 along K: s = bf16(max(amax, 1e-10) / 7),
               q = clip(rint(w / s), -8, 7) signed two's complement nibble,
               zero point 0, packed 8 per int32 along K with element 8w+j in
               bits [4j, 4j+4) of word w (low nibble first); scales bf16
               [E, N, K/128].

Seeding: every tensor draws from PCG64(SeedSequence([seed, tensor_id, sub]))
where ``sub`` is the expert index for weights and the 64-token block index for
hidden, so any subset of experts can be regenerated independently and in any
order, by any number of threads.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace

import numpy as np
import torch

TID_HIDDEN, TID_LOGITS, TID_LOGIT_BIAS, TID_W1, TID_W2, TID_SEL_BIAS, TID_ROUTER = range(7)
HIDDEN_BLOCK = 64  # tokens per hidden-state substream


@dataclass(frozen=True)
class MoeConfig:
    """Shape, storage format and routing policy of one MoE layer workload."""

    name: str
    T: int
    H: int
    E: int
    I: int
    top_k: int
    wfmt: str = "bf16"          # "bf16" | "fp8" | "int4" | "fp8a16" (fp8 storage, bf16 activations)
                                # | "mxfp4" (MX E2M1 + E8M0 per 32, bf16 activations)
                                # | "mxfp4x8" (the mxfp4 storage, MXFP8 activations)
    mode: str = "softmax"       # "softmax" | "sigmoid"
    renormalize: bool = True
    routed_scale: float = 1.0
    logit_bias: str = "none"    # "none" | "normal:<std>" | "zipf:<s>"
    sel_bias_std: float = 0.0   # sigmoid selection-bias standard deviation (0 = no bias)
    seed: int = 0

    @property
    def n_routed(self) -> int:
        return self.T * self.top_k

    def active_flops(self) -> float:
        """Active-expert FLOPs of one layer: 2*T*k*(2I*H + H*I)."""
        return 6.0 * self.T * self.top_k * self.H * self.I


CONFIGS = {
    1: MoeConfig("tiny", T=64, H=256, E=8, I=128, top_k=2, seed=1),
    2: MoeConfig("decode", T=16, H=4096, E=64, I=1408, top_k=6, seed=2),
    3: MoeConfig("prefill", T=4096, H=4096, E=64, I=1408, top_k=6,
                 logit_bias="normal:0.5", seed=3),
    4: MoeConfig("fp8", T=8192, H=7168, E=256, I=2048, top_k=8, wfmt="fp8",
                 mode="sigmoid", routed_scale=2.5, sel_bias_std=0.1, seed=4),
    5: MoeConfig("int4", T=512, H=4096, E=128, I=1536, top_k=8, wfmt="int4",
                 logit_bias="zipf:1.1", seed=5),
    # one decode step of workload 4's layer on its fp8 weights, activations
    # kept bf16 (the weight-only fp8 route)
    6: MoeConfig("fp8-decode", T=16, H=7168, E=256, I=2048, top_k=8, wfmt="fp8a16",
                 mode="sigmoid", routed_scale=2.5, sel_bias_std=0.1, seed=6),
    # the same decode step with MXFP4 expert weights (bf16 activations)
    7: MoeConfig("mxfp4-decode", T=16, H=7168, E=256, I=2048, top_k=8, wfmt="mxfp4",
                 mode="sigmoid", routed_scale=2.5, sel_bias_std=0.1, seed=7),
    # workload 4's prefill batch on MXFP4 expert weights (bf16 activations)
    8: MoeConfig("mxfp4-prefill", T=8192, H=7168, E=256, I=2048, top_k=8, wfmt="mxfp4",
                 mode="sigmoid", routed_scale=2.5, sel_bias_std=0.1, seed=8),
    # the same batch and weights (seed 8) with MXFP8 activations: both
    # products on the block-scaled fp8 x fp4 matrix instruction
    9: MoeConfig("mxfp4x8-prefill", T=8192, H=7168, E=256, I=2048, top_k=8, wfmt="mxfp4x8",
                 mode="sigmoid", routed_scale=2.5, sel_bias_std=0.1, seed=8),
    # one decode step of workload 5's layer (int4 weights, Zipf-skewed routing)
    10: MoeConfig("int4-decode", T=16, H=4096, E=128, I=1536, top_k=8, wfmt="int4",
                  logit_bias="zipf:1.1", seed=10),
}


def config(n: int) -> MoeConfig:
    return CONFIGS[n]


def tiny_config(n: int, **overrides) -> MoeConfig:
    """A small variant of workload ``n`` with the same format and routing
    policy, sized so the fp64 oracle finishes in well under a second while the
    kernels still see several tiles and a ragged tail."""
    base = CONFIGS[n]
    small = dict(T=77, H=384, E=8, I=256, top_k=min(base.top_k, 3))
    if base.wfmt in ("fp8", "fp8a16", "mxfp4", "mxfp4x8"):
        small.update(E=16, top_k=4)
    if base.wfmt == "int4":
        small.update(E=12, top_k=4)
    small.update(overrides)
    return replace(base, name=base.name + "-small", **small)


def _rng(seed: int, tid: int, sub: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tid, sub])))


def _threads(threads):
    if threads:
        return threads
    return max(1, min(16, os.cpu_count() or 1))


def _bf16_bits(x32: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round-to-nearest-even (torch cast)."""
    return torch.from_numpy(np.ascontiguousarray(x32, dtype=np.float32)).to(
        torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).view(
        torch.bfloat16).to(torch.float32).numpy()


# ---------------------------------------------------------------- routing inputs
def make_routing_inputs(cfg: MoeConfig, threads=None) -> dict:
    """hidden (bf16 bits [T,H]), logits (fp32 [T,E]) and sel_bias (fp32 [E] or None)."""
    T, H, E = cfg.T, cfg.H, cfg.E
    hidden = np.empty((T, H), dtype=np.uint16)
    nblk = (T + HIDDEN_BLOCK - 1) // HIDDEN_BLOCK

    def fill(b):
        r0, r1 = b * HIDDEN_BLOCK, min(T, (b + 1) * HIDDEN_BLOCK)
        x = _rng(cfg.seed, TID_HIDDEN, b).standard_normal((r1 - r0, H), dtype=np.float32)
        hidden[r0:r1] = _bf16_bits(x)

    if nblk:
        with ThreadPoolExecutor(_threads(threads)) as ex:
            list(ex.map(fill, range(nblk)))

    logits = _rng(cfg.seed, TID_LOGITS).standard_normal((T, E), dtype=np.float32)
    kind, _, arg = cfg.logit_bias.partition(":")
    if kind == "normal":
        std = np.float32(float(arg))
        b = _rng(cfg.seed, TID_LOGIT_BIAS).standard_normal(E, dtype=np.float32) * std
        logits = (logits + b[None, :]).astype(np.float32)
    elif kind == "zipf":
        s = float(arg)
        rank = _rng(cfg.seed, TID_LOGIT_BIAS).permutation(E) + 1
        b = (-s * np.log(rank.astype(np.float64))).astype(np.float32)
        logits = (logits + b[None, :]).astype(np.float32)
    elif kind != "none":
        raise ValueError(f"unknown logit bias {cfg.logit_bias!r}")

    sel_bias = None
    if cfg.sel_bias_std > 0:
        std = np.float32(cfg.sel_bias_std)
        sel_bias = (_rng(cfg.seed, TID_SEL_BIAS).standard_normal(E, dtype=np.float32) * std).astype(np.float32)
    return {"hidden": hidden, "logits": np.ascontiguousarray(logits), "sel_bias": sel_bias}


def make_router_weights(cfg: MoeConfig) -> np.ndarray:
    """Router weights for the fused router + gate: bf16 bits [E, H] drawn
    N(0, 1/H) (LeCun), so with N(0, 1) hidden rows the logits are about
    N(0, 1) like the workloads' direct logits."""
    w = _rng(cfg.seed, TID_ROUTER).standard_normal((cfg.E, cfg.H), dtype=np.float32)
    return _bf16_bits(w * np.float32(1.0 / np.sqrt(cfg.H)))


# ---------------------------------------------------------------- weight storage
def _fp8_block_quant(w: np.ndarray):
    """[N,K] fp32 -> (uint8 e4m3fn codes [N,K], fp32 scales [N/128, K/128])."""
    N, K = w.shape
    blk = w.reshape(N // 128, 128, K // 128, 128)
    amax = np.abs(blk).max(axis=(1, 3))
    s = (np.maximum(amax, np.float32(1e-10)) / np.float32(448.0)).astype(np.float32)
    x = (blk / s[:, None, :, None]).astype(np.float32).reshape(N, K)
    x = np.clip(x, -448.0, 448.0)
    q = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    return q, s


_E2M1_GRID = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])  # magnitude of codes 0..7


def _mxfp4_quant(w: np.ndarray):
    """[N,K] fp32 -> (uint8 [N,K/2] two E2M1 codes per byte, low nibble
    first; uint8 E8M0 scales [N,K/32]).  Per 32-element block the OCP MX
    rule: X = 2^(floor(log2 amax) - 2) (2 = the largest E2M1 exponent), the
    elements w / X rounded to the nearest E2M1 magnitude (ties to the even
    code) and saturated to 6.  An all-zero block takes X = 1."""
    N, K = w.shape
    blk = w.astype(np.float64).reshape(N, K // 32, 32)
    amax = np.abs(blk).max(axis=2)
    e = np.where(amax > 0, np.floor(np.log2(np.where(amax > 0, amax, 1.0))) - 2, 0).astype(np.int64)
    e = np.clip(e, -126, 127)
    x = blk / np.ldexp(1.0, e)[:, :, None]
    a = np.minimum(np.abs(x), 6.0)
    d = np.abs(a[..., None] - _E2M1_GRID)                   # [N, K/32, 32, 8]
    idx = d.argmin(axis=-1)
    nxt = np.minimum(idx + 1, 7)
    tie = (np.take_along_axis(d, nxt[..., None], -1)[..., 0] == np.take_along_axis(d, idx[..., None], -1)[..., 0])
    idx = np.where(tie & (idx % 2 == 1) & (nxt != idx), nxt, idx)
    code = (idx | np.where(np.signbit(x) & (idx > 0), 8, 0)).astype(np.uint8).reshape(N, K)
    packed = (code[:, 0::2] | (code[:, 1::2] << 4)).astype(np.uint8)
    return packed, (e + 127).astype(np.uint8)


def _int4_group_quant(w: np.ndarray):
    """[N,K] fp32 -> (int32 packed words [N,K/8], bf16-bit scales [N,K/128])."""
    N, K = w.shape
    g = w.reshape(N, K // 128, 128)
    amax = np.abs(g).max(axis=2)
    s_bits = _bf16_bits((np.maximum(amax, np.float32(1e-10)) / np.float32(7.0)).astype(np.float32))
    s = _bf16_bits_to_f32(s_bits)
    q = np.clip(np.rint(g / s[:, :, None]), -8, 7).astype(np.int32).reshape(N, K // 8, 8)
    nib = (q & 0xF).astype(np.uint32)
    word = np.zeros((N, K // 8), dtype=np.uint32)
    for j in range(8):
        word |= nib[:, :, j] << np.uint32(4 * j)
    return word.view(np.int32), s_bits


def _weight_arrays(cfg: MoeConfig, N: int, K: int, n_exp: int):
    if cfg.wfmt == "bf16":
        return np.empty((n_exp, N, K), np.uint16), None
    if cfg.wfmt in ("fp8", "fp8a16"):
        return np.empty((n_exp, N, K), np.uint8), np.empty((n_exp, N // 128, K // 128), np.float32)
    if cfg.wfmt == "int4":
        return np.empty((n_exp, N, K // 8), np.int32), np.empty((n_exp, N, K // 128), np.uint16)
    if cfg.wfmt in ("mxfp4", "mxfp4x8"):
        return np.empty((n_exp, N, K // 2), np.uint8), np.empty((n_exp, N, K // 32), np.uint8)
    raise ValueError(f"unknown weight format {cfg.wfmt!r}")


def make_expert_weights(cfg: MoeConfig, experts=None, threads=None, identical_experts=False) -> dict:
    """W1/W2 (and scales) of the listed experts (all by default), stacked in
    the order given.  ``identical_experts`` draws every expert from expert 0's
    stream (a test fixture: all experts then hold the same weights)."""
    experts = list(range(cfg.E)) if experts is None else list(experts)
    H, I = cfg.H, cfg.I
    if cfg.wfmt != "bf16" and (H % 128 or I % 128):
        raise ValueError("fp8/int4 storage needs H and I to be multiples of 128")
    w1, w1s = _weight_arrays(cfg, 2 * I, H, len(experts))
    w2, w2s = _weight_arrays(cfg, H, I, len(experts))

    def encode(dst, dst_s, slot, w):
        if cfg.wfmt == "bf16":
            dst[slot] = _bf16_bits(w)
        elif cfg.wfmt in ("fp8", "fp8a16"):
            dst[slot], dst_s[slot] = _fp8_block_quant(w)
        elif cfg.wfmt in ("mxfp4", "mxfp4x8"):
            dst[slot], dst_s[slot] = _mxfp4_quant(w)
        else:
            dst[slot], dst_s[slot] = _int4_group_quant(w)

    def fill(slot):
        e = 0 if identical_experts else experts[slot]
        a = _rng(cfg.seed, TID_W1, e).standard_normal((2 * I, H), dtype=np.float32)
        a *= np.float32(1.0 / np.sqrt(H))
        encode(w1, w1s, slot, a)
        del a
        b = _rng(cfg.seed, TID_W2, e).standard_normal((H, I), dtype=np.float32)
        b *= np.float32(1.0 / np.sqrt(I))
        encode(w2, w2s, slot, b)

    with ThreadPoolExecutor(_threads(threads)) as ex:
        list(ex.map(fill, range(len(experts))))
    return {"w1": w1, "w2": w2, "w1_scale": w1s, "w2_scale": w2s}


def make_inputs(cfg: MoeConfig, threads=None, identical_experts=False) -> dict:
    """Every input of one layer call, as numpy arrays (see the module doc)."""
    out = make_routing_inputs(cfg, threads)
    out.update(make_expert_weights(cfg, threads=threads, identical_experts=identical_experts))
    return out


# ---------------------------------------------------------------- device upload
def to_device(inputs: dict, device="cuda") -> dict:
    """Numpy inputs -> torch tensors on ``device`` in the library's dtypes:
    bf16 bits as torch.bfloat16, fp8 codes as uint8, int4 words as int32,
    fp32 scales as float32, bf16 scales as torch.bfloat16."""
    out = {}
    for k, v in inputs.items():
        if v is None:
            out[k] = None
            continue
        t = torch.from_numpy(np.ascontiguousarray(v))
        if v.dtype == np.uint16:
            t = t.view(torch.int16).view(torch.bfloat16)
        out[k] = t.to(device)
    return out
