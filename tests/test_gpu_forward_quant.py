"""GPU parity of the quantised expert routes against the fp64 oracle with
the same quantisation points: the e4m3 activation quantiser bit-exact, the
fp8 layer within 6e-2 * rms and the int4 layer within 8e-2 * rms; routing
and permutation bit-exact."""
import numpy as np
import pytest
import torch

import paper_2607_12875_amd as moe
import synth
from oracle import moe_oracle as O
from tests.gpu_util import check_forward, require_gpu, run_forward, ws_view

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def _bf16(x32):
    return O.f32_to_bf16_rne(np.asarray(x32, np.float32))


def _act_quant_check(bits):
    x = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()
    q, s = moe.moe_act_quant_fp8(x)
    torch.cuda.synchronize()
    rq, rs = O.act_quant_fp8(O.bf16_to_f64(bits).astype(np.float32))
    assert np.array_equal(s.cpu().numpy(), rs)
    qq = q.cpu().numpy()
    bad = np.argwhere(qq != rq)
    assert bad.size == 0, (bad[:5], qq[tuple(bad[0])], rq[tuple(bad[0])])


def test_act_quant_bit_exact_crafted(dev):
    x = np.zeros((4, 256), np.float32)
    x[0, :6] = [448.0, -1.0, 0.015625, 240.0, 2.0 ** -9, -(2.0 ** -10)]
    x[1, 5], x[1, 6] = 1.0, -0.5                        # amax 1: top code, non-exact scale
    x[2, 128], x[2, 129], x[2, 130] = 896.0, 2.125, 2.375   # s = 2: ties 1.0625 / 1.1875
    x[3] = np.linspace(-3, 3, 256)
    x[3, 100] = -0.0                                    # keeps its sign: code 0x80
    _act_quant_check(_bf16(x))


def test_act_quant_bit_exact_structured(dev):
    # Groups whose scale is set by one amax (255 bf16 patterns across the
    # normal range, plus zero and denormal ones) holding every bf16 magnitude
    # up to it, signs alternating: the quantiser's per-element quotient is
    # checked code for code against the oracle's IEEE division.
    amaxes = list(range(0x0080, 0x7F80, 128)) + [0x0000, 0x0001, 0x007F]
    groups = []
    for a in amaxes:
        xs = np.arange(0, a + 1, dtype=np.uint16)
        sign = (np.arange(xs.size) & 1).astype(np.uint16) << 15
        xs = np.concatenate([xs | sign, np.array([0x8000], np.uint16)])  # and -0
        for g0 in range(0, xs.size, 127):
            grp = np.zeros(128, np.uint16)
            grp[0] = a
            piece = xs[g0:g0 + 127]
            grp[1:1 + piece.size] = piece
            groups.append(grp)
    while len(groups) % 8:
        groups.append(np.zeros(128, np.uint16))
    bits = np.stack(groups).reshape(-1, 8 * 128)
    _act_quant_check(bits)


def test_act_quant_bit_exact_fp8_workload_rows(dev):
    r = synth.make_routing_inputs(synth.tiny_config(4, T=777, H=7168))
    _act_quant_check(r["hidden"])


def _check(cfg, inp=None):
    return check_forward(cfg, inp)[0]


# gfx950's fp8 MFMA aligns the 64 products of one instruction with truncation
# (65536 + 63 * 2^-6 comes back as 65536.875, not 65536.984), so the GPU's
# intermediate before requantisation differs from the oracle's by ~1e-5
# relative and an e4m3 code whose value sits on a rounding tie can land one
# step away.  One such step moves an output by ~1/sqrt(I) of its rms, so the
# output-level fp8 cases use I >= 1024 (the workload has I = 2048); the codes
# themselves are pinned by test_fp8_intermediate_codes at small I.
@pytest.mark.parametrize("T", [1, 33, 200, 700])
def test_fp8_small(dev, T):
    _check(synth.tiny_config(4, T=T, H=512, I=1024, E=16, top_k=4))


def _oracle_preq_intermediate(cfg, inp):
    """The oracle's SwiGLU intermediate of every routed row, before its
    requantisation, rounded once to fp32 (the precision the quantiser sees)."""
    n = cfg.T * cfg.top_k
    ids, _ = O.gate(inp["logits"], inp["sel_bias"], cfg.top_k, cfg.mode, cfg.renormalize, cfg.routed_scale)
    x = O.activation_operand(inp["hidden"], cfg.wfmt, True)
    flat = ids.reshape(-1)
    a = np.zeros((n, cfg.I))
    for e in np.unique(flat):
        rows = np.nonzero(flat == e)[0]
        w1 = O.dequant_weight(cfg.wfmt, inp["w1"][e], inp["w1_scale"][e])
        w2 = O.dequant_weight(cfg.wfmt, inp["w2"][e], inp["w2_scale"][e])
        a[rows] = O.swiglu_expert(x[rows // cfg.top_k], w1, w2, cfg.wfmt, mirror=False)[0]
    return a.astype(np.float32)


@pytest.mark.parametrize("shape", [dict(T=700, H=512, I=256, E=16, top_k=4),
                                   dict(T=1500, H=384, I=384, E=8, top_k=2, logit_bias="zipf:6.0", sel_bias_std=0.0)])
def test_fp8_intermediate_codes(dev, shape):
    """The requantised intermediate GEMM1 writes (e4m3 codes + per (row, 128)
    scales) against the oracle's quantiser applied to its own fp32
    intermediate: scales within 2e-4 relative; every code the rounding of a
    value within 2e-4 * 448 (in units of the scale) of the oracle's a/s --
    exact away from rounding ties, at most the neighbouring code at a tie."""
    cfg = synth.tiny_config(4, **shape)
    inp = synth.make_inputs(cfg)
    out, ws, L, _ = run_forward(cfg, inp)
    n, I, cap = cfg.T * cfg.top_k, cfg.I, L["cap"]
    sid = ws_view(ws, L, "sorted_ids", torch.int32, cap)
    codes = ws_view(ws, L, "inter", torch.uint8, cap * I).reshape(cap, I)
    scales = ws_view(ws, L, "inter_s", torch.float32, cap * (I // 128)).reshape(cap, I // 128)
    rows = np.nonzero(sid < n)[0]
    a32 = _oracle_preq_intermediate(cfg, inp)[sid[rows]]
    qref, sref = O.act_quant_fp8(a32)
    s_gpu = scales[rows]
    assert np.all(np.abs(s_gpu.astype(np.float64) - sref) <= 2e-4 * sref)
    x = a32.astype(np.float64) / np.repeat(sref, 128, axis=1).astype(np.float64)
    slack = 2e-4 * O.E4M3_MAX
    v_lo = O.e4m3_decode(O.e4m3_encode(x - slack))
    v_hi = O.e4m3_decode(O.e4m3_encode(x + slack))
    v_g = O.e4m3_decode(codes[rows])
    ok = (v_g >= v_lo) & (v_g <= v_hi)
    bad = np.argwhere(~ok)
    assert bad.size == 0, (bad[:3], x[tuple(bad[0])], v_g[tuple(bad[0])], v_lo[tuple(bad[0])], v_hi[tuple(bad[0])])
    ties = int((codes[rows] != qref).sum())
    print(f"  {ties} of {qref.size} codes one tie away from the oracle's", flush=True)
    assert ties <= 0.01 * qref.size


def test_fp8_h_not_multiple_of_256(dev):
    _check(synth.tiny_config(4, T=150, H=384, I=384, E=8, top_k=3))


# A single K step in GEMM2 (I = 128) with a full-width GEMM2 tile (H = 256),
# and several row tiles per expert on a wider layer.
@pytest.mark.parametrize("shape", [dict(T=400, H=256, I=128, E=4, top_k=2),
                                   dict(T=2000, H=768, I=1024, E=24, top_k=3)])
def test_fp8_more_shapes(dev, shape):
    _check(synth.tiny_config(4, **shape))


@pytest.mark.parametrize("T", [1, 45, 300, 1000])
def test_int4_small(dev, T):
    _check(synth.tiny_config(5, T=T, H=512, I=256, E=12, top_k=4))


def test_int4_h_not_multiple_of_256(dev):
    _check(synth.tiny_config(5, T=150, H=384, I=384, E=8, top_k=3))


@pytest.mark.parametrize("wcfg", [4, 5])
def test_quant_minimum_k(dev, wcfg):
    # H = I = 128: a single K step per tile
    _check(synth.tiny_config(wcfg, T=400, H=128, I=128, E=4, top_k=2))


def test_int4_workload_full_size(dev):
    _check(synth.config(5))


def test_fp8_workload_full_size(dev):
    # all 8192 tokens (58.7M outputs) and every row's activation codes
    _check(synth.config(4))


def test_quant_run_twice_bit_identical(dev):
    for cfg in (synth.tiny_config(4, T=300), synth.tiny_config(5, T=300)):
        inp = synth.make_inputs(cfg)
        a, ws, _, _ = run_forward(cfg, inp)
        b, _, _, _ = run_forward(cfg, inp, workspace=ws)
        assert np.array_equal(a, b)


def _scale_blocks(inp, wfmt, seed=1):
    """Multiply every stored weight scale by its own power of two in
    [2^-3, 2^3] (exact in fp32 and bf16).  The inputs stay valid and the
    oracle reads the same tensors, but a scale applied to the wrong K block or
    row block now moves the outputs far beyond the tolerance."""
    rng = np.random.default_rng(seed)
    out = dict(inp)
    for k in ("w1_scale", "w2_scale"):
        d = rng.integers(-3, 4, size=inp[k].shape)
        if wfmt == "int4":      # bf16 bits
            out[k] = O.f32_to_bf16_rne((O.bf16_to_f64(inp[k]) * 2.0 ** d).astype(np.float32))
        elif wfmt in ("mxfp4", "mxfp4x8"):   # E8M0 exponent bytes
            out[k] = (inp[k].astype(np.int64) + d).astype(np.uint8)
        else:                   # fp32
            out[k] = (inp[k] * 2.0 ** d).astype(np.float32)
    return out


@pytest.mark.parametrize("wcfg", [4, 5, 6, 7])
def test_block_scales_vary(dev, wcfg):
    cfg = synth.tiny_config(wcfg, T=100, H=512, I=1024 if wcfg == 4 else 256, E=8, top_k=2)
    _check(cfg, inp=_scale_blocks(synth.make_inputs(cfg), cfg.wfmt))


def test_int4_hidden_group_sums(dev):
    # the int4 GEMM1's pre-pass: act_s holds -136 times each hidden row's sum
    # over every 128-column group (fp32 sums of the bf16 values)
    cfg = synth.tiny_config(5, T=37, H=640, I=256, E=6, top_k=2)
    inp = synth.make_inputs(cfg)
    _, ws, L, _ = run_forward(cfg, inp)
    assert L["act_s"] >= 0 and L["act_q"] < 0
    got = ws_view(ws, L, "act_s", torch.float32, cfg.T * cfg.H // 128).reshape(cfg.T, cfg.H // 128)
    x = O.bf16_to_f64(inp["hidden"]).reshape(cfg.T, cfg.H // 128, 128)
    want = -136.0 * x.sum(axis=2)
    bound = 136.0 * np.abs(x).sum(axis=2) * 2.0 ** -20   # fp32 summation of 128 terms, with room
    assert np.all(np.abs(got - want) <= bound)


def test_int4_zero_and_wide_scales(dev):
    # int4 group scales of zero (scattered, leading runs, whole rows) and
    # scales spread over 2^-8 .. 2^8 along one weight row: the GEMM1 applies
    # each group's scale to its partial sums, carrying the accumulators
    # divided by the current scale from group to group.  (Wider spreads make
    # the output so heavy-tailed -- max|out| tens of times its rms -- that one
    # bf16 rounding step of the intermediate exceeds the rms-relative bound.)
    cfg = synth.tiny_config(5, T=200, H=1024, I=256, E=6, top_k=2)
    inp = synth.make_inputs(cfg)
    rng = np.random.default_rng(7)
    out = dict(inp)
    for k in ("w1_scale", "w2_scale"):
        f = O.bf16_to_f64(inp[k]) * 2.0 ** rng.integers(-8, 9, size=inp[k].shape)
        f[rng.random(f.shape) < 0.2] = 0.0
        f[:, ::7, :2] = 0.0    # rows whose first groups are zero
        f[:, 3::11, :] = 0.0   # rows with no nonzero group
        out[k] = O.f32_to_bf16_rne(f.astype(np.float32))
    _check(cfg, inp=out)


# ---- int4 decode route: the 16-row streamed kernels up to 8 routed rows per
# expert on average; both products sum each 128-group of codes exactly and
# apply the row's group scale to the group's partial in fp32
def _int4_decode_layout(cfg):
    a = moe.make_args(cfg.T, cfg.H, cfg.E, cfg.I, cfg.top_k, wfmt=cfg.wfmt)
    return moe.moe_workspace_layout(a)["block_m"]


@pytest.mark.parametrize("T", [1, 5, 16, 32])
def test_int4_decode_small(dev, T):
    # T = 32: T * top_k = 128 = 8 * E, the largest batch of the decode route
    cfg = synth.tiny_config(5, T=T, H=1024, I=512, E=16, top_k=4)
    assert _int4_decode_layout(cfg) == 16
    _check(cfg)


def test_int4_decode_route_boundary(dev):
    # one token more than the decode route takes: the 64-row tiled kernels
    cfg = synth.tiny_config(5, T=33, H=1024, I=512, E=16, top_k=4)
    assert _int4_decode_layout(cfg) == 64
    _check(cfg)


@pytest.mark.parametrize("H,I", [(512, 2048), (1536, 1024), (2048, 3072), (3072, 512), (4096, 1536)])
def test_int4_decode_streamed(dev, H, I):
    # K up to 2048 splits over two waves, 3072 and 4096 over four; every piece
    # carries its 16 rows' group scales (randomised here by up to 2^+-3)
    cfg = synth.tiny_config(5, T=12, H=H, I=I, E=9, top_k=3)
    assert _int4_decode_layout(cfg) == 16
    _check(cfg, inp=_scale_blocks(synth.make_inputs(cfg), cfg.wfmt, seed=H + I))


def test_int4_decode_zero_and_wide_scales(dev):
    # zero group scales (scattered, leading runs, whole rows) and scales
    # spread over 2^-8 .. 2^8 along a row, on the decode route
    cfg = synth.tiny_config(5, T=12, H=2048, I=1024, E=6, top_k=2)
    assert _int4_decode_layout(cfg) == 16
    inp = synth.make_inputs(cfg)
    rng = np.random.default_rng(11)
    out = dict(inp)
    for k in ("w1_scale", "w2_scale"):
        f = O.bf16_to_f64(inp[k]) * 2.0 ** rng.integers(-8, 9, size=inp[k].shape)
        f[rng.random(f.shape) < 0.2] = 0.0
        f[:, ::7, :2] = 0.0
        f[:, 3::11, :] = 0.0
        out[k] = O.f32_to_bf16_rne(f.astype(np.float32))
    _check(cfg, inp=out)


@pytest.mark.parametrize("shape", [dict(T=8, H=512, I=512, E=1, top_k=1),     # one expert, both K minimal
                                   dict(T=1, H=4096, I=4096, E=4, top_k=1),    # one token, the largest K
                                   dict(T=3, H=2048, I=512, E=64, top_k=2)])   # most experts empty
def test_int4_decode_edges(dev, shape):
    cfg = synth.tiny_config(5, **shape)
    assert _int4_decode_layout(cfg) == 16
    _check(cfg)


def test_int4_decode_scales_beyond_tiled_range(dev):
    # group scales alternating by 2^+-36 along every weight row: ratios of
    # 2^72 between neighbouring groups, past the 64-row kernels' 2^64 limit;
    # the decode kernels scale each group's own partial, so none applies
    cfg = synth.tiny_config(5, T=12, H=2048, I=1024, E=6, top_k=2)
    assert _int4_decode_layout(cfg) == 16
    inp = synth.make_inputs(cfg)
    out = dict(inp)
    for k in ("w1_scale", "w2_scale"):
        f = O.bf16_to_f64(inp[k])
        f = f * 2.0 ** np.where(np.arange(f.shape[-1]) % 2 == 0, 36, -36)
        out[k] = O.f32_to_bf16_rne(f.astype(np.float32))
    _check(cfg, inp=out)


def test_int4_decode_concentrated_routing(dev):
    # every token routed to the same four experts: 32 rows each, so each of
    # them spans two 16-row tiles and the other experts hold none
    cfg = synth.tiny_config(5, T=32, H=2048, I=1536, E=16, top_k=4)
    assert _int4_decode_layout(cfg) == 16
    inp = synth.make_inputs(cfg)
    inp = dict(inp)
    lg = inp["logits"].copy()
    lg[:, [3, 7, 8, 13]] += 20.0
    inp["logits"] = lg
    _check(cfg, inp=inp)


def test_int4_decode_workload_full_size(dev):
    # workload 5's layer at 16 tokens: every output against the oracle
    cfg = synth.config(10)
    assert _int4_decode_layout(cfg) == 16
    _check(cfg)


# ---- weight-only fp8: e4m3 weights with their block scales, bf16 activations
@pytest.mark.parametrize("T", [1, 5, 16, 33, 128])
def test_w8a16_small(dev, T):
    # T = 128: T * top_k = 512 = 32 * E, the largest batch the route accepts
    _check(synth.tiny_config(6, T=T, H=512, I=256, E=16, top_k=4))


def test_w8a16_ragged_k(dev):
    # H = I = 384: three 128-wide K blocks over four waves (one wave idle);
    # H = I = 128: a single block
    _check(synth.tiny_config(6, T=40, H=384, I=384, E=8, top_k=3))
    _check(synth.tiny_config(6, T=60, H=128, I=128, E=4, top_k=2))


@pytest.mark.parametrize("H,I", [(512, 1024), (1024, 512), (2048, 3072), (4096, 1536), (5120, 2048)])
def test_w8a16_streamed(dev, H, I):
    # K a multiple of 512 up to 4096 takes the streamed kernel (one piece of
    # K/4 bytes per wave and row, carrying its 128-wide block scales); K =
    # 5120 the skinny one
    cfg = synth.tiny_config(6, T=37, H=H, I=I, E=9, top_k=3)
    _check(cfg, inp=_scale_blocks(synth.make_inputs(cfg), cfg.wfmt, seed=H + I))


def test_w8a16_workload_full_size(dev):
    _check(synth.config(6))


def test_w8a16_large_batch_rejected(dev):
    cfg = synth.tiny_config(6, T=129, H=256, I=128, E=16, top_k=4)   # T*k = 516 > 32*E
    inp = synth.make_inputs(cfg)
    with pytest.raises(moe.MoeError) as ei:
        run_forward(cfg, inp)
    assert ei.value.status == 3   # MOE_ERR_UNSUPPORTED


# ---- MXFP4 weights (OCP MX E2M1 + E8M0 per 32), bf16 activations: the
# 16-row decode kernels up to 32 routed rows per expert, tiled above
@pytest.mark.parametrize("T", [1, 5, 16, 33, 128])
def test_mxfp4_small(dev, T):
    # T = 128: T * top_k = 512 = 32 * E, the largest batch of the decode kernels
    _check(synth.tiny_config(7, T=T, H=512, I=256, E=16, top_k=4))


def test_mxfp4_ragged_and_minimum_k(dev):
    # H = I = 384: three 128-wide blocks over four waves; H = I = 128: one
    _check(synth.tiny_config(7, T=40, H=384, I=384, E=8, top_k=3))
    _check(synth.tiny_config(7, T=60, H=128, I=128, E=4, top_k=2))


@pytest.mark.parametrize("H,I", [(512, 1024), (1536, 2048), (3072, 2560), (4096, 512), (5120, 1536), (7168, 3584)])
def test_mxfp4_streamed(dev, H, I):
    # K a multiple of 512: the streamed kernel splits K over two waves up to
    # 2048, four up to 4096 and eight up to 7168; every piece carries its
    # rows' E8M0 bytes (randomised here by up to 2^+-3)
    cfg = synth.tiny_config(7, T=37, H=H, I=I, E=9, top_k=3)
    _check(cfg, inp=_scale_blocks(synth.make_inputs(cfg), cfg.wfmt, seed=H + I))


def test_mxfp4_workload_full_size(dev):
    _check(synth.config(7))


@pytest.mark.parametrize("T", [129, 300, 1000])
def test_mxfp4_tiled(dev, T):
    # above 32 routed rows per expert: 128-row tiles, 128-element K steps, each
    # weight row's four E8M0 bytes per step (randomised here by up to 2^+-3)
    cfg = synth.tiny_config(7, T=T, H=512, I=256, E=16, top_k=4)
    a = moe.make_args(cfg.T, cfg.H, cfg.E, cfg.I, cfg.top_k, wfmt=cfg.wfmt)
    assert moe.moe_workspace_layout(a)["block_m"] == 128
    _check(cfg, inp=_scale_blocks(synth.make_inputs(cfg), cfg.wfmt, seed=T))


def test_mxfp4_tiled_ragged_and_minimum_k(dev):
    # H = I = 384: three K steps and H % 256 != 0 (128-wide GEMM2 tiles);
    # H = I = 128: a single K step
    _check(synth.tiny_config(7, T=300, H=384, I=384, E=8, top_k=3))
    _check(synth.tiny_config(7, T=400, H=128, I=128, E=4, top_k=2))


def test_mxfp4_prefill_workload_full_size(dev):
    _check(synth.config(8))


# ---- MXFP4 weights x MXFP8 activations (OCP MX on both operands): the
# block-scaled fp8 x fp4 matrix instruction, tiled kernels at every batch
def _mx8_layer(cfg, inp):
    out, ws, L, _ = run_forward(cfg, inp)
    return ws, L


def test_mxfp8_act_quant_bit_exact_crafted(dev):
    # the worked blocks of the oracle's pin (ties, saturation, zero block, an
    # fp32-subnormal amax), fed as bf16 hidden rows through the layer's own
    # quantiser: codes and E8M0 bytes bit-exact
    cfg = synth.tiny_config(9, T=4, H=128, I=128, E=4, top_k=2)
    inp = synth.make_inputs(cfg)
    x = np.zeros((4, 128), np.float32)
    x[0, :5] = [1.0, -0.5, 17 / 256, 2.0 ** -17, 2.0 ** -18]
    x[0, 32:35] = [1.875, -1.75, 1.8125]
    x[0, 96], x[0, 97] = 3.0 * 2 ** 20, -(2.0 ** 5)
    x[1, 0] = 2.0 ** -130
    x[2] = np.linspace(-3, 3, 128)
    x[3] = np.random.default_rng(1).standard_normal(128) * 1e-3
    inp["hidden"] = _bf16(x)
    assert O.bf16_to_f64(inp["hidden"])[1, 0] == 2.0 ** -130
    out, ws, L, _ = run_forward(cfg, inp)
    q = ws_view(ws, L, "act_q", torch.uint8, cfg.T * cfg.H).reshape(cfg.T, cfg.H)
    sx = ws_view(ws, L, "act_s", torch.uint8, cfg.T * cfg.H // 32).reshape(cfg.T, cfg.H // 32)
    rq, rsx = O.act_quant_mxfp8(O.bf16_to_f64(inp["hidden"]).astype(np.float32))
    assert np.array_equal(sx, rsx)
    assert np.array_equal(q, rq)


@pytest.mark.parametrize("T", [1, 33, 200, 700])
def test_mxfp4x8_small(dev, T):
    _check(synth.tiny_config(9, T=T, H=512, I=1024, E=16, top_k=4))


def test_mxfp4x8_ragged_and_minimum_k(dev):
    # H = I = 384: three K steps, H % 256 != 0 (128-wide GEMM2 tiles);
    # H = I = 128: a single K step (I = 128 so the tolerance is looser in
    # practice: one intermediate code step weighs more)
    _check(synth.tiny_config(9, T=300, H=384, I=1152, E=8, top_k=3))
    _check(synth.tiny_config(9, T=400, H=128, I=1024, E=4, top_k=2))


def test_mxfp4x8_block_scales_vary(dev):
    cfg = synth.tiny_config(9, T=100, H=512, I=1024, E=8, top_k=2)
    _check(cfg, inp=_scale_blocks(synth.make_inputs(cfg), cfg.wfmt, seed=9))


def test_mxfp4x8_intermediate_codes(dev):
    """The MXFP8 intermediate GEMM1 writes (e4m3 codes + E8M0 bytes per (row,
    32 of I)) against the oracle's quantiser on its own fp32 intermediate.
    The kernel's intermediate differs from the oracle's by ~1e-5 relative
    (fp32 accumulation order), so: every E8M0 byte equal, except where the
    block's amax lies within 2e-4 of a power of two (then one step either
    way); where the bytes agree, every code the rounding of a value within
    2e-4 * 448 (in scale units) of the oracle's a / X."""
    cfg = synth.tiny_config(9, T=700, H=512, I=512, E=16, top_k=4)
    inp = synth.make_inputs(cfg)
    out, ws, L, _ = run_forward(cfg, inp)
    n, I, cap = cfg.T * cfg.top_k, cfg.I, L["cap"]
    sid = ws_view(ws, L, "sorted_ids", torch.int32, cap)
    codes = ws_view(ws, L, "inter", torch.uint8, cap * I).reshape(cap, I)
    sbytes = ws_view(ws, L, "inter_s", torch.uint8, cap * (I // 32)).reshape(cap, I // 32)
    rows = np.nonzero(sid < n)[0]
    a32 = _oracle_preq_intermediate(cfg, inp)[sid[rows]]
    qref, sref = O.act_quant_mxfp8(a32)
    sg = sbytes[rows]
    amax = np.abs(a32.astype(np.float64)).reshape(-1, I // 32, 32).max(axis=2)
    frac = amax / np.exp2(np.floor(np.log2(np.maximum(amax, 1e-300))))   # in [1, 2)
    near = (frac < 1 + 2e-4) | (frac > 2 - 4e-4)
    assert np.all((sg == sref) | (near & (np.abs(sg.astype(int) - sref.astype(int)) == 1)))
    same = np.repeat(sg == sref, 32, axis=1)
    X = np.repeat(O.e8m0_value(sref), 32, axis=1)
    x = a32.astype(np.float64) / X
    slack = 2e-4 * O.E4M3_MAX
    v_lo = O.e4m3_decode(O.e4m3_encode(x - slack))
    v_hi = O.e4m3_decode(O.e4m3_encode(x + slack))
    v_g = O.e4m3_decode(codes[rows])
    ok = ~same | ((v_g >= v_lo) & (v_g <= v_hi))
    bad = np.argwhere(~ok)
    assert bad.size == 0, (bad[:3], x[tuple(bad[0])], v_g[tuple(bad[0])])
    ties = int((codes[rows] != qref).sum())
    print(f"  {ties} of {qref.size} codes and {int((sg != sref).sum())} scale bytes differ by a tie", flush=True)
    assert ties <= 0.01 * qref.size


def test_mxfp4x8_prefill_workload_full_size(dev):
    _check(synth.config(9))
