"""Pins of the oracle's storage codecs (bf16, OCP e4m3fn, packed int4) and of
its weight dequantisation, against published tables, hand-derived rounding
cases and an independent implementation (torch's CPU casts)."""
import math
import os

import numpy as np
import pytest
import torch

from oracle import moe_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                yield line.split()


def test_e4m3_decode_matches_ocp_table():
    for code, val, *_ in _rows("e4m3_ocp_table.txt"):
        got = O.e4m3_decode(np.array([int(code, 16)]))[0]
        if val == "nan":
            assert math.isnan(got), code
        else:
            assert got == float(val) and math.copysign(1, got) == math.copysign(1, float(val)), code


def test_e4m3_decode_all_codes_vs_torch():
    codes = np.arange(256, dtype=np.uint8)
    ours = O.e4m3_decode(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])
    assert nan.sum() == 2  # only S.1111.111


def test_e4m3_encode_hand_rounding_cases():
    for x, code, *_ in _rows("e4m3_rounding.txt"):
        assert O.e4m3_encode(np.array([float(x)]))[0] == int(code, 16), x


def test_e4m3_encode_roundtrip_every_finite_code():
    codes = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], dtype=np.uint8)
    vals = O.e4m3_decode(codes)
    assert np.array_equal(O.e4m3_encode(vals), codes)


def test_e4m3_encode_dense_sweep_vs_torch():
    rng = np.random.default_rng(0)
    # every fp32 value on a fine grid across all binades, plus exact midpoints
    grid = O.e4m3_decode(np.arange(0, 0x7F, dtype=np.uint8))
    mids = (grid[:-1] + grid[1:]) / 2
    x = np.concatenate([
        np.ldexp(rng.uniform(1, 2, 200000), rng.integers(-12, 9, 200000)),
        rng.uniform(0, 448, 200000), mids, grid,
    ]).astype(np.float32)
    x = np.concatenate([x, -x])
    x = x[np.abs(x) <= 448]
    ours = O.e4m3_encode(x)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(ours, ref)


def test_bf16_rne_hand_cases():
    for xin, want, *_ in _rows("bf16_rounding.txt"):
        x = np.array([int(xin, 16)], dtype=np.uint32).view(np.float32)
        assert O.f32_to_bf16_rne(x)[0] == int(want, 16), xin


def test_bf16_rne_sweep_vs_torch_and_exact_decode():
    rng = np.random.default_rng(1)
    bits = rng.integers(0, 2 ** 32, 400000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[np.isfinite(x)]
    ours = O.f32_to_bf16_rne(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    # decode is exact: every bf16 value is an fp32 value with 16 zero low bits
    dec = O.bf16_to_f64(ours)
    assert np.array_equal(dec.astype(np.float32).view(np.uint32) & 0xFFFF, np.zeros_like(ours, dtype=np.uint32))


def test_int4_unpack_hand_cases():
    for word, *elems in _rows("int4_packing.txt"):
        w = np.array([int(word, 16)], dtype=np.uint32).view(np.int32)
        assert O.int4_unpack(w).tolist() == [int(e) for e in elems], word


def test_int4_pack_unpack_roundtrip():
    rng = np.random.default_rng(2)
    q = rng.integers(-8, 8, (5, 64)).astype(np.int64)
    words = np.zeros((5, 8), dtype=np.uint32)
    for j in range(8):
        words |= (q[:, j::8] & 0xF).astype(np.uint32) << np.uint32(4 * j)
    assert np.array_equal(O.int4_unpack(words.view(np.int32)), q)


def test_fp8_block_dequant_scale_orientation():
    # [N=256, K=384] all codes 1.0; block scales differ along both axes
    w = np.full((256, 384), 0x38, dtype=np.uint8)
    s = np.array([[1, 2, 3], [10, 20, 30]], dtype=np.float32)  # [N/128, K/128]
    d = O.dequant_weight("fp8", w, s)
    assert d[0, 0] == 1 and d[0, 200] == 2 and d[0, 300] == 3
    assert d[200, 0] == 10 and d[200, 383] == 30 and d[127, 255] == 2 and d[128, 255] == 20


def test_int4_group_dequant():
    # [N=2, K=256]: element (n,k) = q * s[n, k // 128]
    q = np.zeros((2, 256), dtype=np.int64)
    q[0, 3], q[1, 130], q[1, 255] = -8, 7, -1
    words = np.zeros((2, 32), dtype=np.uint32)
    for j in range(8):
        words |= (q[:, j::8] & 0xF).astype(np.uint32) << np.uint32(4 * j)
    s = O.f32_to_bf16_rne(np.array([[0.5, 2.0], [0.25, 3.0]], dtype=np.float32))
    d = O.dequant_weight("int4", words.view(np.int32), s)
    assert d[0, 3] == -4.0 and d[1, 130] == 21.0 and d[1, 255] == -3.0
    assert np.count_nonzero(d) == 3


def test_act_quant_worked_groups():
    x = np.zeros((3, 256), dtype=np.float32)
    # group (0,0): amax = 448 -> scale exactly 1, on-grid values stay exact
    x[0, :4] = [448.0, -1.0, 0.015625, 240.0]
    # group (0,1): all zero -> scale 1e-10/448, codes 0
    # group (1,0): amax 1 -> the max element hits the top code 0x7E
    x[1, 5] = 1.0
    x[1, 6] = -0.5
    # group (2,1): halfway case after scaling by s = 2 (amax 896)
    x[2, 128] = 896.0
    x[2, 129] = 2.0 * 1.0625     # -> 1.0625 -> ties to 1.0
    codes, s = O.act_quant_fp8(x)
    assert s[0, 0] == 1.0 and s[2, 1] == 2.0
    assert s[0, 1] == np.float32(np.float32(1e-10) / np.float32(448.0))
    assert codes[0, :4].tolist() == [0x7E, 0xB8, 0x08, 0x77]
    assert np.all(codes[0, 128:] == 0)
    assert codes[1, 5] == 0x7E
    assert codes[2, 128] == 0x7E and codes[2, 129] == 0x38
    dq = O.act_dequant_fp8(codes, s)
    assert dq[0, 0] == 448.0 and dq[2, 129] == 2.0
    # every element is within half a grid step (relative 1/16) of its input
    nz = x != 0
    assert np.all(np.abs(dq[nz] - x[nz]) <= np.abs(x[nz]) / 16 + 1e-12)


# ---------------------------------------------------------------- MXFP4 (OCP MX)
def _e2m1_golden():
    rows = [r for r in _rows("e2m1_ocp_table.txt") if r[0] != "e8m0"]
    return {int(c, 16): float(v) for c, v in rows}


def test_e2m1_decode_matches_ocp_table():
    table = _e2m1_golden()
    assert len(table) == 16
    # every code in the low and in the high nibble, scale 2^0
    for code, val in table.items():
        packed = np.full((1, 16), code | (code << 4), np.uint8)
        got = O.dequant_weight("mxfp4", packed, np.array([[127]], np.uint8))
        assert np.all(got == val) and np.all(np.signbit(got) == (math.copysign(1, val) < 0)), code


def test_e8m0_matches_table_and_torch():
    for r in _rows("e2m1_ocp_table.txt"):
        if r[0] != "e8m0":
            continue
        got = O.e8m0_value(np.array([int(r[1])]))[0]
        assert (math.isnan(got) and r[2] == "nan") or got == float(r[2]), r
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e8m0fnu).to(torch.float64).numpy()
    ours = O.e8m0_value(codes)
    assert np.array_equal(np.isnan(ours), np.isnan(ref)) and np.isnan(ref).sum() == 1
    assert np.array_equal(ours[:255], ref[:255])


def test_mxfp4_nibble_order_and_block_scales():
    # byte 0x21: element 0 is the low nibble (code 1 = 0.5), element 1 the high (code 2 = 1.0)
    packed = np.zeros((2, 32), np.uint8)
    packed[0, 0] = 0x21
    packed[1, 20] = 0xF7          # elements 40 (6.0) and 41 (-6.0), in the second block
    scale = np.array([[127, 130], [125, 124]], np.uint8)
    w = O.dequant_weight("mxfp4", packed, scale)
    table = _e2m1_golden()
    expect = np.zeros((2, 64))
    for n in range(2):
        for k in range(64):
            b = int(packed[n, k // 2])
            code = (b >> 4) if k % 2 else (b & 0xF)
            expect[n, k] = table[code] * 2.0 ** (int(scale[n, k // 32]) - 127)
    assert np.array_equal(w, expect)
    assert w[0, 0] == 0.5 and w[0, 1] == 1.0 and w[1, 40] == 6.0 * 2.0 ** -3 and w[1, 41] == -6.0 * 2.0 ** -3


def test_mxfp4_storage_encoder_roundtrip():
    from synth import moe_inputs as M
    rng = np.random.default_rng(5)
    grid = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])
    # blocks whose amax is exactly 4 * 2^e (so X = 2^e) with every element on the grid
    v = rng.choice(grid, size=(3, 96)) * rng.choice([-1.0, 1.0], size=(3, 96))
    v[:, ::32] = 4.0
    ex = rng.integers(-6, 6, size=(3, 3))
    w = (v.reshape(3, 3, 32) * np.ldexp(1.0, ex)[:, :, None]).reshape(3, 96).astype(np.float32)
    packed, scale = M._mxfp4_quant(w)
    assert np.array_equal(scale, (ex + 127).astype(np.uint8))
    assert np.array_equal(O.dequant_weight("mxfp4", packed, scale), w.astype(np.float64))


# ---------------------------------------------------------------- MXFP8 activations (OCP MX)
def test_mxfp8_quant_worked_blocks():
    # OCP MX v1.0 conversion: X = 2^(floor(log2 amax) - emax), emax = 8 for
    # e4m3 (its largest power of two is 2^8), elements e4m3(x / X), saturated
    x = np.zeros((2, 128), np.float32)
    # block (0,0): amax 1 -> X = 2^-8 (byte 119); 17/256 -> 17 is a tie
    # between 16 and 18 -> even mantissa 16; 2^-17 -> 2^-9 (smallest
    # subnormal); 2^-18 -> 2^-10, a tie between 0 and 2^-9 -> 0
    x[0, :5] = [1.0, -0.5, 17 / 256, 2.0 ** -17, 2.0 ** -18]
    # block (0,1): amax 1.875 -> X = 2^-8; 480 saturates to 448; 464 is a tie
    # between 448 and 480 -> 448 (even mantissa)
    x[0, 32:35] = [1.875, -1.75, 1.8125]
    # block (0,2): all zero -> byte 0, codes 0
    # block (0,3): amax 3 * 2^20 -> X = 2^13 (byte 140): 384 -> 0x7C; -2^5 -> -2^-8
    x[0, 96], x[0, 97] = 3.0 * 2 ** 20, -(2.0 ** 5)
    # block (1,0): amax 2^-130 (an fp32 subnormal): the exponent clamps at
    # 2^-127 (byte 0) and x / X = 2^-3 is still exact
    x[1, 0] = 2.0 ** -130
    q, s = O.act_quant_mxfp8(x)
    assert s.dtype == np.uint8 and s.shape == (2, 4)
    assert s[0].tolist() == [119, 119, 0, 140] and s[1, 0] == 0
    assert q[0, :5].tolist() == [0x78, 0xF0, 0x58, 0x01, 0x00]
    assert q[0, 32:35].tolist() == [0x7E, 0xFE, 0x7E]
    assert np.all(q[0, 64:96] == 0)
    assert q[0, 96] == 0x7C and q[0, 97] == 0x82
    assert q[1, 0] == 0x20
    d = O.act_dequant_mxfp8(q, s)
    assert d[0, 0] == 1.0 and d[0, 32] == 1.75 and d[0, 96] == 3.0 * 2 ** 20 and d[1, 0] == 2.0 ** -130


def test_mxfp8_quant_sweep_vs_torch():
    # rows of mixed magnitudes: the scale byte is the one power of two with
    # amax / X in [256, 512) (checked from the byte alone), and every element
    # is torch's float8_e4m3fn cast of x / X clamped to +-448; decode through
    # torch's E8M0 and e4m3 casts
    rng = np.random.default_rng(5)
    x = (rng.standard_normal((64, 1024)) * np.exp2(rng.integers(-30, 30, (64, 1)))).astype(np.float32)
    x[3, 64:96] = 0.0
    x[5, :32] *= 1e-30
    q, s = O.act_quant_mxfp8(x)
    X = torch.from_numpy(s.copy()).view(torch.float8_e8m0fnu).to(torch.float64).numpy()
    amax = np.abs(x.astype(np.float64)).reshape(64, 32, 32).max(axis=2)
    nz = amax > 0
    assert np.all((amax[nz] / X[nz] >= 256) & (amax[nz] / X[nz] < 512))
    assert np.all(s[~nz] == 0)
    y = x.astype(np.float64).reshape(64, 32, 32) / X[:, :, None]
    want = torch.from_numpy(np.clip(y, -448, 448).reshape(64, 1024)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(q, want)
    d = O.act_dequant_mxfp8(q, s)
    dq = torch.from_numpy(q.copy()).view(torch.float8_e4m3fn).to(torch.float64).numpy() * np.repeat(X, 32, axis=1)
    assert np.array_equal(d, dq)
    # within half a step (1/16 relative for normal elements, 2^-10 X below),
    # except where the rule's scale leaves |x| / X above 448: saturation
    err = np.abs(d - x.astype(np.float64))
    Xr = np.repeat(X, 32, axis=1)
    sat = np.abs(x) - 448 * Xr
    assert np.all(err <= np.maximum(np.maximum(np.abs(x) / 16, Xr * 2.0 ** -10), sat) + 1e-300)
    assert np.any(sat > np.abs(x) / 16)    # the sweep does reach the saturated range


def test_mxfp8_blocks_are_independent():
    # one element changed in block j changes only block j's scale and codes
    rng = np.random.default_rng(9)
    x = rng.standard_normal((1, 256)).astype(np.float32)
    q0, s0 = O.act_quant_mxfp8(x)
    x2 = x.copy()
    x2[0, 100] = 1000.0                    # block 3
    q1, s1 = O.act_quant_mxfp8(x2)
    assert np.array_equal(np.nonzero(s0[0] != s1[0])[0], [3])
    changed = np.nonzero(q0[0] != q1[0])[0]
    assert changed.size > 0 and np.all((changed >= 96) & (changed < 128))
