"""Pins of the oracle's router GEMM (the logits in front of the MoE Gate):
a hand-worked example, one-hot router rows that must pick hidden columns
exactly, and an exact rational brute force on random bf16 inputs."""
import os
import struct
from fractions import Fraction

import numpy as np

from oracle import moe_oracle as O
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "router_worked_example.txt")


def _bits(vals):
    """Exact decimal values -> bf16 bit patterns (values must be bf16-exact)."""
    out = []
    for v in vals:
        b = struct.unpack("<I", struct.pack("<f", float(v)))[0]
        assert b & 0xFFFF == 0, v
        out.append(b >> 16)
    return np.array(out, dtype=np.uint16)


def _value(bits16):
    """bf16 bits -> exact Fraction (decoded independently of the oracle)."""
    return Fraction(struct.unpack("<f", struct.pack("<I", int(bits16) << 16))[0])


def _golden():
    rows = {}
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        key, *vals = line.split()
        rows.setdefault(key, []).append([float(v) for v in vals])
    return {k: np.array(v) for k, v in rows.items()}


def test_router_worked_example():
    g = _golden()
    hid = np.stack([_bits(r) for r in g["hidden"]])
    wr = np.stack([_bits(r) for r in g["w_router"]])
    lg = O.router_logits(hid, wr)
    assert np.array_equal(lg, g["logits"])
    ids, _ = O.gate(lg.astype(np.float32), None, 2, "softmax", True, 1.0)
    assert np.array_equal(ids, g["top2"].astype(np.int32))


def test_router_one_hot_rows_pick_hidden_columns():
    cfg = synth.tiny_config(1, T=9, H=256, E=8)
    hid = synth.make_routing_inputs(cfg)["hidden"]
    cols = np.array([0, 5, 255, 17, 128, 5, 64, 200])
    vals = [1.0, -1.0, 2.0, 0.5, -4.0, 1.0, 0.125, 3.0]
    wr = np.zeros((8, 256), dtype=np.uint16)
    for e, (c, v) in enumerate(zip(cols, vals)):
        wr[e, c] = _bits([v])[0]
    lg = O.router_logits(hid, wr)
    x = O.bf16_to_f64(hid)
    assert np.array_equal(lg, x[:, cols] * np.array(vals)[None, :])


def test_router_exact_rational_brute_force():
    rng = np.random.default_rng(7)
    T, E, H = 3, 5, 24
    hid = synth.moe_inputs._bf16_bits(rng.standard_normal((T, H)).astype(np.float32))
    wr = synth.moe_inputs._bf16_bits((rng.standard_normal((E, H)) / np.sqrt(H)).astype(np.float32))
    lg = O.router_logits(hid, wr)
    for t in range(T):
        for e in range(E):
            exact = sum(_value(hid[t, h]) * _value(wr[e, h]) for h in range(H))
            mag = sum(abs(_value(hid[t, h]) * _value(wr[e, h])) for h in range(H))
            # float64 sums of H exact products: within H * 2^-53 of the magnitude
            assert abs(Fraction(lg[t, e]) - exact) <= Fraction(H, 2 ** 53) * mag


def test_router_weights_recipe():
    cfg = synth.tiny_config(2, T=64, H=1024, E=16)
    w = O.bf16_to_f64(synth.make_router_weights(cfg))
    assert w.shape == (16, 1024)
    # N(0, 1/H): the sample variance of 16k draws is within 5 % of 1/H
    assert abs(w.var() * 1024 - 1.0) < 0.05
    assert np.array_equal(synth.make_router_weights(cfg), synth.make_router_weights(cfg))
