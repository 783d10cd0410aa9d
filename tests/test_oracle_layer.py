"""Pins of the oracle's whole layer: a hand-worked example, the dense SwiGLU
special case against torch, identical-expert and token-order invariants, and a
per-token brute force over every expert on tiny shapes."""
import dataclasses
import math

import numpy as np
import pytest
import torch

import synth
from oracle import moe_oracle as O


def _bits(x):
    return O.f32_to_bf16_rne(np.asarray(x, dtype=np.float32))


def _sig(x):
    return 1 / (1 + math.exp(-x))


def test_worked_two_expert_example():
    """H=2, I=1, E=2.  Gate rows [0,I) of W1 and up rows [I,2I) are asymmetric,
    so a gate/up swap, a transposed W2 or a dropped SiLU all change the result."""
    cfg = synth.MoeConfig("worked", T=2, H=2, E=2, I=1, top_k=1)
    inputs = {
        "hidden": _bits([[1.0, 2.0], [0.5, -1.0]]),
        "logits": np.array([[1.0, 0.0], [0.0, 1.0]], np.float32),
        "sel_bias": None,
        "w1": _bits([[[1.0, 0.0], [0.0, 1.0]], [[0.0, -1.0], [2.0, 0.0]]]),
        "w2": _bits([[[1.0], [-2.0]], [[3.0], [0.5]]]),
        "w1_scale": None, "w2_scale": None,
    }
    r = O.forward(cfg, inputs, mirror=False)
    s1 = _sig(1.0)
    # token 0 -> expert 0: g = 1, u = 2, a = 2*sigmoid(1); y = [a, -2a]
    # token 1 -> expert 1: g = 1, u = 1, a = sigmoid(1);  y = [3a, a/2]
    want = np.array([[2 * s1, -4 * s1], [3 * s1, 0.5 * s1]])
    assert r["ids"].tolist() == [[0], [1]]
    assert np.allclose(r["out"], want, rtol=0, atol=1e-15)
    # top-2: token 0 mixes both experts with weights sigmoid(1), sigmoid(-1)
    cfg2 = synth.MoeConfig("worked2", T=2, H=2, E=2, I=1, top_k=2)
    r2 = O.forward(cfg2, inputs, mirror=False)
    x0 = np.array([1.0, 2.0])
    a1 = (lambda g, u: g * _sig(g) * u)(-2.0, 2.0)          # expert 1 on token 0
    y1 = np.array([3 * a1, 0.5 * a1])
    y0 = np.array([2 * s1, -4 * s1])
    assert np.allclose(r2["out"][0], s1 * y0 + _sig(-1.0) * y1, rtol=0, atol=1e-15)
    del x0


def _dense_torch(x, w1, w2, round_intermediate=False):
    x, w1, w2 = (torch.from_numpy(np.asarray(v, np.float64)) for v in (x, w1, w2))
    I = w1.shape[0] // 2
    a = torch.nn.functional.silu(x @ w1[:I].T) * (x @ w1[I:].T)
    if round_intermediate:
        a = a.to(torch.float32).to(torch.bfloat16).to(torch.float64)
    return (a @ w2.T).numpy()


@pytest.mark.parametrize("mirror", [False, True])
def test_single_expert_top1_is_dense_swiglu(mirror):
    cfg = synth.MoeConfig("dense", T=33, H=256, E=1, I=128, top_k=1, seed=11)
    inp = synth.make_inputs(cfg)
    r = O.forward(cfg, inp, mirror=mirror)
    x = O.bf16_to_f64(inp["hidden"])
    ref = _dense_torch(x, O.bf16_to_f64(inp["w1"][0]), O.bf16_to_f64(inp["w2"][0]), mirror)
    rms = np.sqrt((ref ** 2).mean())
    # unmirrored: identical math; mirrored: a bf16 tie may round the other way
    tol = 1e-12 if not mirror else 2 ** -8
    assert np.max(np.abs(r["out"] - ref)) <= tol * rms
    assert np.all(r["w"] == 1.0)


@pytest.mark.parametrize("mirror", [False, True])
def test_fp8_weights_bf16_activations_single_expert(mirror):
    # the weight-only fp8 route: E = 1, k = 1 is a dense SwiGLU on the exactly
    # dequantised fp8 weights with the hidden rows unquantised -- operands
    # built here with torch's own float8_e4m3fn decode
    cfg = synth.MoeConfig("dense8", T=33, H=256, E=1, I=128, top_k=1, wfmt="fp8a16", seed=12)
    inp = synth.make_inputs(cfg)
    r = O.forward(cfg, inp, mirror=mirror)

    def deq(codes, s):
        q = torch.from_numpy(np.ascontiguousarray(codes)).view(torch.float8_e4m3fn).to(torch.float64)
        sc = torch.from_numpy(s).to(torch.float64).repeat_interleave(128, 0).repeat_interleave(128, 1)
        return (q * sc).numpy()

    x = torch.from_numpy(inp["hidden"].view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    ref = _dense_torch(x, deq(inp["w1"][0], inp["w1_scale"][0]), deq(inp["w2"][0], inp["w2_scale"][0]), mirror)
    rms = np.sqrt((ref ** 2).mean())
    tol = 1e-12 if not mirror else 2 ** -8
    assert np.max(np.abs(r["out"] - ref)) <= tol * rms


@pytest.mark.parametrize("mirror", [False, True])
def test_mxfp4_weights_single_expert(mirror):
    # MXFP4 weights with bf16 activations: E = 1, k = 1 is a dense SwiGLU on
    # weights decoded here from the OCP E2M1 table and torch's E8M0 cast
    cfg = synth.MoeConfig("dense4", T=33, H=256, E=1, I=128, top_k=1, wfmt="mxfp4", seed=13)
    inp = synth.make_inputs(cfg)
    r = O.forward(cfg, inp, mirror=mirror)
    e2m1 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0, -0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0])

    def deq(packed, s):
        codes = np.stack([packed & 0xF, packed >> 4], axis=-1).reshape(packed.shape[0], -1)
        sc = torch.from_numpy(np.ascontiguousarray(s)).view(torch.float8_e8m0fnu).to(torch.float64).numpy()
        return e2m1[codes] * np.repeat(sc, 32, axis=1)

    x = torch.from_numpy(inp["hidden"].view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    ref = _dense_torch(x, deq(inp["w1"][0], inp["w1_scale"][0]), deq(inp["w2"][0], inp["w2_scale"][0]), mirror)
    rms = np.sqrt((ref ** 2).mean())
    tol = 1e-12 if not mirror else 2 ** -8
    assert np.max(np.abs(r["out"] - ref)) <= tol * rms


@pytest.mark.parametrize("mirror", [False, True])
def test_mxfp4_weights_mxfp8_activations_single_expert(mirror):
    # MXFP4 weights with MXFP8 activations: E = 1, k = 1 is a dense SwiGLU.
    # Unmirrored it is exactly the MXFP4 layer with bf16 activations.
    # Mirrored: the hidden rows and the fp32 intermediate each go through the
    # (separately pinned) MXFP8 quantiser, their codes decoded here through
    # torch's e4m3 and E8M0 casts, the weights through the OCP E2M1 table
    cfg = synth.MoeConfig("dense48", T=33, H=256, E=1, I=128, top_k=1, wfmt="mxfp4x8", seed=14)
    inp = synth.make_inputs(cfg)
    r = O.forward(cfg, inp, mirror=mirror)
    if not mirror:
        r4 = O.forward(dataclasses.replace(cfg, wfmt="mxfp4"), inp, mirror=False)
        assert np.array_equal(r["out"], r4["out"])
        return
    e2m1 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0, -0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0])

    def deq_w(packed, s):
        codes = np.stack([packed & 0xF, packed >> 4], axis=-1).reshape(packed.shape[0], -1)
        sc = torch.from_numpy(np.ascontiguousarray(s)).view(torch.float8_e8m0fnu).to(torch.float64)
        return torch.from_numpy(e2m1[codes]) * sc.repeat_interleave(32, 1)

    def mx_round(v):
        q, sb = O.act_quant_mxfp8(np.asarray(v, np.float32))
        qv = torch.from_numpy(q).view(torch.float8_e4m3fn).to(torch.float64)
        return qv * torch.from_numpy(sb).view(torch.float8_e8m0fnu).to(torch.float64).repeat_interleave(32, 1)

    x = torch.from_numpy(inp["hidden"].view(np.int16)).view(torch.bfloat16).to(torch.float64)
    w1, w2 = deq_w(inp["w1"][0], inp["w1_scale"][0]), deq_w(inp["w2"][0], inp["w2_scale"][0])
    xq = mx_round(x.numpy().astype(np.float32))
    a = torch.nn.functional.silu(xq @ w1[:cfg.I].T) * (xq @ w1[cfg.I:].T)
    ref = (mx_round(a.numpy().astype(np.float32)) @ w2.T).numpy()
    rms = np.sqrt((ref ** 2).mean())
    # a tie of the intermediate's rounding may go the other way (one e4m3 step)
    assert np.max(np.abs(r["out"] - ref)) <= 2 ** -4 * rms
    assert np.mean(np.abs(r["out"] - ref)) <= 1e-10 * rms


@pytest.mark.parametrize("n", [1, 4, 5, 6, 7, 9])
def test_identical_experts_any_routing(n):
    cfg = synth.tiny_config(n)
    inp = synth.make_inputs(cfg, identical_experts=True)
    r = O.forward(cfg, inp, mirror=False)
    w1 = O.dequant_weight(cfg.wfmt, inp["w1"][0], None if inp["w1_scale"] is None else inp["w1_scale"][0])
    w2 = O.dequant_weight(cfg.wfmt, inp["w2"][0], None if inp["w2_scale"] is None else inp["w2_scale"][0])
    ref = cfg.routed_scale * _dense_torch(O.bf16_to_f64(inp["hidden"]), w1, w2)
    assert np.max(np.abs(r["out"] - ref)) <= 1e-12 * np.sqrt((ref ** 2).mean())


@pytest.mark.parametrize("n", [1, 4, 5, 6, 7, 9])
def test_token_order_invariance(n):
    cfg = synth.tiny_config(n)
    inp = synth.make_inputs(cfg)
    perm = np.random.default_rng(7).permutation(cfg.T)
    inp2 = dict(inp, hidden=inp["hidden"][perm], logits=inp["logits"][perm])
    r1 = O.forward(cfg, inp)
    r2 = O.forward(cfg, inp2)
    assert np.array_equal(r2["ids"], r1["ids"][perm])
    rms = np.sqrt((r1["out"] ** 2).mean())
    assert np.max(np.abs(r2["out"] - r1["out"][perm])) <= 1e-12 * rms


def _brute_layer(cfg, inp, mirror):
    """Per token: evaluate EVERY expert on the token, then pick the top-k by a
    scan and weight-sum them in slot order.  Shares only the codecs."""
    outs = []
    lg = inp["logits"].astype(np.float64)
    b = np.zeros(cfg.E) if inp["sel_bias"] is None else inp["sel_bias"].astype(np.float64)
    ws = [(O.dequant_weight(cfg.wfmt, inp["w1"][e], None if inp["w1_scale"] is None else inp["w1_scale"][e]),
           O.dequant_weight(cfg.wfmt, inp["w2"][e], None if inp["w2_scale"] is None else inp["w2_scale"][e]))
          for e in range(cfg.E)]
    for t in range(cfg.T):
        x = O.activation_operand(inp["hidden"][t:t + 1], cfg.wfmt, mirror)[0]
        ys = []
        for w1, w2 in ws:
            g = np.array([np.dot(w1[i], x) for i in range(cfg.I)])
            u = np.array([np.dot(w1[cfg.I + i], x) for i in range(cfg.I)])
            a = g * (1 / (1 + np.exp(-g))) * u
            if mirror:
                a = O._round_intermediate(a[None, :], cfg.wfmt)[0]
            ys.append(np.array([np.dot(w2[h], a) for h in range(cfg.H)]))
        if cfg.mode == "softmax":
            key = lg[t] + b
        else:
            sc = 1 / (1 + np.exp(-lg[t]))
            key = sc + b
        chosen = []
        for _ in range(cfg.top_k):
            best = max((e for e in range(cfg.E) if e not in chosen), key=lambda e: (key[e], -e))
            chosen.append(best)
        if cfg.mode == "softmax":
            z = np.exp(np.array([lg[t][e] for e in chosen]) - max(lg[t][e] for e in chosen))
            w = z / z.sum()
        else:
            s = np.array([sc[e] for e in chosen])
            w = s / s.sum()
        w = w * cfg.routed_scale
        outs.append(sum(w[j] * ys[chosen[j]] for j in range(cfg.top_k)))
    return np.array(outs)


@pytest.mark.parametrize("n", [1, 4, 5, 6, 7, 9])
@pytest.mark.parametrize("mirror", [False, True])
def test_brute_force_tiny(n, mirror):
    cfg = synth.tiny_config(n, T=9, H=256, I=128, E=6, top_k=3)
    inp = synth.make_inputs(cfg)
    r = O.forward(cfg, inp, mirror=mirror)
    ref = _brute_layer(cfg, inp, mirror)
    rms = np.sqrt((ref ** 2).mean())
    assert np.max(np.abs(r["out"] - ref)) <= 1e-12 * rms


def test_token_subset_matches_full():
    cfg = synth.tiny_config(4)
    inp = synth.make_inputs(cfg)
    full = O.forward(cfg, inp)
    tok = np.array([5, 0, cfg.T - 1, 17])
    sub = O.forward(cfg, inp, tokens=tok)
    assert np.array_equal(sub["ids"], full["ids"][tok])
    assert np.allclose(sub["out"], full["out"][tok], rtol=0, atol=1e-12)
