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
from tests.gpu_util import TOL, rel_err, require_gpu, run_forward, ws_view

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
    _act_quant_check(_bf16(x))


def test_act_quant_bit_exact_fp8_workload_rows(dev):
    r = synth.make_routing_inputs(synth.tiny_config(4, T=777, H=7168))
    _act_quant_check(r["hidden"])


def _check(cfg, inp=None, tokens=None):
    print(f"forward parity {cfg}", flush=True)
    inp = synth.make_inputs(cfg) if inp is None else inp
    out, ws, L, _ = run_forward(cfg, inp)
    n = cfg.T * cfg.top_k
    ids = ws_view(ws, L, "topk_ids", torch.int32, n).reshape(cfg.T, cfg.top_k)
    rid, _ = O.gate(inp["logits"], inp["sel_bias"], cfg.top_k, cfg.mode, cfg.renormalize, cfg.routed_scale)
    assert np.array_equal(ids, rid)
    ro, rs, ri = O.permute(rid, cfg.E, L["block_m"])
    assert np.array_equal(ws_view(ws, L, "expert_offsets", torch.int32, cfg.E + 1), ro)
    assert np.array_equal(ws_view(ws, L, "sorted_ids", torch.int32, L["cap"]), rs)
    assert np.array_equal(ws_view(ws, L, "inv_pos", torch.int32, n), ri)
    if cfg.wfmt == "fp8":   # the layer's own activation quantisation, bit-exact
        q = ws_view(ws, L, "act_q", torch.uint8, cfg.T * cfg.H).reshape(cfg.T, cfg.H)
        rows = np.arange(cfg.T) if tokens is None else tokens
        rq, _ = O.act_quant_fp8(O.bf16_to_f64(inp["hidden"][rows]).astype(np.float32))
        assert np.array_equal(q[rows], rq)
    ref = O.forward(cfg, inp, tokens=tokens)
    got = out if tokens is None else out[tokens]
    err = rel_err(got, ref["out"])
    print(f"  max|err|/rms = {err:.3e} (block_m={L['block_m']})", flush=True)
    assert err <= TOL[cfg.wfmt]
    return err


@pytest.mark.parametrize("T", [1, 33, 200, 700])
def test_fp8_small(dev, T):
    _check(synth.tiny_config(4, T=T, H=512, I=256, E=16, top_k=4))


def test_fp8_h_not_multiple_of_256(dev):
    _check(synth.tiny_config(4, T=150, H=384, I=384, E=8, top_k=3))


@pytest.mark.parametrize("T", [1, 45, 300, 1000])
def test_int4_small(dev, T):
    _check(synth.tiny_config(5, T=T, H=512, I=256, E=12, top_k=4))


def test_int4_h_not_multiple_of_256(dev):
    _check(synth.tiny_config(5, T=150, H=384, I=384, E=8, top_k=3))


@pytest.mark.parametrize("wcfg", [4, 5])
def test_quant_minimum_k(dev, wcfg):
    # H = I = 128: one (fp8) or two (int4) K steps per tile
    _check(synth.tiny_config(wcfg, T=400, H=128, I=128, E=4, top_k=2))


def test_int4_workload_full_size(dev):
    _check(synth.config(5))


def test_fp8_workload_full_size_sampled(dev):
    cfg = synth.config(4)
    tokens = np.array([0, 1, 777, 2048, 4095, 5000, 8190, 8191])
    _check(cfg, tokens=tokens)


def test_quant_run_twice_bit_identical(dev):
    for cfg in (synth.tiny_config(4, T=300), synth.tiny_config(5, T=300)):
        inp = synth.make_inputs(cfg)
        a, ws, _, _ = run_forward(cfg, inp)
        b, _, _, _ = run_forward(cfg, inp, workspace=ws)
        assert np.array_equal(a, b)
