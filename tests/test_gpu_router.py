"""GPU parity of the router GEMM fused with the gate (moe_router_gate_topk,
and moe_forward with a router weight) against the oracle.

The kernel accumulates bf16 products in fp32 in its own order, so:
  * its fp32 logits must lie within an fp32-accumulation bound of the fp64
    oracle's, |l - l_exact| <= 2 (H/32 + 32) 2^-24 sum_h |x_h w_h| (one
    rounding per 32-product MFMA step plus one per product inside it, doubled);
  * the selection, a floating-point decision, is checked where both sides
    decide it on the same numbers: the oracle gate run on the kernel's own
    fp32 logits must give the same ids bit for bit (weights within 1e-6);
  * the layer output must match the oracle layer on those logits within the
    format's tolerance."""
import numpy as np
import pytest
import torch

import paper_2607_12875_amd as moe
import synth
from oracle import moe_oracle as O
from tests.gpu_util import TOL, rel_err, require_gpu, ws_view

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def _bound(hid, wr):
    x, w = O.bf16_to_f64(hid), O.bf16_to_f64(wr)
    return 2.0 * (x.shape[1] / 32 + 32) * 2.0 ** -24 * (np.abs(x) @ np.abs(w).T)


def _bf16(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)


def _check_router(dev, cfg, sample=None):
    print(f"router parity {cfg}", flush=True)
    r = synth.make_routing_inputs(cfg)
    wr = synth.make_router_weights(cfg)
    bias = None if r["sel_bias"] is None else torch.from_numpy(r["sel_bias"]).to(dev)
    logits = torch.empty((cfg.T, cfg.E), dtype=torch.float32, device=dev)
    ids, w = moe.moe_router_gate_topk(_bf16(r["hidden"], dev), _bf16(wr, dev), cfg.top_k, cfg.mode,
                                      cfg.renormalize, cfg.routed_scale, sel_bias=bias, logits=logits)
    torch.cuda.synchronize()
    lg, ids, w = logits.cpu().numpy(), ids.cpu().numpy(), w.cpu().numpy()
    rows = np.arange(cfg.T) if sample is None else np.asarray(sample)
    ref = O.router_logits(r["hidden"][rows], wr)
    dev_ = np.abs(lg[rows] - ref) / np.maximum(_bound(r["hidden"][rows], wr), 1e-300)
    print(f"  logits: max |err| / bound = {dev_.max():.3f}", flush=True)
    assert dev_.max() <= 1.0
    rid, rw = O.gate(lg, r["sel_bias"], cfg.top_k, cfg.mode, cfg.renormalize, cfg.routed_scale)
    assert np.array_equal(ids, rid), np.argwhere(ids != rid)[:5]
    assert np.all(np.abs(w - rw) <= 1e-6 * np.abs(rw))
    return lg


@pytest.mark.parametrize("T,H,E,k", [(1, 128, 8, 2), (16, 4096, 64, 6), (37, 512, 100, 7),
                                     (77, 256, 16, 4), (300, 1024, 300, 8), (20, 384, 1024, 32),
                                     (4100, 512, 256, 8)])
@pytest.mark.parametrize("n", [2, 4])
def test_router_gate_shapes(dev, T, H, E, k, n):
    # n = 2: softmax renormalised; n = 4: sigmoid + selection bias x 2.5 (rank
    # selection up to 64 experts, arg-max rounds above)
    _check_router(dev, synth.tiny_config(n, T=T, H=H, E=E, top_k=k))


def test_router_gemm_route_unaligned_logits(dev):
    # many tokens x many experts take the logits product on the tiled GEMM
    # (4100 tokens: a ragged last 128-row tile); a logits buffer that is only
    # 4-byte aligned gets the same values through the workspace copy
    cfg = synth.tiny_config(4, T=4100, H=512, E=256, top_k=8)
    r = synth.make_routing_inputs(cfg)
    wr = _bf16(synth.make_router_weights(cfg), dev)
    hid = _bf16(r["hidden"], dev)
    bias = torch.from_numpy(r["sel_bias"]).to(dev)
    a = torch.empty((cfg.T, cfg.E), dtype=torch.float32, device=dev)
    buf = torch.empty(cfg.T * cfg.E + 1, dtype=torch.float32, device=dev)
    b = buf[1:].view(cfg.T, cfg.E)
    assert b.data_ptr() % 16 != 0
    args = (cfg.top_k, cfg.mode, cfg.renormalize, cfg.routed_scale)
    ia, wa = moe.moe_router_gate_topk(hid, wr, *args, sel_bias=bias, logits=a)
    ib, wb = moe.moe_router_gate_topk(hid, wr, *args, sel_bias=bias, logits=b)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(ia, ib) and torch.equal(wa, wb)


def test_router_gate_workload_shapes(dev):
    # decode (T=16, H=4096, E=64) and the fp8 workload's routing (T=8192,
    # H=7168, E=256): logits of every token against the fp64 sums
    _check_router(dev, synth.config(2))
    _check_router(dev, synth.config(4))


@pytest.mark.parametrize("n,T,over", [(2, 16, {}), (1, 300, {}), (4, 200, {}), (6, 16, {}),
                                      (2, 4096, dict(H=256, E=256, I=128))])
def test_forward_with_router(dev, n, T, over):
    # the last case's logits come from the tiled GEMM (4096 tokens x 256 experts)
    cfg = synth.tiny_config(n, T=T, **over)
    print(f"forward with router {cfg}", flush=True)
    inp = synth.make_inputs(cfg)
    wr = synth.make_router_weights(cfg)
    d = synth.to_device(inp)
    logits = torch.empty((cfg.T, cfg.E), dtype=torch.float32, device=dev)
    out, ws = moe.moe_forward(d["hidden"], None, d["w1"], d["w2"], cfg.top_k, mode=cfg.mode,
                              renormalize=cfg.renormalize, routed_scale=cfg.routed_scale, wfmt=cfg.wfmt,
                              sel_bias=d["sel_bias"], w1_scale=d["w1_scale"], w2_scale=d["w2_scale"],
                              w_router=_bf16(wr, dev), logits_out=logits)
    torch.cuda.synchronize()
    lg = logits.cpu().numpy()
    assert np.all(np.abs(lg - O.router_logits(inp["hidden"], wr)) <= _bound(inp["hidden"], wr))
    L = moe.moe_workspace_layout(moe.make_args(cfg.T, cfg.H, cfg.E, cfg.I, cfg.top_k, wfmt=cfg.wfmt))
    ids = ws_view(ws, L, "topk_ids", torch.int32, cfg.T * cfg.top_k).reshape(cfg.T, cfg.top_k)
    ref = O.forward(cfg, dict(inp, logits=lg))
    assert np.array_equal(ids, ref["ids"])
    err = rel_err(out.float().cpu().numpy().astype(np.float64), ref["out"])
    print(f"  max|err|/rms = {err:.3e}", flush=True)
    assert err <= TOL[cfg.wfmt]
