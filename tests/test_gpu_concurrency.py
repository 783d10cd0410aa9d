"""Layer calls on several streams at once.  The library keeps no state
between calls beyond the caller's buffers, so two layers with their own
workspaces and outputs, enqueued on two streams and running concurrently,
give bit for bit what the same calls give one after the other.  The layers
differ in format and shape, so their kernels overlap on the device with
different grids."""
import numpy as np
import pytest
import torch

import paper_2607_12875_amd as moe
import synth
from tests.gpu_util import require_gpu

pytestmark = pytest.mark.gpu


def _launch(cfg, d, ws, out, stream):
    return moe.moe_forward(
        d["hidden"], d["logits"], d["w1"], d["w2"], cfg.top_k, mode=cfg.mode,
        renormalize=cfg.renormalize, routed_scale=cfg.routed_scale, wfmt=cfg.wfmt,
        sel_bias=d["sel_bias"], w1_scale=d["w1_scale"], w2_scale=d["w2_scale"],
        out=out, workspace=ws, stream=stream)


def test_two_streams_match_sequential():
    require_gpu()
    cfgs = [synth.tiny_config(4, T=600, H=512, I=1024, E=16, top_k=4),   # fp8, tiled
            synth.tiny_config(3, T=900, H=384, I=256, E=12, top_k=3),    # bf16, tiled
            synth.tiny_config(2, T=12, H=1024, I=512, E=24, top_k=4),    # bf16, streamed decode
            synth.tiny_config(5, T=12, H=1024, I=512, E=12, top_k=4)]    # int4, streamed decode
    layers = []
    for cfg in cfgs:
        print(f"concurrency layer {cfg}", flush=True)
        d = synth.to_device(synth.make_inputs(cfg))
        args = moe.make_args(cfg.T, cfg.H, cfg.E, cfg.I, cfg.top_k, wfmt=cfg.wfmt)
        ws = torch.empty(moe.moe_workspace_bytes(args), dtype=torch.uint8, device="cuda")
        out = torch.empty((cfg.T, cfg.H), dtype=torch.float32, device="cuda")
        layers.append((cfg, d, ws, out))
    # one after the other on the current stream
    ref = []
    for cfg, d, ws, out in layers:
        _launch(cfg, d, ws, out, None)
        torch.cuda.synchronize()
        ref.append(out.clone())
    # all at once, one stream each (default priority), several rounds
    streams = [torch.cuda.Stream() for _ in layers]
    for rnd in range(4):
        for (cfg, d, ws, out), s in zip(layers, streams):
            out.fill_(float("nan"))
        torch.cuda.synchronize()
        for (cfg, d, ws, out), s in zip(layers, streams):
            _launch(cfg, d, ws, out, s)
        torch.cuda.synchronize()
        for (cfg, d, ws, out), r in zip(layers, ref):
            assert torch.equal(out, r), f"round {rnd}: {cfg}"
    print("  concurrent rounds bit-identical to the sequential calls", flush=True)
