"""The layer under HIP graph capture.  moe_forward allocates nothing, never
synchronises and enqueues only kernel launches (no memset or copy nodes), so a
serving loop can capture it once and replay it.  Every replay -- with eager
layer calls on other inputs run in between, on the same workspace -- must
reproduce the eager result bit for bit: nothing a call relies on survives
from an earlier one."""
import numpy as np
import pytest
import torch

import paper_2607_12875_amd as moe
import synth
from tests.gpu_util import require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return require_gpu()


def _args(cfg, d, out):
    return moe.make_args(cfg.T, cfg.H, cfg.E, cfg.I, cfg.top_k, mode=cfg.mode, renormalize=cfg.renormalize,
                         routed_scale=cfg.routed_scale, wfmt=cfg.wfmt, hidden=d["hidden"], logits=d["logits"],
                         w1=d["w1"], w2=d["w2"], w1_scale=d["w1_scale"], w2_scale=d["w2_scale"],
                         sel_bias=d["sel_bias"], out=out)


@pytest.mark.parametrize("cfg", [
    synth.tiny_config(2, T=16, H=1024, I=1408, E=24, top_k=6),   # streamed decode kernels
    synth.tiny_config(1, T=600, H=512, I=384, E=8, top_k=2),     # tiled bf16 kernels
    synth.tiny_config(5, T=300, H=512, I=256, E=12, top_k=4),    # int4 route
    synth.tiny_config(5, T=12, H=1024, I=512, E=12, top_k=4),    # int4, streamed decode kernels
    synth.tiny_config(7, T=300, H=512, I=256, E=12, top_k=4),    # MXFP4, tiled
    synth.tiny_config(9, T=300, H=512, I=512, E=12, top_k=4),    # MXFP4 x MXFP8
], ids=["decode", "tiled", "int4", "int4-decode", "mxfp4", "mxfp4x8"])
def test_graph_replays_match_eager(dev, cfg):
    print(f"graph replay {cfg}", flush=True)
    d = synth.to_device(synth.make_inputs(cfg))
    out_ref = torch.empty((cfg.T, cfg.H), dtype=torch.float32, device=dev)
    a_ref = _args(cfg, d, out_ref)
    ws = torch.empty(moe.moe_workspace_bytes(a_ref), dtype=torch.uint8, device=dev)
    moe.moe_forward_args(a_ref, ws)
    torch.cuda.synchronize()
    ref = out_ref.clone()

    # other inputs for the eager calls between replays (same shapes, same workspace)
    d2 = dict(d)
    d2["logits"] = torch.flip(d["logits"], dims=[1]).contiguous()
    d2["hidden"] = torch.roll(d["hidden"], shifts=1, dims=0).contiguous()
    out2 = torch.empty_like(out_ref)
    a2 = _args(cfg, d2, out2)

    out_g = torch.empty_like(out_ref)
    a_g = _args(cfg, d, out_g)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        moe.moe_forward_args(a_g, ws)  # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        moe.moe_forward_args(a_g, ws)
    torch.cuda.synchronize()

    eager2 = None
    for r in range(3):
        out_g.fill_(np.nan)
        moe.moe_forward_args(a2, ws)  # clobbers every workspace region
        torch.cuda.synchronize()
        if eager2 is None:
            eager2 = out2.clone()
        else:
            assert torch.equal(out2, eager2)
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out_g, ref), f"replay {r} differs from the eager result"
    assert not torch.equal(eager2, ref)  # the eager calls between replays computed something else
