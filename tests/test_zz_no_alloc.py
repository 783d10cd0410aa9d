"""moe_forward_static_ws (the layer in the library's own per-GPU workspace,
for callers that cannot allocate) against moe_forward with a caller
workspace: identical outputs on two calls in a row, the second smaller, and
both within the format's tolerance of the oracle; oversized requests are
refused on the host."""
import numpy as np
import pytest
import torch

import paper_2607_12875_amd as moe
import synth
from oracle import moe_oracle as O
from tests.gpu_util import TOL, rel_err, require_gpu

pytestmark = pytest.mark.gpu


def _args(cfg, d, out):
    return moe.make_args(cfg.T, cfg.H, cfg.E, cfg.I, cfg.top_k, mode=cfg.mode, renormalize=cfg.renormalize,
                         routed_scale=cfg.routed_scale, wfmt=cfg.wfmt, out_dtype="f32", hidden=d["hidden"],
                         logits=d["logits"], w1=d["w1"], w2=d["w2"], w1_scale=d["w1_scale"],
                         w2_scale=d["w2_scale"], sel_bias=d["sel_bias"], out=out)


@pytest.mark.parametrize("pair", [
    # bf16: the tiled kernels (300 tokens), then the decode ones (12 tokens)
    (dict(n=1, T=300, H=512, I=256, E=8, top_k=2), dict(n=1, T=12, H=512, I=256, E=8, top_k=2)),
    # fp8: 700 tokens, then 40 on a smaller layer
    (dict(n=4, T=700, H=512, I=1024, E=16, top_k=4), dict(n=4, T=40, H=256, I=1024, E=8, top_k=2)),
    # int4, the full-size skewed workload (226 MiB of workspace, tiled
    # kernels), then a small batch on the streamed decode kernels
    (dict(n=5), dict(n=5, T=12, H=1024, I=512, E=12, top_k=4)),
])
def test_static_workspace_matches_caller_workspace(pair):
    require_gpu()
    for spec in pair:
        spec = dict(spec)
        n = spec.pop("n")
        cfg = synth.config(n) if not spec else synth.tiny_config(n, **spec)
        print(f"static-workspace parity {cfg}", flush=True)
        inp = synth.make_inputs(cfg)
        d = synth.to_device(inp)
        out = torch.full((cfg.T, cfg.H), float("nan"), dtype=torch.float32, device="cuda")
        args = _args(cfg, d, out)
        assert moe.moe_workspace_bytes(args) <= moe.STATIC_WS_BYTES
        moe.moe_forward_static_ws(args)
        ref_out = torch.empty_like(out)
        ws = torch.empty(moe.moe_workspace_bytes(args), dtype=torch.uint8, device="cuda")
        moe.moe_forward_args(_args(cfg, d, ref_out), ws)
        torch.cuda.synchronize()
        assert torch.equal(out, ref_out)
        ref = O.forward(cfg, inp)
        err = rel_err(out.cpu().numpy().astype(np.float64), ref["out"])
        print(f"  max|err|/rms = {err:.3e}", flush=True)
        assert err <= TOL[cfg.wfmt]


def test_static_workspace_too_small_is_refused():
    require_gpu()
    cfg = synth.config(3)   # 599 MiB of workspace
    a = moe.make_args(cfg.T, cfg.H, cfg.E, cfg.I, cfg.top_k, wfmt=cfg.wfmt)
    assert moe.moe_workspace_bytes(a) > moe.STATIC_WS_BYTES
    for k in ("hidden", "logits", "w1", "w2", "out"):
        setattr(a, k, 0x10000)    # never dereferenced: the size check comes first
    with pytest.raises(moe.MoeError) as ei:
        moe.moe_forward_static_ws(a)
    assert ei.value.status == moe._binding.MOE_ERR_WORKSPACE
