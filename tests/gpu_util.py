"""Shared helpers of the GPU parity tests (test infrastructure)."""
import numpy as np
import pytest
import torch

import paper_2607_12875_amd as moe
import synth

TOL = {"bf16": 2e-2, "fp8": 6e-2, "int4": 8e-2}   # max|err| <= TOL * rms(oracle out)


def require_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible MI355X")
    moe.lib()  # raises if the HIP library is missing: no fallback exists
    return torch.device("cuda:0")


def run_forward(cfg, inp, out_dtype="f32", workspace=None):
    """Upload numpy inputs, run moe_forward, return (out numpy f64, workspace, layout, dev tensors)."""
    d = synth.to_device(inp)
    out, ws = moe.moe_forward(
        d["hidden"], d["logits"], d["w1"], d["w2"], cfg.top_k, mode=cfg.mode,
        renormalize=cfg.renormalize, routed_scale=cfg.routed_scale, wfmt=cfg.wfmt,
        sel_bias=d["sel_bias"], w1_scale=d["w1_scale"], w2_scale=d["w2_scale"],
        out_dtype=out_dtype, workspace=workspace)
    torch.cuda.synchronize()
    args = moe.make_args(cfg.T, cfg.H, cfg.E, cfg.I, cfg.top_k, wfmt=cfg.wfmt)
    layout = moe.moe_workspace_layout(args)
    return out.float().cpu().numpy().astype(np.float64), ws, layout, d


def ws_view(ws, layout, name, dtype, count):
    off = layout[name]
    nbytes = count * torch.tensor([], dtype=dtype).element_size()
    return ws[off:off + nbytes].view(dtype)[:count].cpu().numpy()


def rel_err(out, ref):
    rms = np.sqrt((ref ** 2).mean())
    return np.max(np.abs(out - ref)) / rms
