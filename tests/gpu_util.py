"""Shared helpers of the GPU parity tests (test infrastructure)."""
import numpy as np
import pytest
import torch

import paper_2607_12875_amd as moe
import synth

# MXFP4 x MXFP8: the fp8 budget times 448/256.  Its error is the fp8
# route's (requantisation ties the hardware's accumulation tips over, plus
# bf16 y), but a power-of-two block scale can leave the block maximum as low
# as 256 X, where one e4m3 step is 32/256 of it, against 32/448 when the
# maximum maps to 448.
TOL = {"bf16": 2e-2, "fp8": 6e-2, "int4": 8e-2, "fp8a16": 2e-2, "mxfp4": 2e-2, "mxfp4x8": 1.05e-1}   # max|err| <= TOL * rms(oracle out)


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


def check_forward(cfg, inp=None, out_dtype="f32"):
    """Whole-layer parity against the oracle on every token: ids, offsets,
    sorted ids and inverse positions bit-exact; for fp8 weights the layer's
    own activation codes bit-exact on every row; max|err| <= TOL * rms(oracle
    out), rms over all T*H outputs (plus, for a bf16 output, its own rounding
    of at most 2^-9 of each element)."""
    from oracle import moe_oracle as O
    print(f"forward parity {cfg}", flush=True)
    inp = synth.make_inputs(cfg) if inp is None else inp
    out, ws, L, _ = run_forward(cfg, inp, out_dtype)
    ref = O.forward(cfg, inp)
    n = cfg.T * cfg.top_k
    ids = ws_view(ws, L, "topk_ids", torch.int32, n).reshape(cfg.T, cfg.top_k)
    assert np.array_equal(ids, ref["ids"])
    ro, rs, ri = O.permute(ref["ids"], cfg.E, L["block_m"])
    assert np.array_equal(ws_view(ws, L, "expert_offsets", torch.int32, cfg.E + 1), ro)
    assert np.array_equal(ws_view(ws, L, "sorted_ids", torch.int32, L["cap"]), rs)
    assert np.array_equal(ws_view(ws, L, "inv_pos", torch.int32, n), ri)
    if cfg.wfmt == "fp8":   # the layer's own activation quantisation, every row
        q = ws_view(ws, L, "act_q", torch.uint8, cfg.T * cfg.H).reshape(cfg.T, cfg.H)
        s = ws_view(ws, L, "act_s", torch.float32, cfg.T * cfg.H // 128).reshape(cfg.T, cfg.H // 128)
        rq, rsc = O.act_quant_fp8(O.bf16_to_f64(inp["hidden"]).astype(np.float32))
        assert np.array_equal(s, rsc)
        assert np.array_equal(q, rq)
    if cfg.wfmt == "mxfp4x8":   # the layer's own MXFP8 quantisation of the hidden rows, every row
        q = ws_view(ws, L, "act_q", torch.uint8, cfg.T * cfg.H).reshape(cfg.T, cfg.H)
        s = ws_view(ws, L, "act_s", torch.uint8, cfg.T * cfg.H // 32).reshape(cfg.T, cfg.H // 32)
        rq, rsx = O.act_quant_mxfp8(O.bf16_to_f64(inp["hidden"]).astype(np.float32))
        assert np.array_equal(s, rsx)
        assert np.array_equal(q, rq)
    err = rel_err(out, ref["out"])
    print(f"  max|err|/rms = {err:.3e} over {out.size} outputs (block_m={L['block_m']})", flush=True)
    rms = np.sqrt((ref["out"] ** 2).mean())
    slack = 0.0 if out_dtype == "f32" else 2 ** -9 * np.abs(ref["out"]).max() / rms
    assert err <= TOL[cfg.wfmt] + slack
    return out, ref, L


def rel_err(out, ref):
    rms = np.sqrt((ref ** 2).mean())
    return np.max(np.abs(out - ref)) / rms
