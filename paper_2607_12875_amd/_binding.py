"""Thin ctypes binding of ``libmoe_mi355x.so`` (declared in include/moe.h).

Argument marshalling only: every step of the layer runs in the library's HIP
kernels.  torch supplies device memory and the current HIP stream.  There is no
fallback of any kind: a missing library or a non-OK status raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmoe_mi355x.so")

MOE_OK = 0
MOE_ERR_NULL, MOE_ERR_SHAPE, MOE_ERR_UNSUPPORTED, MOE_ERR_ALIGN, MOE_ERR_WORKSPACE, MOE_ERR_HIP = range(1, 7)
STATUS_NAMES = {0: "MOE_OK", 1: "MOE_ERR_NULL", 2: "MOE_ERR_SHAPE", 3: "MOE_ERR_UNSUPPORTED",
                4: "MOE_ERR_ALIGN", 5: "MOE_ERR_WORKSPACE", 6: "MOE_ERR_HIP"}
SCORE = {"softmax": 0, "sigmoid": 1}
WFMT = {"bf16": 0, "fp8": 1, "int4": 2, "fp8a16": 3, "mxfp4": 4, "mxfp4x8": 5}
OFMT = {"f32": 0, "bf16": 1}

EXPORTED = ("moe_status_str", "moe_permute_capacity", "moe_permute_workspace_bytes",
            "moe_gate_topk", "moe_router_gate_topk", "moe_router_workspace_bytes", "moe_permute", "moe_act_quant_fp8", "moe_workspace_bytes",
            "moe_workspace_layout", "moe_forward", "moe_forward_profiled", "moe_forward_static_ws",
            # include/moe_peaks.h: achievable-peak probes
            "moe_peak_mfma_flops_per_launch", "moe_peak_sink_elems", "moe_peak_mfma", "moe_peak_read", "moe_peak_copy",
            "moe_peak_lds_copy_bytes_per_launch", "moe_peak_lds_copy", "moe_peak_lds_read_bytes_per_launch",
            "moe_peak_lds_read")
STATIC_WS_BYTES = 256 << 20  # MOE_STATIC_WS_BYTES: the library's own per-GPU workspace
NUM_STAGES = 6
STAGES = ("gate", "permute", "act_quant", "gemm1", "gemm2", "combine")


class MoeError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)}")
        self.status = status


class MoeArgs(ctypes.Structure):
    _fields_ = [
        ("T", ctypes.c_int32), ("H", ctypes.c_int32), ("E", ctypes.c_int32),
        ("I", ctypes.c_int32), ("top_k", ctypes.c_int32),
        ("score_mode", ctypes.c_int32), ("renormalize", ctypes.c_int32),
        ("routed_scale", ctypes.c_float), ("wfmt", ctypes.c_int32), ("ofmt", ctypes.c_int32),
        ("sel_bias", ctypes.c_void_p), ("hidden", ctypes.c_void_p), ("logits", ctypes.c_void_p),
        ("w1", ctypes.c_void_p), ("w2", ctypes.c_void_p),
        ("w1_scale", ctypes.c_void_p), ("w2_scale", ctypes.c_void_p),
        ("out", ctypes.c_void_p), ("topk_ids_out", ctypes.c_void_p), ("topk_w_out", ctypes.c_void_p),
        ("w_router", ctypes.c_void_p), ("logits_out", ctypes.c_void_p),
    ]


class MoeWsLayout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in (
        "topk_ids", "topk_w", "expert_offsets", "sorted_ids", "inv_pos", "act_q", "act_s",
        "inter", "inter_s", "y", "permute_ws", "router_ws")] + [
        ("block_m", ctypes.c_int32), ("cap", ctypes.c_int32), ("total", ctypes.c_int64)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load the library once; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2607_12875_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, f32, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
        L.moe_status_str.restype = ctypes.c_char_p
        L.moe_status_str.argtypes = [i32]
        L.moe_permute_capacity.restype = sz
        L.moe_permute_capacity.argtypes = [i32, i32, i32, i32]
        L.moe_permute_workspace_bytes.restype = sz
        L.moe_permute_workspace_bytes.argtypes = [i32, i32, i32]
        L.moe_gate_topk.restype = i32
        L.moe_gate_topk.argtypes = [vp, vp, i32, i32, i32, i32, i32, f32, vp, vp, vp]
        L.moe_router_gate_topk.restype = i32
        L.moe_router_gate_topk.argtypes = [vp, vp, i32, i32, i32, i32, i32, i32, f32, vp, vp, vp, vp, vp, sz, vp]
        L.moe_router_workspace_bytes.restype = sz
        L.moe_router_workspace_bytes.argtypes = [i32, i32, i32]
        L.moe_permute.restype = i32
        L.moe_permute.argtypes = [vp, i32, i32, i32, i32, vp, vp, vp, i32, vp, sz, vp]
        L.moe_act_quant_fp8.restype = i32
        L.moe_act_quant_fp8.argtypes = [vp, i32, i32, vp, vp, vp]
        L.moe_workspace_bytes.restype = sz
        L.moe_workspace_bytes.argtypes = [ctypes.POINTER(MoeArgs)]
        L.moe_workspace_layout.restype = i32
        L.moe_workspace_layout.argtypes = [ctypes.POINTER(MoeArgs), ctypes.POINTER(MoeWsLayout)]
        L.moe_forward.restype = i32
        L.moe_forward.argtypes = [ctypes.POINTER(MoeArgs), vp, sz, vp]
        L.moe_forward_static_ws.restype = i32
        L.moe_forward_static_ws.argtypes = [ctypes.POINTER(MoeArgs), vp]
        L.moe_peak_mfma_flops_per_launch.restype = ctypes.c_longlong
        L.moe_peak_mfma_flops_per_launch.argtypes = [i32, i32]
        L.moe_peak_sink_elems.restype = i32
        L.moe_peak_sink_elems.argtypes = []
        L.moe_peak_read.restype = i32
        L.moe_peak_read.argtypes = [vp, sz, vp, vp]
        L.moe_peak_mfma.restype = i32
        L.moe_peak_mfma.argtypes = [i32, i32, vp, vp]
        L.moe_peak_copy.restype = i32
        L.moe_peak_copy.argtypes = [vp, vp, sz, vp]
        L.moe_peak_lds_copy_bytes_per_launch.restype = ctypes.c_longlong
        L.moe_peak_lds_copy_bytes_per_launch.argtypes = [i32, i32, i32]
        L.moe_peak_lds_copy.restype = i32
        L.moe_peak_lds_copy.argtypes = [vp, sz, i32, i32, i32, vp]
        L.moe_peak_lds_read_bytes_per_launch.restype = ctypes.c_longlong
        L.moe_peak_lds_read_bytes_per_launch.argtypes = [i32, i32]
        L.moe_peak_lds_read.restype = i32
        L.moe_peak_lds_read.argtypes = [i32, i32, vp, vp]
        L.moe_forward_profiled.restype = i32
        L.moe_forward_profiled.argtypes = [ctypes.POINTER(MoeArgs), vp, sz,
                                           ctypes.POINTER(ctypes.c_void_p), vp]
        _lib = L
    return _lib


def _check(status: int, where: str):
    if status != MOE_OK:
        raise MoeError(status, where)


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dev(*ts):
    for t in ts:
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise ValueError("tensors must be contiguous device tensors")


# ------------------------------------------------------------------ entry points
def moe_permute_capacity(T: int, top_k: int, E: int, block_m: int) -> int:
    return lib().moe_permute_capacity(T, top_k, E, block_m)


def moe_permute_workspace_bytes(T: int, top_k: int, E: int) -> int:
    return lib().moe_permute_workspace_bytes(T, top_k, E)


def moe_gate_topk(logits, top_k, mode="softmax", renormalize=True, routed_scale=1.0,
                  sel_bias=None, topk_ids=None, topk_w=None, stream=None):
    """MoE Gate: returns (topk_ids int32 [T,k], topk_w fp32 [T,k])."""
    _dev(logits, sel_bias)
    T, E = logits.shape
    if topk_ids is None:
        topk_ids = torch.empty((T, top_k), dtype=torch.int32, device=logits.device)
    if topk_w is None:
        topk_w = torch.empty((T, top_k), dtype=torch.float32, device=logits.device)
    _check(lib().moe_gate_topk(_ptr(logits), _ptr(sel_bias), T, E, top_k, SCORE[mode],
                               int(renormalize), float(routed_scale), _ptr(topk_ids),
                               _ptr(topk_w), _stream(stream)), "moe_gate_topk")
    return topk_ids, topk_w


def moe_router_gate_topk(hidden, w_router, top_k, mode="softmax", renormalize=True, routed_scale=1.0,
                         sel_bias=None, logits=None, topk_ids=None, topk_w=None, stream=None):
    """Router GEMM (bf16 hidden [T,H] x w_router [E,H]^T, fp32) then the
    gate: returns (topk_ids int32 [T,k], topk_w fp32 [T,k]); logits, if given
    (fp32 [T,E]), receives the logits the selection used."""
    _dev(hidden, w_router, sel_bias, logits)
    T, H = hidden.shape
    E = w_router.shape[0]
    if topk_ids is None:
        topk_ids = torch.empty((T, top_k), dtype=torch.int32, device=hidden.device)
    if topk_w is None:
        topk_w = torch.empty((T, top_k), dtype=torch.float32, device=hidden.device)
    nws = lib().moe_router_workspace_bytes(T, H, E)
    ws = torch.empty(max(nws, 16), dtype=torch.uint8, device=hidden.device)
    _check(lib().moe_router_gate_topk(_ptr(hidden), _ptr(w_router), T, H, E, top_k, SCORE[mode],
                                      int(renormalize), float(routed_scale), _ptr(sel_bias),
                                      _ptr(logits), _ptr(topk_ids), _ptr(topk_w), _ptr(ws), ws.numel(),
                                      _stream(stream)),
           "moe_router_gate_topk")
    return topk_ids, topk_w


def moe_permute(topk_ids, E: int, block_m: int, stream=None):
    """Permute/align: returns (expert_offsets [E+1], sorted_ids [cap], inv_pos [T*k])."""
    _dev(topk_ids)
    T, k = topk_ids.shape
    dev = topk_ids.device
    cap = moe_permute_capacity(T, k, E, block_m)
    offsets = torch.empty(E + 1, dtype=torch.int32, device=dev)
    sorted_ids = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
    inv_pos = torch.empty(max(T * k, 1), dtype=torch.int32, device=dev)
    nws = moe_permute_workspace_bytes(T, k, E)
    ws = torch.empty(max(nws, 16), dtype=torch.uint8, device=dev)
    _check(lib().moe_permute(_ptr(topk_ids), T, k, E, block_m, _ptr(offsets), _ptr(sorted_ids),
                             _ptr(inv_pos), cap, _ptr(ws), nws, _stream(stream)), "moe_permute")
    return offsets, sorted_ids[:cap], inv_pos[:T * k]


def moe_act_quant_fp8(x, stream=None):
    """Per (row, 128-column) e4m3 quantisation of bf16 x [M,K] -> (codes uint8, scales fp32)."""
    _dev(x)
    M, K = x.shape
    q = torch.empty((M, K), dtype=torch.uint8, device=x.device)
    s = torch.empty((M, max(K // 128, 1)), dtype=torch.float32, device=x.device)
    _check(lib().moe_act_quant_fp8(_ptr(x), M, K, _ptr(q), _ptr(s), _stream(stream)),
           "moe_act_quant_fp8")
    return q, s


def make_args(T, H, E, I, top_k, *, mode="softmax", renormalize=True, routed_scale=1.0,
              wfmt="bf16", out_dtype="f32", hidden=None, logits=None, w1=None, w2=None,
              w1_scale=None, w2_scale=None, sel_bias=None, out=None, topk_ids_out=None,
              topk_w_out=None, w_router=None, logits_out=None) -> MoeArgs:
    return MoeArgs(T, H, E, I, top_k, SCORE[mode], int(renormalize), float(routed_scale),
                   WFMT[wfmt], OFMT[out_dtype], _ptr(sel_bias), _ptr(hidden), _ptr(logits),
                   _ptr(w1), _ptr(w2), _ptr(w1_scale), _ptr(w2_scale), _ptr(out),
                   _ptr(topk_ids_out), _ptr(topk_w_out), _ptr(w_router), _ptr(logits_out))


def moe_workspace_bytes(args: MoeArgs) -> int:
    return lib().moe_workspace_bytes(ctypes.byref(args))


def moe_workspace_layout(args: MoeArgs) -> dict:
    L = MoeWsLayout()
    _check(lib().moe_workspace_layout(ctypes.byref(args), ctypes.byref(L)), "moe_workspace_layout")
    return {name: getattr(L, name) for name, _ in MoeWsLayout._fields_}


def moe_forward_args(args: MoeArgs, workspace, stream=None):
    """Run the layer on a prepared MoeArgs with a caller-owned uint8 workspace."""
    _check(lib().moe_forward(ctypes.byref(args), _ptr(workspace), workspace.numel(),
                             _stream(stream)), "moe_forward")


def moe_forward_static_ws(args: MoeArgs, stream=None):
    """Run the layer on a prepared MoeArgs in the library's own per-GPU
    workspace (no workspace argument, nothing allocated); the workspace the
    sizes need must not exceed STATIC_WS_BYTES."""
    _check(lib().moe_forward_static_ws(ctypes.byref(args), _stream(stream)), "moe_forward_static_ws")


def moe_forward_profiled(args: MoeArgs, workspace, events, stream=None):
    """moe_forward with hipEvent_t handles (ints) recorded around each stage."""
    arr = (ctypes.c_void_p * (NUM_STAGES + 1))(*events)
    _check(lib().moe_forward_profiled(ctypes.byref(args), _ptr(workspace), workspace.numel(),
                                      arr, _stream(stream)), "moe_forward_profiled")


def moe_forward(hidden, logits, w1, w2, top_k, *, mode="softmax", renormalize=True,
                routed_scale=1.0, wfmt="bf16", sel_bias=None, w1_scale=None, w2_scale=None,
                out_dtype="f32", out=None, workspace=None, topk_ids_out=None, topk_w_out=None,
                w_router=None, logits_out=None, stream=None):
    """The whole layer on device tensors; returns (out [T,H], workspace).

    hidden bf16 [T,H]; logits fp32 [T,E]; weights in the wfmt storage:
    bf16 [E,2I,H] / [E,H,I]; fp8 uint8 codes with fp32 block scales
    [E,2I/128,H/128] / [E,H/128,I/128]; int4 int32 [E,2I,H/8] / [E,H,I/8] with
    bf16 scales [E,2I,H/128] / [E,H,I/128]; "fp8a16" (weight-only fp8, a decode
    route) takes the fp8 storage with bf16 activations; "mxfp4" uint8
    [E,2I,H/2] / [E,H,I/2] two E2M1 codes per byte with uint8 E8M0 scales
    [E,2I,H/32] / [E,H,I/32] (bf16 activations); "mxfp4x8" the same storage
    with MXFP8 activations quantised in-layer.  With w_router (bf16
    [E,H]) the layer computes its own logits (pass logits=None); logits_out
    (fp32 [T,E]) then receives them."""
    _dev(hidden, logits, w1, w2, sel_bias, w1_scale, w2_scale, out, topk_ids_out, topk_w_out,
         w_router, logits_out)
    T, H = hidden.shape
    E = (w_router if w_router is not None else logits).shape[0 if w_router is not None else 1]
    I = w2.shape[2] * {"int4": 8, "mxfp4": 2, "mxfp4x8": 2}.get(wfmt, 1)
    if out is None:
        out = torch.empty((T, H), dtype=torch.float32 if out_dtype == "f32" else torch.bfloat16,
                          device=hidden.device)
    args = make_args(T, H, E, I, top_k, mode=mode, renormalize=renormalize,
                     routed_scale=routed_scale, wfmt=wfmt, out_dtype=out_dtype, hidden=hidden,
                     logits=logits, w1=w1, w2=w2, w1_scale=w1_scale, w2_scale=w2_scale,
                     sel_bias=sel_bias, out=out, topk_ids_out=topk_ids_out, topk_w_out=topk_w_out,
                     w_router=w_router, logits_out=logits_out)
    need = moe_workspace_bytes(args)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=hidden.device)
    moe_forward_args(args, workspace, stream)
    return out, workspace


# ------------------------------------------------------------ peak probes
def moe_peak_mfma_flops_per_launch(fp8: bool, iters: int) -> int:
    return lib().moe_peak_mfma_flops_per_launch(int(bool(fp8)), iters)


def moe_peak_sink_elems() -> int:
    return lib().moe_peak_sink_elems()


def moe_peak_mfma(fp8: bool, iters: int, sink, stream=None):
    """One launch of the MFMA-only probe; sink: float32 device tensor of at
    least moe_peak_sink_elems() elements."""
    _dev(sink)
    if sink.dtype != torch.float32 or sink.numel() < moe_peak_sink_elems():
        raise ValueError("sink: float32, moe_peak_sink_elems() elements")
    _check(lib().moe_peak_mfma(int(bool(fp8)), iters, _ptr(sink), _stream(stream)), "moe_peak_mfma")


def moe_peak_read(src, sink, stream=None):
    """Read src once with the streaming probe; sink: int32 device tensor of at
    least moe_peak_sink_elems() zeroed elements, XORed with per-workgroup folds."""
    _dev(src, sink)
    if sink.dtype != torch.int32 or sink.numel() < moe_peak_sink_elems():
        raise ValueError("sink: int32, moe_peak_sink_elems() elements")
    n = src.numel() * src.element_size()
    _check(lib().moe_peak_read(_ptr(src), n, _ptr(sink), _stream(stream)), "moe_peak_read")


def moe_peak_copy(src, dst, stream=None):
    """dst[:] = src[:] (same byte size, 16-byte multiple) with the streaming copy probe."""
    _dev(src, dst)
    n = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != n:
        raise ValueError("src and dst must have the same size in bytes")
    _check(lib().moe_peak_copy(_ptr(src), _ptr(dst), n, _stream(stream)), "moe_peak_copy")


def moe_peak_lds_copy_bytes_per_launch(waves: int, copies: int, steps: int) -> int:
    return lib().moe_peak_lds_copy_bytes_per_launch(waves, copies, steps)


def moe_peak_lds_copy(src, region_bytes: int, waves: int, copies: int, steps: int, stream=None):
    """One launch of the global -> LDS copy probe over region b % 8 of src per
    workgroup b; src must hold 8 * region_bytes bytes."""
    _dev(src)
    if src.numel() * src.element_size() < 8 * region_bytes:
        raise ValueError("src must hold 8 * region_bytes bytes")
    _check(lib().moe_peak_lds_copy(_ptr(src), region_bytes, waves, copies, steps, _stream(stream)),
           "moe_peak_lds_copy")


def moe_peak_lds_read_bytes_per_launch(waves: int, iters: int) -> int:
    return lib().moe_peak_lds_read_bytes_per_launch(waves, iters)


def moe_peak_lds_read(waves: int, iters: int, sink, stream=None):
    """One launch of the LDS fragment-read probe; sink: int32 device tensor of
    at least moe_peak_sink_elems() elements."""
    _dev(sink)
    if sink.dtype != torch.int32 or sink.numel() < moe_peak_sink_elems():
        raise ValueError("sink: int32, moe_peak_sink_elems() elements")
    _check(lib().moe_peak_lds_read(waves, iters, _ptr(sink), _stream(stream)), "moe_peak_lds_read")
