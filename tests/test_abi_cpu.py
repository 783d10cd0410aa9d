"""The C ABI without a GPU: the library loads, exports every function
include/moe.h declares, and rejects bad arguments on the host before any HIP
call (the only failures a test can force without a device)."""
import ctypes
import os
import re

import pytest

import paper_2607_12875_amd as moe
from paper_2607_12875_amd import _binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x10000  # a 16-byte aligned non-null address; never dereferenced on these paths


def _declared():
    names = set()
    for h in ("moe.h", "moe_peaks.h"):
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names |= set(re.findall(r"\b(moe_[a-z0-9_]+)\s*\(", src))
    return names


def test_every_declared_symbol_is_exported():
    L = moe.lib()
    declared = _declared()
    assert declared == set(B.EXPORTED)
    for name in declared:
        assert hasattr(L, name), name


def test_peak_probes_validate_on_host():
    L = moe.lib()
    assert L.moe_peak_mfma_flops_per_launch(1, 0) == 0
    n_cu = L.moe_peak_sink_elems() // 8
    assert n_cu >= 1 and L.moe_peak_sink_elems() == 8 * n_cu
    # fp8 32x32x64 and bf16 32x32x16 per instruction, 4 chains, 8 waves per CU
    assert L.moe_peak_mfma_flops_per_launch(1, 10) == n_cu * 8 * 10 * 4 * 2 * 32 * 32 * 64
    assert L.moe_peak_mfma_flops_per_launch(0, 10) == n_cu * 8 * 10 * 4 * 2 * 32 * 32 * 16
    assert L.moe_peak_mfma(1, 10, None, None) == B.MOE_ERR_NULL
    assert L.moe_peak_mfma(1, 0, FAKE, None) == B.MOE_ERR_SHAPE
    assert L.moe_peak_mfma(2, 10, FAKE, None) == B.MOE_ERR_SHAPE
    assert L.moe_peak_copy(None, FAKE, 16, None) == B.MOE_ERR_NULL
    assert L.moe_peak_copy(FAKE, FAKE, 24, None) == B.MOE_ERR_SHAPE
    assert L.moe_peak_copy(FAKE + 8, FAKE, 16, None) == B.MOE_ERR_ALIGN
    assert L.moe_peak_copy(FAKE, FAKE, 0, None) == B.MOE_OK
    assert L.moe_peak_read(None, 16, FAKE, None) == B.MOE_ERR_NULL
    assert L.moe_peak_read(FAKE, 16, None, None) == B.MOE_ERR_NULL
    assert L.moe_peak_read(FAKE, 20, FAKE, None) == B.MOE_ERR_SHAPE
    assert L.moe_peak_read(FAKE + 4, 16, FAKE, None) == B.MOE_ERR_ALIGN
    assert L.moe_peak_read(FAKE, 0, FAKE, None) == B.MOE_OK
    # global -> LDS copy and LDS read probes: 1 KB per copy, 16 x 16 B per lane per read round
    assert L.moe_peak_lds_copy_bytes_per_launch(4, 8, 10) == n_cu * 4 * 8 * 10 * 1024
    assert L.moe_peak_lds_copy_bytes_per_launch(17, 8, 10) == 0
    assert L.moe_peak_lds_copy_bytes_per_launch(4, 6, 10) == 0
    assert L.moe_peak_lds_read_bytes_per_launch(4, 10) == n_cu * 4 * 64 * 16 * 16 * 10
    assert L.moe_peak_lds_read_bytes_per_launch(0, 10) == 0
    mib = 1 << 20
    assert L.moe_peak_lds_copy(None, mib, 4, 8, 1, None) == B.MOE_ERR_NULL
    assert L.moe_peak_lds_copy(FAKE, mib, 0, 8, 1, None) == B.MOE_ERR_SHAPE
    assert L.moe_peak_lds_copy(FAKE, mib, 17, 8, 1, None) == B.MOE_ERR_SHAPE
    assert L.moe_peak_lds_copy(FAKE, mib, 4, 5, 1, None) == B.MOE_ERR_SHAPE
    assert L.moe_peak_lds_copy(FAKE, mib, 4, 8, 0, None) == B.MOE_ERR_SHAPE
    assert L.moe_peak_lds_copy(FAKE, 3 * mib, 4, 8, 1, None) == B.MOE_ERR_SHAPE  # not a power of two
    assert L.moe_peak_lds_copy(FAKE, 32 << 10, 4, 8, 1, None) == B.MOE_ERR_SHAPE  # below 64 KiB
    assert L.moe_peak_lds_copy(FAKE, 512 * mib, 4, 8, 1, None) == B.MOE_ERR_SHAPE  # above 256 MiB
    assert L.moe_peak_lds_copy(FAKE + 8, mib, 4, 8, 1, None) == B.MOE_ERR_ALIGN
    assert L.moe_peak_lds_read(4, 10, None, None) == B.MOE_ERR_NULL
    assert L.moe_peak_lds_read(0, 10, FAKE, None) == B.MOE_ERR_SHAPE
    assert L.moe_peak_lds_read(4, 0, FAKE, None) == B.MOE_ERR_SHAPE


def test_status_strings():
    L = moe.lib()
    for code, name in B.STATUS_NAMES.items():
        assert L.moe_status_str(code).decode() == name
    assert L.moe_status_str(99).decode() == "MOE_ERR_UNKNOWN"


def _args(**kw):
    base = dict(T=64, H=256, E=8, I=128, top_k=2)
    base.update({k: kw.pop(k) for k in list(kw) if k in base})
    a = B.make_args(**base, **{k: v for k, v in kw.items() if k in ("mode", "wfmt", "out_dtype", "renormalize")})
    for k in ("hidden", "logits", "w1", "w2", "w1_scale", "w2_scale", "out"):
        setattr(a, k, kw.get(k, FAKE))
    return a


def _fwd(a, ws=FAKE, nbytes=1 << 40):
    return moe.lib().moe_forward(ctypes.byref(a), ws, nbytes, None)


def test_forward_argument_validation():
    assert _fwd(_args(top_k=9)) == B.MOE_ERR_SHAPE
    assert _fwd(_args(top_k=0)) == 2
    assert _fwd(_args(E=0)) == 2
    assert _fwd(_args(E=2000, top_k=2)) == 2
    assert _fwd(_args(H=196)) == 2                      # bf16: H, I multiples of 8
    assert _fwd(_args(I=100)) == 2
    assert _fwd(_args(H=200, wfmt="fp8")) == 2          # quantised formats: multiples of 128
    assert _fwd(_args(I=200, wfmt="int4")) == 2
    assert _fwd(_args(H=0)) == 2
    assert _fwd(_args(T=-1)) == 2
    assert _fwd(_args(hidden=None)) == 1
    assert _fwd(_args(out=None)) == 1
    assert _fwd(_args(wfmt="fp8", w1_scale=None)) == 1
    assert _fwd(_args(wfmt="fp8a16", w2_scale=None)) == 1
    # the weight-only fp8 route is a decode route: T*k <= 32*E or UNSUPPORTED
    assert _fwd(_args(T=129, E=8, top_k=2, wfmt="fp8a16")) == 3
    assert _fwd(_args(T=128, E=8, top_k=2, wfmt="fp8a16"), ws=None) == 5  # accepted, then no workspace
    assert _fwd(_args(wfmt="mxfp4", w1_scale=None)) == 1
    # MXFP4 takes any batch (decode kernels up to 32 rows per expert, tiled above)
    assert _fwd(_args(T=129, E=8, top_k=2, wfmt="mxfp4"), ws=None) == 5
    assert _fwd(_args(T=128, E=8, top_k=2, wfmt="mxfp4"), ws=None) == 5
    assert _fwd(_args(hidden=FAKE + 8)) == 4
    assert _fwd(_args(), ws=None) == 5
    a = _args()
    need = moe.moe_workspace_bytes(a)
    assert need > 0
    assert _fwd(a, nbytes=need - 1) == 5
    a.score_mode = 7
    assert _fwd(a) == 3
    a = _args()
    a.wfmt = 9
    assert _fwd(a) == 3
    # a router weight replaces the logits input (16-byte aligned); one of the two is required
    a = _args(logits=None)
    assert _fwd(a) == 1
    a.w_router = FAKE
    assert _fwd(a, ws=None) == 5  # accepted, then no workspace
    a.w_router = FAKE + 4
    assert _fwd(a) == 4
    a.w_router, a.logits_out = FAKE, FAKE + 2
    assert _fwd(a) == 4
    # T == 0 is a no-op that touches no device memory
    assert _fwd(_args(T=0, hidden=None, logits=None, w1=None, w2=None, out=None), ws=None, nbytes=0) == 0


def test_gate_and_permute_validation():
    L = moe.lib()
    assert L.moe_gate_topk(FAKE, None, 4, 8, 9, 0, 1, 1.0, FAKE, FAKE, None) == 2
    assert L.moe_gate_topk(None, None, 4, 8, 2, 0, 1, 1.0, FAKE, FAKE, None) == 1
    assert L.moe_gate_topk(FAKE, None, 4, 8, 2, 5, 1, 1.0, FAKE, FAKE, None) == 3
    assert L.moe_gate_topk(FAKE + 2, None, 4, 8, 2, 0, 1, 1.0, FAKE, FAKE, None) == 4
    assert L.moe_gate_topk(None, None, 0, 8, 2, 0, 1, 1.0, None, None, None) == 0
    R = L.moe_router_gate_topk
    BIG = 1 << 40
    assert R(FAKE, FAKE, 4, 256, 8, 9, 0, 1, 1.0, None, None, FAKE, FAKE, FAKE, BIG, None) == 2   # top_k > E
    assert R(FAKE, FAKE, 4, 200, 8, 2, 0, 1, 1.0, None, None, FAKE, FAKE, FAKE, BIG, None) == 2   # H % 128
    assert R(FAKE, None, 4, 256, 8, 2, 0, 1, 1.0, None, None, FAKE, FAKE, FAKE, BIG, None) == 1
    assert R(FAKE, FAKE, 4, 256, 8, 2, 3, 1, 1.0, None, None, FAKE, FAKE, FAKE, BIG, None) == 3
    assert R(FAKE + 8, FAKE, 4, 256, 8, 2, 0, 1, 1.0, None, None, FAKE, FAKE, FAKE, BIG, None) == 4
    assert R(FAKE, FAKE, 4, 256, 8, 2, 0, 1, 1.0, None, FAKE + 1, FAKE, FAKE, FAKE, BIG, None) == 4
    assert R(FAKE, FAKE, 4, 256, 8, 2, 0, 1, 1.0, None, None, FAKE, FAKE, FAKE + 4, BIG, None) == 4
    need = L.moe_router_workspace_bytes(4, 256, 8)
    assert need > 0 and L.moe_router_workspace_bytes(4, 200, 8) == 0
    # many tokens x many experts: row ids (padded to 128 rows), offsets and
    # the logits of the GEMM form; fewer: the single kernel needs none
    al = lambda b: (b + 255) // 256 * 256  # noqa: E731
    assert L.moe_router_workspace_bytes(8192, 7168, 256) == al(8192 * 4) + 256 + al(8192 * 256 * 4)
    assert L.moe_router_workspace_bytes(4100, 512, 256) == al(4224 * 4) + 256 + al(4100 * 256 * 4)
    assert L.moe_router_workspace_bytes(4096, 4096, 64) == 0
    assert L.moe_router_workspace_bytes(300, 1024, 300) > 0    # 64-token tiles in K slices up to 1024 tokens
    assert L.moe_router_workspace_bytes(1025, 1024, 300) == 0
    assert L.moe_router_workspace_bytes(8192, 512, 100) == 0   # E % 8 != 0: the single kernel
    assert R(FAKE, FAKE, 4, 256, 8, 2, 0, 1, 1.0, None, None, FAKE, FAKE, FAKE, need - 1, None) == 5
    assert R(FAKE, FAKE, 4, 256, 8, 2, 0, 1, 1.0, None, None, FAKE, FAKE, None, BIG, None) == 5
    assert R(None, None, 0, 256, 8, 2, 0, 1, 1.0, None, None, None, None, None, 0, None) == 0
    cap = moe.moe_permute_capacity(10, 2, 8, 16)
    assert cap == 10 * 2 + 8 * 15
    assert L.moe_permute(FAKE, 10, 2, 8, 16, FAKE, FAKE, FAKE, cap - 1, None, 0, None) == 2
    assert L.moe_permute(FAKE, 10, 2, 8, 0, FAKE, FAKE, FAKE, cap, None, 0, None) == 2
    assert L.moe_permute(FAKE, 10, 2, 8, 16, None, FAKE, FAKE, cap, None, 0, None) == 1
    big = moe.moe_permute_workspace_bytes(100000, 8, 256)
    assert big > 0 and moe.moe_permute_workspace_bytes(10, 2, 8) == 0
    cap = moe.moe_permute_capacity(100000, 8, 256, 1)
    assert L.moe_permute(FAKE, 100000, 8, 256, 1, FAKE, FAKE, FAKE, cap, None, 0, None) == 5
    assert L.moe_act_quant_fp8(FAKE, 4, 100, FAKE, FAKE, None) == 2
    assert L.moe_act_quant_fp8(FAKE + 4, 4, 128, FAKE, FAKE, None) == 4


def test_workspace_layout_is_consistent():
    for wfmt, (T, H, E, I, k) in [("bf16", (16, 4096, 64, 1408, 6)), ("bf16", (4096, 4096, 64, 1408, 6)),
                                  ("fp8", (8192, 7168, 256, 2048, 8)), ("int4", (512, 4096, 128, 1536, 8)),
                                  ("fp8a16", (16, 7168, 256, 2048, 8)), ("mxfp4", (16, 7168, 256, 2048, 8)),
                                  ("mxfp4", (4096, 4096, 64, 1408, 6))]:
        a = B.make_args(T, H, E, I, k, wfmt=wfmt)
        L = moe.moe_workspace_layout(a)
        assert L["total"] == moe.moe_workspace_bytes(a)
        assert L["cap"] == T * k + E * (L["block_m"] - 1)
        offs = sorted(v for n, v in L.items() if n not in ("block_m", "cap", "total") and v >= 0)
        assert offs[0] == 0 and all(o % 256 == 0 for o in offs) and offs[-1] <= L["total"]
        assert (L["act_q"] >= 0) == (wfmt == "fp8")
        if wfmt == "mxfp4":  # the decode kernels' 16-row tile, the tiled kernels' 128 above 32 rows per expert
            assert L["block_m"] == (16 if T * k <= 32 * E else 128)


def test_int4_route_choice():
    # int4 takes the 16-row streamed kernels up to 8 routed rows per expert on
    # average when H and I are both K sizes they take (512..2048 in steps of
    # 512, 3072, 4096), the 64-row tiled kernels otherwise
    cases = [((16, 4096, 128, 1536, 8), 16), ((128, 4096, 128, 1536, 8), 16),
             ((129, 4096, 128, 1536, 8), 64), ((512, 4096, 128, 1536, 8), 64),
             ((4, 512, 8, 3072, 2), 16), ((4, 2048, 8, 512, 2), 16),
             ((4, 2560, 8, 512, 2), 64), ((4, 7168, 8, 2048, 2), 64),
             ((4, 1024, 8, 384, 2), 64), ((4, 384, 8, 1024, 2), 64)]
    for (T, H, E, I, k), bm in cases:
        a = B.make_args(T, H, E, I, k, wfmt="int4")
        L = moe.moe_workspace_layout(a)
        assert L["block_m"] == bm, (T, H, E, I, k, L["block_m"])
        assert L["act_s"] >= 0 and L["cap"] == T * k + E * (bm - 1)


def test_static_workspace_entry_point_validation():
    L = moe.lib()
    st = lambda a: L.moe_forward_static_ws(ctypes.byref(a), None)  # noqa: E731
    assert st(_args(top_k=9)) == B.MOE_ERR_SHAPE
    assert st(_args(hidden=None)) == B.MOE_ERR_NULL
    big = _args(T=4096, H=4096, E=64, I=1408, top_k=6)   # 599 MiB > the static workspace
    assert moe.moe_workspace_bytes(big) > B.STATIC_WS_BYTES
    assert st(big) == B.MOE_ERR_WORKSPACE
    assert st(_args(T=0)) == B.MOE_OK


def test_static_workspace_size_matches_header():
    src = open(os.path.join(ROOT, "include", "moe.h")).read()
    m = re.search(r"#define MOE_STATIC_WS_BYTES \((\d+)u << (\d+)\)", src)
    assert m and int(m.group(1)) << int(m.group(2)) == B.STATIC_WS_BYTES


def test_bf16_shapes_multiple_of_8_accepted():
    # bf16 weights take any H, I that are multiples of 8 (the tiled kernels
    # mask the ragged K step and column tile); the quantised formats keep 128
    for H, I in ((392, 200), (4104, 1416), (8, 8)):
        a = _args(H=H, I=I, T=4)
        assert moe.moe_workspace_bytes(a) > 0
        L = moe.moe_workspace_layout(a)
        assert L["block_m"] == 128      # never the 16-row decode kernels
        for wfmt in ("fp8", "int4", "fp8a16", "mxfp4"):
            assert moe.moe_workspace_bytes(_args(H=H, I=I, T=4, wfmt=wfmt)) == 0
    # a fused router needs H % 128 == 0
    a = _args(H=392, I=200)
    a.logits = None
    a.w_router = FAKE
    assert _fwd(a) == B.MOE_ERR_UNSUPPORTED
