"""The achievable-peak probes (include/moe_peaks.h) on the GPU: the copy
reproduces its source byte for byte, the read touches every word, the
MFMA-only loops, the read and the copy reach plausible fractions of
MI355X's published peaks (they are the denominators bench.py reports beside
those peaks), and the per-CU staging probes (global -> LDS copies, LDS
fragment reads) report rates in a plausible range."""
import pytest
import torch

import paper_2607_12875_amd as moe
from tests.gpu_util import require_gpu

pytestmark = pytest.mark.gpu


def test_peak_copy_is_exact():
    require_gpu()
    g = torch.Generator(device="cuda").manual_seed(5)
    src = torch.randint(0, 256, (3 << 20,), dtype=torch.uint8, device="cuda", generator=g)
    dst = torch.zeros_like(src)
    moe.moe_peak_copy(src, dst)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)


def test_peak_read_touches_every_word():
    # each 16-byte element is read by exactly one thread, so the XOR of all
    # per-workgroup folds is the XOR of every 32-bit word of the buffer
    require_gpu()
    g = torch.Generator(device="cuda").manual_seed(6)
    src = torch.randint(-2**31, 2**31 - 1, ((5 << 20) + 12,), dtype=torch.int32, device="cuda", generator=g)
    sink = torch.zeros(moe.moe_peak_sink_elems(), dtype=torch.int32, device="cuda")
    moe.moe_peak_read(src, sink)
    torch.cuda.synchronize()
    a = src.cpu().numpy().view("uint32")
    b = sink.cpu().numpy().view("uint32")
    import numpy as np
    assert int(np.bitwise_xor.reduce(a)) == int(np.bitwise_xor.reduce(b))


def test_measured_peaks_are_plausible():
    require_gpu()
    import bench
    p = bench.measure_peaks(moe, torch)
    print(f"  measured peaks: {p}", flush=True)
    # published: dense bf16 2.5 PFLOP/s, dense fp8 5.0 PFLOP/s, HBM 8 TB/s
    assert 0.3 * 2500 < p["mfma_bf16_tflops"] < 1.05 * 2500
    assert 0.3 * 5000 < p["mfma_fp8_tflops"] < 1.05 * 5000
    assert 0.3 * 8000 < p["hbm_read_gbs"] < 1.05 * 8000
    assert 0.3 * 8000 < p["hbm_copy_gbs"] < 1.05 * 8000
    # per-CU staging paths, bytes per clock per CU at 2.4 GHz (measured on
    # MI355X: about 35 / 55 from L2 with 4 / 8 copy waves, 10-12 from HBM
    # with either, LDS reads about 160 / 240 with 4 / 16 waves); the bounds
    # only catch a probe that stopped measuring what it names
    for w in (4, 8):
        assert 8 < p[f"l2_to_lds_w{w}_bytes_per_clk_cu"] < 128
        assert 3 < p[f"hbm_to_lds_w{w}_bytes_per_clk_cu"] < 20
    assert p["l2_to_lds_w8_bytes_per_clk_cu"] > p["hbm_to_lds_w8_bytes_per_clk_cu"]
    for w in (4, 16):
        assert 60 < p[f"lds_read_w{w}_bytes_per_clk_cu"] < 520
