"""Host-side logic of bench.py: the GEMM1 kernel-name match used to pick the
dominant kernel out of rocprofv3 output, the counter-to-bytes scaling, and
the code-only source hash the committed counter summaries are keyed to."""
import csv
import os

import bench


def test_code_only_ignores_comments_and_whitespace():
    a = "int f(int x) {  // one\n  return x + 1; /* two\n lines */ }\n"
    b = "int f(int x) {\n\treturn x + 1;\n}  // other words\n"
    assert bench._code_only(a) == bench._code_only(b)
    assert bench._code_only(a) != bench._code_only(a.replace("x + 1", "x + 2"))


def test_kernel_source_hash_is_stable():
    h = bench.kernel_source_hash()
    assert len(h) == 16 and h == bench.kernel_source_hash()


def test_gemm1_kernel_match():
    yes = ["void moe::gemm_bf16_stream<0, 4, 4, 4, 8, true>(moe::GroupedGemm)",
           "void moe::moe_gemm_tiled<1, true, 128, 256, 2, 2, 8, 128, 3, 4>(moe::GroupedGemm)",
           "void moe::gemm_w4a16_skinny<4, 2, true>(moe::GroupedGemm)"]
    no = ["void moe::gemm_bf16_stream<0, 4, 4, 1, 11, false>(moe::GroupedGemm)",
          "void moe::moe_gemm_tiled<0, false, 128, 256, 2, 2, 8, 128, 3, 4>(moe::GroupedGemm)",
          "void moe::combine_kernel<true, false, 6>(void const*, float const*, int const*, int, int, int, void*)"]
    assert all(bench.gemm1_kernel_match(n) for n in yes)
    assert not any(bench.gemm1_kernel_match(n) for n in no)


def _write(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Value"])
        w.writeheader()
        for name, v in rows:
            w.writerow({"Kernel_Name": name, "Counter_Value": v})


def test_traffic_summary_scales_by_the_copy_kernel(tmp_path):
    g1 = "void moe::moe_gemm_tiled<0, true, 128, 256, 2, 2, 8, 128, 3, 4>(moe::GroupedGemm)"
    other = "void moe::combine_kernel<true, false, 6>(void const*)"
    copy = "__amd_rocclr_copyBuffer"
    f, w, cf, cw = (os.path.join(tmp_path, n) for n in ("f.csv", "w.csv", "cf.csv", "cw.csv"))
    _write(f, [(g1, 1000.0), (g1, 3000.0), (other, 9.0)])      # mean 2000 KiB
    _write(w, [(g1, 500.0), (other, 7.0)])
    _write(cf, [(copy, 512.0)])    # a 1 MiB copy reads as 512 KiB: scale 2
    _write(cw, [(copy, 2048.0)])   # and writes as 2048 KiB: scale 0.5
    r = bench.traffic_summary(f, w, cf, cw, 1)
    assert r["dispatches"] == [2, 1]
    assert r["fetch_scale"] == 2.0 and r["write_scale"] == 0.5
    assert r["hbm_fetch_bytes_per_launch"] == 2000 * 1024 * 2.0
    assert r["hbm_write_bytes_per_launch"] == 500 * 1024 * 0.5
    assert r["kernel_source_hash"] == bench.kernel_source_hash()
