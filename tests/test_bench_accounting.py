"""The algorithmic work bench.py divides by (CPU only): FLOP and byte counts
of the roofline against closed forms for known layers, and the choice of the
bound."""
import os
import sys

import pytest

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402
from paper_1903_01521_amd import workloads as wl  # noqa: E402


def test_bench_layer_counts():
    # N=1, C=K=64, 112x112, pad 1, F(4x4,3x3): 28 x 28 tiles, 36 positions
    L = wl.WORKLOADS["f4_n1_c64_k64_112x112"].first
    f = bench.layer_numbers(1, L)
    assert (f["Ho"], f["Wo"], f["P"], f["T"]) == (112, 112, 784, 36)
    assert f["direct_flops"] == 2 * 64 * 64 * 9 * 112 * 112
    # the multiplication count drops exactly 4x when the tiles cover the output
    assert f["gemm_flops"] * 4 == f["direct_flops"]
    assert f["bytes"]["fused"] == 4 * (64 * 112 * 112 * 2 + 36 * 64 * 64)


def test_f2_ratio_and_ragged_tiles():
    L = wl.WORKLOADS["f2_n1_c32_k32_56x56"].first
    f = bench.layer_numbers(1, L)
    assert f["gemm_flops"] * 9 == f["direct_flops"] * 4          # 2.25x fewer
    # 57x57 with m = 4: 15 x 15 tiles, the last row and column mostly padding
    L = wl.WORKLOADS["f4_n1_c48_k48_57x57"].first
    f = bench.layer_numbers(1, L)
    assert (f["Ho"], f["P"]) == (57, 225)
    assert f["gemm_flops"] == 2 * 36 * 225 * 48 * 48


def test_1d_and_5x5_counts():
    L = wl.WORKLOADS["f2r7w_n32_c192_k160_17x17"].first   # 1 x 7 along W, pad 3, m = 2
    f = bench.layer_numbers(32, L)
    assert (f["Ho"], f["Wo"], f["T"]) == (17, 17, 8)
    assert f["P"] == 32 * 17 * 9
    assert f["direct_flops"] == 2 * 32 * 160 * 192 * 7 * 17 * 17
    L = wl.WORKLOADS["f2r5_n32_c48_k64_35x35"].first       # 5 x 5, pad 2, m = 2: alpha = 6
    f = bench.layer_numbers(32, L)
    assert (f["Ho"], f["T"], f["P"]) == (35, 36, 32 * 18 * 18)


@pytest.mark.parametrize("name,kind,bound", [("f4_n1_c64_k64_112x112", "fused", "mfma"),
                                              ("f4_lowc_n64_c3_k64_224x224", "lowc", "hbm"),
                                              ("f4_n64_c256_k256_56x56", "input", "hbm"),
                                              ("f4_n64_c256_k256_56x56", "gemm", "mfma")])
def test_roofline_bound(name, kind, bound):
    w = wl.WORKLOADS[name]
    f = bench.layer_numbers(w.N, w.first)
    r = bench.roofline(kind, f, 1e-3)
    assert r["bound"] == bound
    if bound == "mfma":
        assert r["achieved"] == pytest.approx(f["flops"][kind] / 1e-3 / 1e12, rel=1e-3)
    else:
        assert r["achieved"] == pytest.approx(f["bytes"][kind] / 1e-3 / 1e9, rel=1e-3)


def test_sliced_fused_accounting_equals_fused():
    # Channel slices change how the fused kernel runs, not the layer's
    # algorithmic work: the same bytes and FLOPs as the unsliced kernel.
    L = wl.WORKLOADS["vgg16_stack_n1"].layers[8]            # 512 -> 512 at 28 x 28
    f = bench.layer_numbers(1, L)
    assert f["bytes"]["fused_sliced"] == f["bytes"]["fused"]
    assert f["flops"]["fused_sliced"] == f["flops"]["fused"]
    assert bench.kernel_label("fused_sliced") == "wino::k_fused + wino::k_slice_sum"
    assert bench.traffic_file("vgg16_stack_n1", "fused_sliced").endswith("traffic_vgg16_stack_n1.txt")


def test_mfma_summary_from_counter_rows(tmp_path, capsys):
    # Synthetic counter rows: the probe busy 0.85 of 1024 SIMDs over its active
    # cycles (summed over 8 XCDs), the bench layer's fused launch with the
    # padded instruction count of 1 x 16 blocks on a 28-tile-wide grid.
    import argparse
    w = wl.WORKLOADS["f4_n1_c64_k64_112x112"]
    need = bench.layer_numbers(w.N, w.first)["flops"]["fused"] / 2048
    insts = need * 32 / 28
    rows = [("void wino::k_mfma_probe(int, float*)", "SQ_VALU_MFMA_BUSY_CYCLES", 0.85 * 1024 * 1000),
            ("void wino::k_mfma_probe(int, float*)", "GRBM_GUI_ACTIVE", 8 * 1000),
            ("void wino::k_fused<4, 2, 4, 16, 1, 3>(float const*)", "SQ_INSTS_MFMA", insts),
            ("void wino::k_fused<4, 2, 4, 16, 1, 3>(float const*)", "SQ_VALU_MFMA_BUSY_CYCLES", 32 * insts),
            ("void wino::k_fused<4, 2, 4, 16, 1, 3>(float const*)", "GRBM_GUI_ACTIVE", 8 * 32 * insts / 1024 / 0.25)]
    with open(tmp_path / "run_counter_collection.csv", "w") as f:
        f.write("Kernel_Name,Counter_Name,Counter_Value\n")
        for k, c, v in rows:
            f.write(f'"{k}",{c},{v}\n')
    args = argparse.Namespace(workload="f4_n1_c64_k64_112x112", kind="fused", mfma_summary=str(tmp_path),
                              flags=None, write_summary=False)
    bench.mfma_summary(args)
    out = dict(l.split(": ", 1) for l in capsys.readouterr().out.splitlines() if not l.startswith("#"))
    assert float(out["mfma_insts_over_algorithmic"]) == pytest.approx(32 / 28, rel=1e-4)
    assert float(out["busy_cycles_per_inst"]) == pytest.approx(32.0)
    assert float(out["util_active"]) == pytest.approx(0.25, abs=1e-3)
    assert out["probe_util_active"].startswith("0.850")


def test_default_workload_is_the_large_layer():
    # N=64, C=K=256, 56x56, pad 1, F(4x4,3x3): 14 x 14 tiles per image
    assert wl.DEFAULT_BENCH == "f4_n64_c256_k256_56x56"
    w = wl.WORKLOADS[wl.DEFAULT_BENCH]
    f = bench.layer_numbers(w.N, w.first)
    assert (f["P"], f["T"]) == (64 * 14 * 14, 36)
    assert f["direct_flops"] == 2 * 64 * 256 * 256 * 9 * 56 * 56          # 236.76 GFLOP
    assert f["gemm_flops"] * 4 == f["direct_flops"]
    # the split call: x read, U read, y written
    assert f["bytes"]["split"] == 4 * (64 * 256 * 56 * 56 * 2 + 36 * 256 * 256)
    r = bench.roofline("split", f, 1e-3)
    assert r["bound"] == "mfma" and r["achieved"] == pytest.approx(f["gemm_flops"] / 1e-3 / 1e12, rel=1e-3)


def test_split_kernel_names():
    # The split call's input transform runs as k_vrows (by tile rows) or, for
    # very wide images, k_vblk (by 16-tile patches): either counts for it.
    assert bench.kernel_label("split") == "wino::k_vrows or wino::k_vblk + wino::k_gemm_out"
    pre = bench.KERNEL_NAMES["split"][0]
    assert bench.kernel_is("void wino::k_vrows<4, 1>(float const*, float*, wino::Geom, int, int, int)", pre)
    assert bench.kernel_is("void wino::k_vblk<4, 16, 1>(float const*, float*, wino::Geom, int, int, int)", pre)
    assert not bench.kernel_is("void wino::k_vrowsx<4>(float const*)", pre)
    assert not bench.kernel_is("void wino::k_gemm_out<4>(float const*)", pre)


def test_gemm16_accounting():
    # The 16-bit GEMM stage reads 16-bit V and U and writes fp32 M; its roof is
    # HBM at every shape here (the 16-bit matrix peak is 16x the fp32 one).
    L = wl.WORKLOADS["f4_n64_c256_k256_56x56"].first
    f = bench.layer_numbers(64, L)
    P = 64 * 14 * 14
    assert f["bytes"]["gemm16"] == 2 * 36 * P * 256 + 2 * 36 * 256 * 256 + 4 * 36 * P * 256
    r = bench.roofline("gemm16", f, 150e-6)
    assert r["bound"] == "hbm" and r["peak"] == 8000.0


def test_stage_table_from_trace(tmp_path, capsys):
    # A synthetic kernel trace of `bench.py --stage-trace` on the N=64 256-channel
    # layer: a weight transform, then per step a marker fill and the split
    # call's two kernels; the first of the four steps is the warm-up.
    import argparse
    import json
    name = "f4_n64_c256_k256_56x56"
    with open(tmp_path / "launches.json", "w") as f:
        json.dump({"workload": name, "flags": 0, "steps": 3, "warmup": 1, "launches": [["L0.conv", 0]]}, f)
    rows = [("void wino::k_filter<4, true, true, 3>(float const*, float*, int, int, int, long)", 5000)]
    for step, (tv, tg) in enumerate([(900e3, 900e3), (110e3, 520e3), (100e3, 500e3), (120e3, 540e3)]):
        rows.append(("void at::native::vectorized_elementwise_kernel<4, at::native::FillFunctor<float>>()", 2000))
        rows.append(("void wino::k_vrows<4, 1, 0>(float const*, float*, wino::Geom, int, int, int)", tv))
        rows.append(("void wino::k_gemm_out<4>(float const*, float const*, float*, wino::Geom)", tg))
    t = 1000
    with open(tmp_path / "run_kernel_trace.csv", "w") as f:
        f.write("Dispatch_Id,Kernel_Name,Start_Timestamp,End_Timestamp\n")
        for i, (k, d) in enumerate(rows):
            f.write(f'{i + 1},"{k}",{t},{t + int(d)}\n')
            t += int(d) + 100
    args = argparse.Namespace(stage_table=str(tmp_path), write_summary=False, tag="")
    bench.stage_table(args)
    out = capsys.readouterr().out.splitlines()
    body = [l.split() for l in out if l.startswith("L0.conv")]
    assert [r[5] for r in body] == ["input", "gemm_out"]
    f = bench.layer_numbers(64, wl.WORKLOADS[name].first)
    # medians of the three timed steps (the warm-up's 900 us is dropped)
    assert float(body[0][6]) == pytest.approx(110.0) and float(body[1][6]) == pytest.approx(520.0)
    # input transform: x read, V written, against HBM; GEMMs: against the fp32 MFMA peak
    assert body[0][9] == "hbm" and float(body[0][12]) == pytest.approx(f["bytes"]["input"] / 110e-6 / 8e12, abs=1e-3)
    assert body[1][9] == "mfma" and float(body[1][12]) == pytest.approx(f["gemm_flops"] / 520e-6 / 157.3e12, abs=1e-3)
    assert any(l.startswith("step: 630.0 us") for l in out)
