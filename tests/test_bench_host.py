"""Host-side logic of bench.py (no GPU): the algorithmic work of each stage
and the splitting of a rocprofv3 kernel trace into scoring calls and stages."""
import csv
import os

import numpy as np

import bench
from paper_2007_16122_amd import synth


def _batch(cfg, R, Q):
    return {"n_rows": R, "req_off": np.linspace(0, R, Q + 1).astype(np.int32),
            "seq_off": np.zeros(1, np.int32)}


def test_fused_stage_work_is_layer_plus_tail():
    cfg = synth.CONFIGS["serving_bf16"]
    b = _batch(cfg, 64_000, 32)
    kind, fused = bench.stage_work(cfg, b, "dense_tail")
    _, layer = bench.stage_work(cfg, b, "dense2")
    _, tail = bench.stage_work(cfg, b, "tail")
    assert kind == "mfma"
    assert fused == layer + tail
    # 2 * R * (512*256 + 256*128 + 128*64 + 64*2) for the serving widths
    assert fused == 2.0 * 64_000 * (512 * 256 + 256 * 128 + 128 * 64 + 64 * 2)


def test_mlp_flops_of_the_staged_path_cover_the_network():
    cfg = synth.CONFIGS["serving_bf16"]
    b = _batch(cfg, 64_000, 32)
    staged = sum(bench.stage_work(cfg, b, st)[1] for st in ("dense0", "dense1", "dense_tail"))
    w = cfg.widths
    assert staged == 2.0 * 64_000 * sum(w[i] * w[i + 1] for i in range(len(w) - 1))


MANGLED = {
    "gather": "_ZN4cold16gather_se_kernelIDF16bLi{m}ELb0ELb0ELi8ELb0EEEvNS_10GatherArgsE",
    "dense": "_ZN4cold21dense_relu_buf_kernelIDF16bLi128ELi128ELi2ELi2ELi2ELi64EEEvPKT_S3_PKfPS1_liiii",
    "fused": "_ZN4cold17dense_tail_kernelIDF16bLi64ELi2EEEvPKT_S3_PKfliiS3_S5_S3_S5_S3_S5_iPf",
}
DEMANGLED_GATHER = "void cold::gather_se_kernel<bool _Accum, int, E, false, false, 8, false>(cold::GatherArgs)"
MASK = ["cold::mask_partial_kernel(float const*, int const*, long, int, int, float*)",
        "cold::mask_select_kernel(float const*, int const*, long, int, int, int, unsigned char*, unsigned char*)"]


def _wide_call():
    """Kernel names of one scoring call of a model with a group mask, with
    the importance pass and the mask kernels printed demangled."""
    return [DEMANGLED_GATHER, *MASK, MANGLED["gather"].format(m=2), MANGLED["dense"],
            MANGLED["dense"], MANGLED["fused"]]


def _write_trace(path, calls):
    t = 1000
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, ["Kernel_Name", "Start_Timestamp", "End_Timestamp", "Grid_Size_X"])
        w.writeheader()
        w.writerow({"Kernel_Name": "void at::native::fill_kernel", "Start_Timestamp": t,
                    "End_Timestamp": t + 5, "Grid_Size_X": 1})
        for call in calls:
            for name in call:
                t += 1000
                w.writerow({"Kernel_Name": name, "Start_Timestamp": t, "End_Timestamp": t + 500,
                            "Grid_Size_X": 256})


def test_trace_split_handles_demangled_names(tmp_path):
    d = tmp_path / "trace"
    d.mkdir()
    _write_trace(os.path.join(d, "bench_kernel_trace.csv"), [_wide_call(), _wide_call()])
    rows = list(csv.DictReader(open(os.path.join(d, "bench_kernel_trace.csv"))))
    stages = [st for st, _ in bench._last_call(rows)]
    assert stages == ["se_weights", "group_mask", "group_mask", "gather_apply", "dense0",
                      "dense1", "dense_tail"]
    text = bench.summarize_trace(str(d), "cmd")
    assert "# 2 calls profiled" in text
    lines = {l.split()[0]: l.split() for l in text.splitlines() if l and not l.startswith(("#", "stage"))}
    assert int(lines["se_weights"][1]) == 2
    assert int(lines["group_mask"][1]) == 4      # two kernels per call
    assert float(lines["dense_tail"][2]) == 0.5  # mean duration in us


def test_trace_split_of_the_topk_rows_path_and_register_gather(tmp_path):
    """The wide workload's passes (gather with squeeze, row-wise SE, one mask
    kernel, compacted reweighting) and the register-resident gathers of the
    other workloads map to their stage names, one call each; the fp32
    matrix-core layer is the SE layer after the raw gather of the literal
    Eq. 2 form and a hidden layer of an fp32 model otherwise."""
    wide = ["_ZN4cold16gather_se_kernelIDF16bLi4ELb0ELb0ELi8ELb0EEEvNS_10GatherArgsE",
            "void cold::se_rows_kernel<16>(float const*, float*, long, int, int, "
            "HIP_vector_type<float, 4u> const*, float const*, HIP_vector_type<float, 4u> const*, "
            "float const*, float*)",
            "cold::mask_select_tiles_kernel(float const*, float const*, int const*, long, int, int, "
            "unsigned char*, unsigned char*, int*)",
            "_ZN4cold20apply_compact_kernelIDF16bLb0EEEvPKT_PS1_PKfPKiS8_lliiiiijlPK15HIP_vector_"
            "typeIjLj4EElPS9_ilPNS_7RowTileEPi",
            MANGLED["dense"], MANGLED["dense"], MANGLED["fused"]]
    tiny = ["void cold::gather_full_chain_kernel<float, false, false, true>(cold::GatherArgs)",
            "void cold::dense_f32_mfma_kernel<1, 1>(float const*, float const*, float const*, "
            "float*, long, int, int)",
            "void cold::dense_f32_mfma_kernel<1, 1>(float const*, float const*, float const*, "
            "float*, long, int, int)",
            "void cold::head_kernel<float>(float const*, float const*, float const*, float*, long, "
            "int, int)"]
    literal = ["_ZN4cold16gather_se_kernelIfLi3ELb0ELb0ELi8ELb0EEEvNS_10GatherArgsE",
               "void cold::dense_f32_mfma_kernel<2, 4>(float const*, float const*, float const*, "
               "float*, long, int, int)",
               "_ZN4cold16gather_se_kernelIfLi2ELb0ELb0ELi8ELb0EEEvNS_10GatherArgsE",
               "void cold::dense_f32_mfma_kernel<1, 1>(float const*, float const*, float const*, "
               "float*, long, int, int)",
               "void cold::head_kernel<float>(float const*, float const*, float const*, float*, "
               "long, int, int)"]
    serving = ["_ZN4cold16user_pool_kernelIDF16bLb0EEEvNS_10GatherArgsE",
               "_ZN4cold18gather_full_kernelIDF16bLb0ELb0ELi12ELb0EEEvNS_10GatherArgsE",
               MANGLED["dense"], MANGLED["dense"], MANGLED["fused"]]
    large = ["_ZN4cold16user_pool_kernelIDF16_Lb1EEEvNS_10GatherArgsE",
             "_ZN4cold24gather_full_split_kernelIDF16_Lb1ELb1ELb0EEEvNS_10GatherArgsE",
             MANGLED["dense"], MANGLED["dense"], MANGLED["fused"]]
    for calls, want in [
            ([wide, wide], ["gather_sq", "se_rows", "group_mask", "apply_compact", "dense0",
                            "dense1", "dense_tail"]),
            ([tiny, tiny], ["gather_se", "dense0", "dense1", "head"]),
            ([literal], ["gather_raw", "se_dense", "gather_apply", "dense0", "head"]),
            ([serving, serving], ["user_pool", "gather_se", "dense0", "dense1", "dense_tail"]),
            ([large], ["user_pool", "gather_se", "dense0", "dense1", "dense_tail"])]:
        d = tmp_path / want[1] / str(len(calls))
        d.mkdir(parents=True)
        _write_trace(os.path.join(d, "bench_kernel_trace.csv"), calls)
        rows = list(csv.DictReader(open(os.path.join(d, "bench_kernel_trace.csv"))))
        assert [st for st, _ in bench._last_call(rows)] == want
        text = bench.summarize_trace(str(d), "cmd")
        assert f"# {len(calls)} calls profiled" in text


def test_single_request_summary_keeps_the_small_calls(tmp_path):
    """The latency-loop trace summary splits the trace into calls at the
    gather kernel, keeps the calls whose kernels are all small (a 2,000-ad
    request), and labels the dense layers in call order."""
    one = ["void cold::gather_full_chain_kernel<__bf16, false, false, true>(cold::GatherArgs)",
           MANGLED["dense"], MANGLED["dense"], MANGLED["fused"]]
    batch = ["_ZN4cold16user_pool_kernelIDF16bLb0EEEvNS_10GatherArgsE",
             "_ZN4cold18gather_full_kernelIDF16bLb0ELb0ELi12ELb0EEEvNS_10GatherArgsE",
             MANGLED["dense"], MANGLED["dense"], MANGLED["fused"]]
    d = tmp_path / "lat"
    d.mkdir()
    path = os.path.join(d, "bench_kernel_trace.csv")
    _write_trace(path, [batch, one, one, one])
    rows = list(csv.DictReader(open(path)))
    big = rows[1]["Kernel_Name"], rows[2]["Kernel_Name"]
    with open(path, "w", newline="") as fh:   # the whole-batch call has a large grid
        w = csv.DictWriter(fh, list(rows[0].keys()))
        w.writeheader()
        for i, r in enumerate(rows):
            if 1 <= i <= 5:
                r["Grid_Size_X"] = 512000
            w.writerow(r)
    assert big[0].startswith("_ZN4cold16user_pool")
    text = bench.summarize_single_request(str(d), "cmd")
    assert "# 3 single-request calls" in text
    assert "a call = gather_se, dense0, dense1, dense_tail on 2,000 rows" in text
    lines = {l.split()[0]: l.split() for l in text.splitlines() if l and not l.startswith(("#", "stage", "gaps", "first"))}
    assert list(lines) == ["gather_se", "dense0", "dense1", "dense_tail"]
    assert float(lines["dense1"][1]) == 0.5                       # median duration in us
    assert "gaps between consecutive kernels, median us: 0.50, 0.50, 0.50" in text
    assert "first kernel start to last kernel end, median us: 3.50" in text


def test_probe_traffic_summary_scales_by_the_largest_copy(tmp_path):
    """The probe's counter summary scales each counter so that the largest
    copy (the 1 GiB probe copy) moves exactly its size, and takes the median
    over the probe's dispatches."""
    dirs = []
    for counter, copy_kib, probe_kib in (("FETCH_SIZE", 524288.0, [1000.0, 1000.0, 5000.0]),
                                         ("WRITE_SIZE", 1048576.0, [2000.0, 2000.0, 2000.0])):
        d = tmp_path / counter
        d.mkdir()
        with open(os.path.join(d, "bench_counter_collection.csv"), "w", newline="") as fh:
            w = csv.DictWriter(fh, ["Kernel_Name", "Counter_Name", "Counter_Value"])
            w.writeheader()
            w.writerow({"Kernel_Name": "__amd_rocclr_copyBuffer", "Counter_Name": counter,
                        "Counter_Value": 12.0})
            w.writerow({"Kernel_Name": "__amd_rocclr_copyBuffer", "Counter_Name": counter,
                        "Counter_Value": copy_kib})
            for v in probe_kib:
                w.writerow({"Kernel_Name": "(anonymous namespace)::row_gather_probe_kernel(...)",
                            "Counter_Name": counter, "Counter_Value": v})
        dirs.append(str(d))
    text = bench.summarize_probe(dirs[0], dirs[1], 1024, "cmd")
    assert "FETCH_SIZE scaled by 2.000, WRITE_SIZE by 1.000" in text
    assert "median over 3 dispatches" in text
    row = [l.split() for l in text.splitlines() if l.startswith("row_gather_probe")][0]
    assert float(row[1]) == round(2000.0 * 1024 / 1e6, 1)   # fetch MB: 1000 KiB x 2
    assert float(row[2]) == round(2000.0 * 1024 / 1e6, 1)   # write MB: 2000 KiB x 1
