"""Host logic of bench.py (no GPU): the kernel-name to timing-class map the
rocprofv3 tables rely on, the counter and trace summaries written from
synthetic rocprofv3 CSV files, and the read-back of stored traffic (which
must refuse numbers taken on other kernel sources)."""
import csv
import json
import os

import pytest

import bench

GEMM = ("void gcn::(anonymous namespace)::gemm_kernel<(gcn::ALayout)1, (gcn::BLayout)0, "
        "(gcn::Epilogue)4, true, (gcn::GemmRole){}>(gcn::GemmBatch)")
GEMM16 = GEMM.replace("gemm_kernel<", "gemm_bf16_kernel<")
H16 = ("void gcn::(anonymous namespace)::gemm_h16_kernel<(gcn::ALayout)1, (gcn::BLayout)0, "
       "(gcn::Epilogue)4, (gcn::GemmRole){}>(gcn::GemmBatch)")
H16S = ("void gcn::(anonymous namespace)::gemm_h16s_kernel<(gcn::Epilogue)3, (gcn::GemmRole){}, "
        "2>(gcn::GemmBatch)")
LIST = ("void gcn::(anonymous namespace)::list_sums_kernel<32, 1, false, 1>(int4 const*, "
        "int const*, int, int const*, gcn::RowSource, float const*, float const*, float*, long, "
        "int, int, int, __bf16*, long)")
PAIR = ("void gcn::(anonymous namespace)::pair_sums_kernel<64, 2, true>(int4 const*, int, "
        "int const*, gcn::RowSource, float const*, float*, long, int, int, int)")


@pytest.mark.parametrize("role,cls", list(enumerate(bench._ROLE_CLASS)))
def test_gemm_roles_map_to_classes(role, cls):
    assert bench.kernel_class(GEMM.format(role)) == cls
    assert bench.kernel_class(GEMM16.format(role)) == cls + "_bf16"
    assert bench.kernel_class(H16.format(role)) == cls + "_bf16"
    assert bench.kernel_class(H16S.format(role)) == cls + "_bf16"


def test_other_kernels_map_to_classes():
    assert bench.kernel_class(PAIR) == "pair_sums"
    assert bench.kernel_class(LIST) == "list_sums"
    cases = {
        "void gcn::(anonymous namespace)::sgd_reduce_kernel<2>(gcn::SgdProblem)": "sgd_reduce",
        "void gcn::(anonymous namespace)::loss_kernel<2, true>(int, int)": "loss_rows",
        "gcn::(anonymous namespace)::mean_kernel(int, float const*, float, float*)": "loss_mean",
        "gcn::(anonymous namespace)::to_bf16_kernel(gcn::(anonymous namespace)::ConvBatch)":
            "to_bf16",
        "__amd_rocclr_copyBuffer": None,
        "void at::native::vectorized_elementwise_kernel<4>(int)": None,
    }
    for name, cls in cases.items():
        assert bench.kernel_class(name) == cls, name


def _write_counters(path, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for name, counter, value in rows:
            w.writerow(dict(Kernel_Name=name, Counter_Name=counter, Counter_Value=value))


@pytest.fixture
def scratch_root(tmp_path, monkeypatch):
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    return tmp_path


def test_pmc_summary_scales_by_the_calibration_copy(scratch_root):
    fetch, write = scratch_root / "fetch.csv", scratch_root / "write.csv"
    dw, lst = GEMM.format(4), LIST.format("false")
    # the 1 MiB copy reads 512 KiB by FETCH_SIZE (factor 2) and 1024 KiB by WRITE_SIZE
    _write_counters(fetch, [("__amd_rocclr_copyBuffer", "FETCH_SIZE", 512.0),
                            (dw, "FETCH_SIZE", 100.0), (dw, "FETCH_SIZE", 300.0),
                            (lst, "FETCH_SIZE", 50.0)])
    _write_counters(write, [("__amd_rocclr_copyBuffer", "WRITE_SIZE", 1024.0),
                            (dw, "WRITE_SIZE", 10.0), (dw, "WRITE_SIZE", 30.0),
                            (lst, "WRITE_SIZE", 5.0)])
    args = dict(steps=3, warmup=1, profile_steps=1, calib_copy_mib=1)
    bench.pmc_summary(str(fetch), str(write), "wl", args)
    txt = (scratch_root / "profiles" / "wl_hbm_traffic.md").read_text()
    blob = json.loads(txt.split("```json", 1)[1].split("```", 1)[0])
    assert blob["scale"] == {"FETCH_SIZE": 2.0, "WRITE_SIZE": 1.0}
    # mean of the two launches: (200 KiB fetch x 2 + 20 KiB write) per launch
    assert blob["classes"]["gemm_dw"]["bytes_per_launch"] == 1024 * (200 * 2 + 20)
    assert blob["classes"]["gemm_dw"]["dispatches"] == 2
    assert blob["classes"]["list_sums"]["bytes_per_launch"] == 1024 * (50 * 2 + 5)
    # read back while the sources are unchanged; refused once a hash differs
    assert bench.stored_traffic("wl", "gemm_dw") == 1024 * 420
    assert bench.stored_traffic("wl", "pair_sums") is None
    blob["classes"]["gemm_dw"]["source_hash"] = "0" * 16
    (scratch_root / "profiles" / "wl_hbm_traffic.md").write_text(
        txt.split("```json")[0] + "```json\n" + json.dumps(blob) + "\n```\n")
    assert bench.stored_traffic("wl", "gemm_dw") is None


def test_pmc_summary_needs_exactly_one_calibration_copy(scratch_root):
    fetch, write = scratch_root / "fetch.csv", scratch_root / "write.csv"
    _write_counters(fetch, [(GEMM.format(0), "FETCH_SIZE", 1.0)])
    _write_counters(write, [(GEMM.format(0), "WRITE_SIZE", 1.0)])
    with pytest.raises(SystemExit):
        bench.pmc_summary(str(fetch), str(write), "wl",
                          dict(steps=1, warmup=1, profile_steps=1, calib_copy_mib=1))


def test_l2_summary_hit_rate(scratch_root):
    path = scratch_root / "l2.csv"
    lst = LIST.format("false")
    _write_counters(path, [(lst, "TCC_HIT_sum", 300.0), (lst, "TCC_MISS_sum", 100.0),
                           (lst, "TCC_HIT_sum", 500.0), (lst, "TCC_MISS_sum", 100.0)])
    bench.l2_summary(str(path), "wl", dict(steps=3, warmup=1, profile_steps=1))
    txt = (scratch_root / "profiles" / "wl_l2_hit_rate.md").read_text()
    row = [ln for ln in txt.splitlines() if ln.startswith("| list_sums |")][0]
    cells = [c.strip() for c in row.strip("|").split("|")]
    assert cells == ["list_sums", "2", "400", "100", "0.800"]


def test_trace_summary_totals_per_class(scratch_root):
    path = scratch_root / "stats.csv"
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Name", "Calls", "TotalDurationNs", "AverageNs"])
        w.writeheader()
        w.writerow(dict(Name=GEMM.format(4), Calls=4, TotalDurationNs=400000, AverageNs=100000))
        w.writerow(dict(Name=GEMM.format(4).replace("true", "false"), Calls=1,
                        TotalDurationNs=200000, AverageNs=200000))
        w.writerow(dict(Name="__amd_rocclr_copyBuffer", Calls=9, TotalDurationNs=9000,
                        AverageNs=1000))
    bench.trace_summary(str(path), "wl", "--no-cpu-baseline --no-direct --no-narrow --no-adam --no-extra")
    txt = (scratch_root / "profiles" / "wl_train_step_kernel_stats.md").read_text()
    row = [ln for ln in txt.splitlines() if ln.startswith("| gemm_dw |")][0]
    cells = [c.strip() for c in row.strip("|").split("|")]
    assert cells == ["gemm_dw", "5", "120.00", "0.600"]   # 5 calls, 600 us in all
    assert "step alone" in txt


def test_trace_summary_names_the_bf16_variant(scratch_root):
    path = scratch_root / "stats.csv"
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Name", "Calls", "TotalDurationNs", "AverageNs"])
        w.writeheader()
        w.writerow(dict(Name=H16.format(0), Calls=2, TotalDurationNs=100000, AverageNs=50000))
    bench.trace_summary(str(path), "wl", "--precision bf16 --no-cpu-baseline")
    txt = (scratch_root / "profiles" / "wl_bf16_train_step_kernel_stats.md").read_text()
    assert "bf16 training step" in txt
    assert "| gemm_fwd_bf16 | 2 | 50.00 | 0.100 |" in txt


def test_infer_workload_is_the_ppi_model_on_a_whole_graph():
    from paper_2001_02498_amd import synth
    ppi = synth.WORKLOADS["ppi8k"]
    wl = bench.infer_workload(20000)
    assert (wl.n, wl.name) == (20000, "full20k")
    assert (wl.L, wl.f_in, wl.h, wl.C, wl.loss) == (ppi.L, ppi.f_in, ppi.h, ppi.C, ppi.loss)
    assert (wl.gamma, wl.dbar, wl.theta, wl.rounds, wl.budget) == (
        ppi.gamma, ppi.dbar, ppi.theta, ppi.rounds, ppi.budget)
    assert wl.reduce


def test_trace_summary_names_inference(scratch_root):
    path = scratch_root / "stats.csv"
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Name", "Calls", "TotalDurationNs", "AverageNs"])
        w.writeheader()
        w.writerow(dict(Name=GEMM.format(0), Calls=2, TotalDurationNs=100000, AverageNs=50000))
    bench.trace_summary(str(path), "full9k", "--infer --no-cpu-baseline --no-direct")
    txt = (scratch_root / "profiles" / "full9k_infer_kernel_stats.md").read_text()
    assert "full9k inference" in txt and "inference calls" in txt
