"""Host logic of bench.py (no GPU): the counter-traffic summaries it writes and reads, the
source-hash check that retires a stale summary, and the roofline entry."""
import argparse
import csv
import importlib.util
import os
import shutil

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _summary(path):
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    return kv


def test_committed_traffic_summaries_match_the_sources(bench):
    """Every committed counter summary was taken on the current kernel sources, so the
    bench reports its traffic rather than null."""
    files = [f for f in os.listdir(os.path.join(ROOT, "profiles")) if f.startswith("traffic_")]
    assert files
    by_symbol = {v: k for k, v in bench.KERNEL_SYMBOL.items()}
    for f in files:
        kv = _summary(os.path.join(ROOT, "profiles", f))
        kernel = by_symbol[kv["kernel"]]
        assert f == f"traffic_{kernel}_{kv['workload']}.txt"
        bytes_, note = bench._traffic(kernel, kv["workload"])
        assert bytes_ is not None, (f, note)
        assert bytes_ == pytest.approx(float(kv["hbm_bytes_per_launch"]))


def _write_pmc(run_dir, counter, rows):
    os.makedirs(run_dir, exist_ok=True)
    with open(os.path.join(run_dir, "run_counter_collection.csv"), "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for i, (name, value) in enumerate(rows):
            w.writerow([i, name, counter, value])


def test_summarize_pmc_scales_by_the_copy_calibration(bench, tmp_path, monkeypatch):
    """FETCH_SIZE and WRITE_SIZE are scaled by what they read for a 1 GiB copy; the summary
    is read back while its source hash matches and retired once the source changes."""
    root = tmp_path / "repo"
    shutil.copytree(os.path.join(ROOT, "paper_2606_28831_amd", "csrc"),
                    root / "paper_2606_28831_amd" / "csrc")
    (root / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(root))
    sym = bench.KERNEL_SYMBOL["compact_gather"]
    d = tmp_path / "pmc"
    # the copy reads as half its bytes on FETCH_SIZE and in full on WRITE_SIZE
    _write_pmc(d / "cf", "FETCH_SIZE", [("__amd_rocclr_copyBuffer", 524288.0)] * 3)
    _write_pmc(d / "cw", "WRITE_SIZE", [("__amd_rocclr_copyBuffer", 1048576.0)] * 3)
    _write_pmc(d / "pf", "FETCH_SIZE", [(f"void hk::{sym}<256>(...)", 1000.0),
                                        (f"void hk::{sym}<256>(...)", 3000.0),
                                        ("hk::other_kernel", 99999.0)])
    _write_pmc(d / "pw", "WRITE_SIZE", [(f"void hk::{sym}<256>(...)", 500.0)])
    args = argparse.Namespace(summarize_pmc=[str(d / "pf"), str(d / "pw"), str(d / "cf"),
                                             str(d / "cw")],
                              kernel="compact_gather", workload="unit", command="test")
    out = bench.summarize_pmc(args)
    read = 2000.0 * 1024 * 2.0          # mean 2000 KiB fetched, scale 2
    write = 500.0 * 1024 * 1.0
    assert out["hbm_bytes_per_launch"] == pytest.approx(read + write)
    kv = _summary(out["traffic_summary"])
    assert float(kv["fetch_scale"]) == pytest.approx(2.0)
    assert float(kv["write_scale"]) == pytest.approx(1.0)
    assert int(kv["dispatches_fetch"]) == 2
    got, note = bench._traffic("compact_gather", "unit")
    assert got == pytest.approx(read + write), note
    src = root / "paper_2606_28831_amd" / "csrc" / bench.KERNEL_SOURCE["compact_gather"]
    src.write_text(src.read_text() + "\n// changed\n")
    got, note = bench._traffic("compact_gather", "unit")
    assert got is None and "changed" in note


def test_roofline_takes_the_kernel_with_the_largest_share(bench, monkeypatch):
    monkeypatch.setattr(bench, "_traffic", lambda k, w: (None, "none"))
    ktime = {"a": {"avg_ms": 0.5, "ms_per_step": 0.5, "launches_per_step": 1.0},
             "b": {"avg_ms": 0.2, "ms_per_step": 0.6, "launches_per_step": 3.0},
             "c": {"avg_ms": 9.0, "ms_per_step": 9.0, "launches_per_step": 1.0}}
    per_launch = {"a": (4e9, 0.0), "b": (1e9, 2e12)}     # "c" has no byte count: not a candidate
    r = bench._roofline(ktime, per_launch, "w")
    assert r["kernel"] == "b"
    assert r["achieved"] == pytest.approx(1e9 / 0.2e-3 / 1e9)
    assert r["frac"] == pytest.approx(r["achieved"] / bench.HBM_PEAK_GBS)
    assert r["mfma_tflops"] == pytest.approx(2e12 / 0.2e-3 / 1e12)


def test_workload_state_is_one_buffer_and_restores_whole():
    """The five mutable metadata tensors are 256-byte-aligned views of one buffer, and a
    clone / restore round trip brings every one of them back."""
    import torch
    import workload as WL
    w = WL.make_workload(WL.config(1), "cpu")
    base = w.meta.data_ptr()
    end = base + w.meta.numel()
    names = ("page_table", "page_mask", "n_pages", "free_ids", "free_top")
    for k in names:
        t = getattr(w, k)
        assert base <= t.data_ptr() and t.data_ptr() + t.numel() * t.element_size() <= end, k
        assert (t.data_ptr() - base) % 256 == 0, k
    before = {k: getattr(w, k).clone() for k in names}
    st = WL.clone_state(w)
    for k in names:
        getattr(w, k).fill_(7)
    WL.restore_state(w, st)
    for k in names:
        assert torch.equal(getattr(w, k), before[k]), k


def test_committed_mfma_summaries_match_the_sources(bench):
    """Every committed MFMA counter summary was taken on the current kernel source."""
    files = [f for f in os.listdir(os.path.join(ROOT, "profiles")) if f.startswith("mfma_")]
    by_symbol = {v: k for k, v in bench.KERNEL_SYMBOL.items()}
    for f in files:
        kv = _summary(os.path.join(ROOT, "profiles", f))
        kernel = by_symbol[kv["kernel"]]
        assert f == f"mfma_{kernel}_{kv['workload']}.txt"
        assert kv["source_sha256"] == bench._source_sha(kernel), f


def test_summarize_mfma_normalisation(bench, tmp_path, monkeypatch):
    """Busy cycles are 32 per MFMA summed over the SIMDs, GRBM_GUI_ACTIVE is summed over the
    XCDs, and the duration comes from each dispatch's timestamps."""
    root = tmp_path / "repo"
    shutil.copytree(os.path.join(ROOT, "paper_2606_28831_amd", "csrc"),
                    root / "paper_2606_28831_amd" / "csrc")
    (root / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(root))
    sym = bench.KERNEL_SYMBOL["score_pass1"]
    run = tmp_path / "pmc"
    run.mkdir()
    ops = 7 * 2 ** 20                           # MFMAs per dispatch
    ns = 300e3                                  # 300 us
    cycles = 2.0 * ns                           # 2 GHz
    with open(run / "run_counter_collection.csv", "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value",
                    "Start_Timestamp", "End_Timestamp"])
        for i in range(2):
            for name, value in (("SQ_VALU_MFMA_BUSY_CYCLES", 32 * ops),
                                ("GRBM_GUI_ACTIVE", 8 * cycles)):
                w.writerow([i, f"void hk::{sym}<128, 7>(...)", name, value, 1000, 1000 + ns])
        w.writerow([9, "hk::other_kernel", "SQ_VALU_MFMA_BUSY_CYCLES", 1, 0, 10])
    args = argparse.Namespace(summarize_mfma=str(run), kernel="score_pass1", workload="unit",
                              command="test")
    out = bench.summarize_mfma(args)
    assert out["dispatches"] == 2
    assert out["mfma_ops_per_dispatch"] == pytest.approx(ops)
    assert out["mfma_flop_per_dispatch"] == pytest.approx(ops * 32768)
    assert out["clock_ghz"] == pytest.approx(2.0)
    assert out["mfma_busy_frac_of_simd_cycles"] == pytest.approx(32 * ops / (cycles * 1024))
    assert out["mfma_tflops"] == pytest.approx(ops * 32768 / ns / 1e3)
    kv = _summary(out["mfma_summary"])
    assert kv["source_sha256"] == bench._source_sha("score_pass1")


def test_bench_line_reads_the_committed_mfma_counters(bench):
    w = "cfg3_l1_b32_h28x4_d128_n32768_bf16_tempered"
    for k in ("score_pass1", "score_pass2"):
        got = bench._mfma_counters(k, w)
        assert got is not None, k
        assert 0.0 < got["busy_frac_of_simd_cycles"] < 1.0
        assert got["flop_counted"] == pytest.approx(2.405e11, rel=1e-3)
    assert bench._mfma_counters("score_pass1", "no_such_workload") is None
