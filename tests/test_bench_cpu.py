"""CPU checks of bench.py's measurement plumbing: the one-GPU guard, the
kernel-kind table against the kinds the library times, and the rocprofv3
summaries (counter scaling by the calibration copy, the source-digest gate on
`roofline.traffic`) on small synthetic CSV files."""
import csv
import json
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert out.returncode == 2
    assert "one GPU" in out.stderr
    assert out.stdout == ""


def test_every_timed_kind_has_a_bound():
    src = open(os.path.join(ROOT, "paper_2512_13728_amd", "csrc", "api.cpp")).read()
    block = re.search(r'"form_buffer", "form_buffer_local".*?};', src, flags=re.S).group(0)
    kinds = re.findall(r'"([a-z0-9_]+)"', block)
    assert len(kinds) == len(set(kinds)) >= 10
    for k in kinds:
        assert k in bench.KIND_BOUND, k
        bound, dtype, mult = bench.KIND_BOUND[k]
        assert bound in ("hbm", "mfma", "alu")
        assert (dtype is None) == (bound == "hbm")
        if dtype is not None:
            assert dtype in bench.PEAK_TFLOPS
    # the kinds with a profiler pattern name existing kinds and sources
    for k, (pat, files) in bench.KIND_KERNEL.items():
        assert k in kinds
        for f in files:
            assert os.path.exists(os.path.join(bench.CSRC, f)), f


def _write_pmc(dirpath, counter, rows):
    os.makedirs(dirpath, exist_ok=True)
    with open(os.path.join(dirpath, "pmc_counter_collection.csv"), "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for i, (name, kib) in enumerate(rows):
            # each dispatch split over two hardware instances, as the profiler reports it
            w.writerow([i, name, counter, kib / 2])
            w.writerow([i, name, counter, kib / 2])


def test_pmc_summary_scales_by_the_calibration_copy(tmp_path, monkeypatch):
    cal_mib = 4
    cal = cal_mib << 20
    form = "void cd::(anonymous namespace)::k_form_buffer<true, 1>(cd::FormArgs)"
    copy = "void neg_kernel(float*, float const*, long)"
    # FETCH_SIZE reads half of the copy's bytes (factor 2), WRITE_SIZE all of them
    fetch_rows = [(copy, cal / 2 / 1024), (form, 3000.0), (form, 3100.0)]
    write_rows = [(copy, cal / 1024), (form, 2400.0), (form, 2400.0)]
    fdir, wdir = str(tmp_path / "f"), str(tmp_path / "w")
    _write_pmc(fdir, "FETCH_SIZE", fetch_rows)
    _write_pmc(wdir, "WRITE_SIZE", write_rows)
    out = str(tmp_path / "gpt1p3b_hbm_traffic_pmc.txt")
    bench.summarize_pmc(fdir, wdir, out, "gpt1p3b", cal_mib)
    text = open(out).read()
    info = json.loads([ln for ln in text.splitlines() if ln.startswith("json ")][0][5:])
    assert info["factor"]["FETCH_SIZE"] == pytest.approx(2.0)
    assert info["factor"]["WRITE_SIZE"] == pytest.approx(1.0)
    k = info["kinds"]["form_buffer_local"]
    assert k["dispatches"] == 2
    assert k["fetch_bytes_per_launch"] == pytest.approx(2.0 * 3050.0 * 1024)
    assert k["write_bytes_per_launch"] == pytest.approx(2400.0 * 1024)
    assert k["traffic_bytes_per_launch"] == pytest.approx((2.0 * 3050.0 + 2400.0) * 1024)
    assert k["source_digest"] == bench.source_digest(bench.KIND_KERNEL["form_buffer_local"][1])
    # the bench line reads it back while the kernel's sources are unchanged ...
    monkeypatch.setattr(bench, "PMC_PROFILE", str(tmp_path / "{workload}_hbm_traffic_pmc.txt"))
    assert bench.counted_traffic("gpt1p3b", "form_buffer_local") == pytest.approx(k["traffic_bytes_per_launch"])
    assert bench.counted_traffic("gpt1p3b", "update_bf16") is None          # not in this run
    assert bench.counted_traffic("gpt160m", "form_buffer_local") is None    # no summary
    # ... and reports none once they differ from the counted build
    monkeypatch.setattr(bench, "source_digest", lambda files: "0000000000000000")
    assert bench.counted_traffic("gpt1p3b", "form_buffer_local") is None


def test_pmc_summary_needs_the_calibration(tmp_path):
    fdir, wdir = str(tmp_path / "f"), str(tmp_path / "w")
    _write_pmc(fdir, "FETCH_SIZE", [("void cd::k_gate(cd::GateArgs)", 1.0)])
    _write_pmc(wdir, "WRITE_SIZE", [("void cd::k_gate(cd::GateArgs)", 1.0)])
    with pytest.raises(SystemExit):
        bench.summarize_pmc(fdir, wdir, str(tmp_path / "o.txt"), "gpt1p3b", 0)
    with pytest.raises(SystemExit):      # no copy dispatch to calibrate against
        bench.summarize_pmc(fdir, wdir, str(tmp_path / "o.txt"), "gpt1p3b", 4)


def test_trace_summary(tmp_path):
    d = tmp_path / "trace"
    d.mkdir()
    with open(d / "bench_kernel_stats.csv", "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Name", "Calls", "TotalDurationNs", "AverageNs"])
        w.writerow(["void cd::(anonymous namespace)::k_form_buffer<true, 1>(cd::FormArgs)", 4, 3.6e6, 9.0e5])
        w.writerow(["void cd::(anonymous namespace)::k_gate(cd::GateArgs)", 2, 2.0e4, 1.0e4])
        w.writerow(["void at::native::elementwise_kernel<...>", 10, 5.0e6, 5.0e5])
    line = {"value": 2.4e11, "ms_per_step": 5.0,
            "config": {"workload": "w", "sync_steps": 1, "local_steps": 19},
            "roofline": {"kernel": "form_buffer_local", "avg_launch_ms": 0.9, "achieved": 6000.0,
                         "unit": "GB/s", "peak": 8000.0, "frac": 0.75},
            "branches": {"local": {"count": 19}}}
    bj = tmp_path / "b.json"
    bj.write_text("noise\n" + json.dumps(line) + "\n")
    out = tmp_path / "stats.txt"
    bench.summarize_trace(str(d), str(bj), str(out))
    text = out.read_text()
    rows = [ln for ln in text.splitlines() if ln.startswith("cd::")]
    assert rows[0].startswith("cd::k_form_buffer<true, 1>")          # largest total first
    assert "900.0" in rows[0] and "3.600" in rows[0]
    assert len(rows) == 2                                                 # torch kernels left out
    assert "5.0 ms in total" in text
    assert "form_buffer_local: avg launch 900.0 us" in text


def test_counted_bytes_per_step_by_branch(tmp_path, monkeypatch):
    """The counter summary cuts the dispatch sequence into steps at each
    step's first buffer-pass launch and adds every library kernel of a step
    (torch kernels left out); a step with a sync-branch kernel is a sync
    step.  The bench line reads the per-branch medians back while no kernel
    source has changed."""
    cal_mib = 4
    cal = cal_mib << 20
    copy = "void neg_kernel(float*, float const*, long)"
    form0 = "void cd::(anonymous namespace)::k_form_buffer<true, 0>(cd::FormArgs)"
    form1 = "void cd::(anonymous namespace)::k_form_buffer<true, 1>(cd::FormArgs)"
    gate = "void cd::(anonymous namespace)::k_gate(cd::GateArgs)"
    gemm = "void cd::(anonymous namespace)::k_gemm_bf<2, 128, 256, true, false, false>(cd::GemmArgs)"
    upd = "void cd::(anonymous namespace)::k_update_pl<1, 64>(cd::UpdatePlArgs)"
    torch_k = "void at::native::elementwise_kernel<128, 4>(int)"
    # step 1 sync: form0 x2, gate, gemm, update; step 2 local: form0, gate, torch noise;
    # step 3 local (fused): form1 x2, gate
    seq = [(copy, cal / 2 / 1024), (form0, 100.0), (form0, 100.0), (gate, 1.0), (gemm, 50.0), (upd, 300.0),
           (form0, 100.0), (gate, 1.0), (torch_k, 999.0), (form1, 200.0), (form1, 200.0), (gate, 1.0)]
    wseq = [(copy, cal / 1024)] + [(n, v / 2) for n, v in seq[1:]]
    fdir, wdir = str(tmp_path / "f"), str(tmp_path / "w")
    _write_pmc(fdir, "FETCH_SIZE", seq)
    _write_pmc(wdir, "WRITE_SIZE", wseq)
    out = str(tmp_path / "gpt1p3b_hbm_traffic_pmc.txt")
    bench.summarize_pmc(fdir, wdir, out, "gpt1p3b", cal_mib)
    info = json.loads([ln for ln in open(out).read().splitlines() if ln.startswith("json ")][0][5:])
    st = info["steps"]
    k = 1024.0
    assert st["sync"]["steps"] == 1 and st["local"]["steps"] == 2
    assert st["sync"]["fetch_bytes"] == pytest.approx(2.0 * 551.0 * k)
    assert st["sync"]["write_bytes"] == pytest.approx(551.0 / 2 * k)
    # local steps: 101 and 401 KiB fetched (x2); the median of two is the larger
    assert st["local"]["fetch_bytes"] == pytest.approx(2.0 * 401.0 * k)
    monkeypatch.setattr(bench, "PMC_PROFILE", str(tmp_path / "{workload}_hbm_traffic_pmc.txt"))
    got = bench.counted_step_bytes("gpt1p3b")
    assert got["sync"] == pytest.approx(2.0 * 551.0 * k + 551.0 / 2 * k)
    assert bench.counted_step_bytes("gpt160m") == {}
    monkeypatch.setattr(bench, "source_digest", lambda files: "0000000000000000")
    assert bench.counted_step_bytes("gpt1p3b") == {}


def test_kernel_digests_cover_their_includes():
    """A kind's counted traffic is trusted only while the digest of its
    source files matches: the list must hold every header its kernel file
    includes, directly or through other headers."""
    import re
    for kind, (_, files) in bench.KIND_KERNEL.items():
        closure, todo = set(), [files[0]]
        while todo:
            f = todo.pop()
            if f in closure:
                continue
            closure.add(f)
            text = open(os.path.join(bench.CSRC, f)).read()
            todo += re.findall(r'#include "([^"]+)"', text)
        assert closure <= set(files), (kind, sorted(closure - set(files)))
