"""bench.py's host-side logic on the CPU: the one-GPU contract, the lookup of
counter-measured traffic (valid only while the kernel's sources are the
ones measured), the per-kernel table, the block-aligned splitting and the
CPU-baseline leg's record on a tiny sample."""
import hashlib
import importlib.util
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def _digest(sources):
    h = hashlib.sha256()
    for fn in sources:
        with open(os.path.join(ROOT, "paper_2407_01614_amd", "csrc", fn), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def test_measured_traffic_only_for_current_sources(bench, tmp_path):
    sources = ["adam.hip", "zpp_adam.h", "zpp_device.h"]
    path = str(tmp_path / "traffic.json")
    entry = {"bytes_per_launch": 6101178697.4, "source_digest": _digest(sources)}
    with open(path, "w") as f:
        json.dump({"workload": "llama-2-13b", "kernels": {"adam": entry}}, f)
    assert bench.measured_traffic(path, "llama-2-13b", "adam", sources) == 6101178697
    # another workload, another kernel, or sources changed since the counters were taken
    assert bench.measured_traffic(path, "llama-2-7b", "adam", sources) is None
    assert bench.measured_traffic(path, "llama-2-13b", "gather", sources) is None
    assert bench.measured_traffic(path, "llama-2-13b", "adam", sources[:2]) is None
    assert bench.measured_traffic(str(tmp_path / "absent.json"), "llama-2-13b", "adam",
                                  sources) is None


def test_kernel_table(bench):
    kb = {"adam": 6.0e9, "gather": 1.0e9}
    times = {"adam": [1.0, 0.9, 1.1, 19.0, 1.0], "gather": [0.2, 0.2]}  # ms per launch
    t = bench.kernel_table(kb, times)
    assert t["adam"]["mean_us"] == 4600.0 and t["adam"]["median_us"] == 1000.0
    assert t["adam"]["min_us"] == 900.0
    # GB/s at the median: the one delayed launch does not move it
    assert t["adam"]["GB/s"] == 6000.0 and t["adam"]["frac_of_peak"] == 0.75
    assert t["gather"]["GB/s"] == 5000.0 and t["gather"]["bytes"] == 1.0e9


@pytest.mark.parametrize("n,parts,align", [(1000, 3, 256), (256, 8, 256), (1 << 20, 16, 256),
                                           (257, 2, 256), (5, 4, 1)])
def test_chunks_cover_in_aligned_ranges(bench, n, parts, align):
    r = bench._chunks(n, parts, align)
    assert r[0][0] == 0 and r[-1][1] == n
    for (a, b), (c, _) in zip(r, r[1:]):
        assert b == c and b % align == 0
    assert all(a < b for a, b in r)


def test_cpu_baseline_record(bench):
    from paper_2407_01614_amd.workloads import WORKLOADS
    wl = WORKLOADS["tiny"]
    for threads in (1, 2):
        rec = bench.cpu_baseline(wl, 0.05, threads=threads, steps=2)
        assert rec["kind"] == "oracle" and rec["unit"] == "GB/s" and rec["cores"] == threads
        assert rec["value"] > 0
        assert set(rec["seconds"]) == {"adam", "refresh", "quant", "gather"}
        assert "2 step(s)" in rec["sample"]


def test_cpu_baseline_other_workloads(bench, monkeypatch):
    monkeypatch.setattr(bench, "CPU_OTHER_SAMPLES",
                        {"tiny": ((0.05, 1), (0.05, 2)), "llama-2-13b": ((0.001, 1), (0.001, 1))})
    monkeypatch.setattr(bench, "host_threads", lambda: 2)
    out = bench.cpu_baseline_others("llama-2-13b")
    assert set(out) == {"tiny"}
    legs = out["tiny"]
    assert legs["one_thread"]["cores"] == 1 and legs["all_cores"]["cores"] == 2
    assert "2 step(s)" in legs["all_cores"]["sample"]
    assert all(leg["value"] > 0 and leg["unit"] == "GB/s" for leg in legs.values())


def test_sustain_runs_whole_chunks_for_the_asked_time(bench, monkeypatch):
    class FakePipe:
        steps = 0

        def step(self):
            FakePipe.steps += 1

        def wait(self):
            pass

    import torch
    monkeypatch.setattr(torch.cuda, "synchronize", lambda: None)
    clock = iter(range(0, 1000))
    monkeypatch.setattr(bench.time, "perf_counter", lambda: float(next(clock)))
    pipe = FakePipe()
    rec = bench.sustain(pipe, 1000.0, 3.0, chunk=5)
    # the clock advances one second per read: start, then one read per chunk
    assert rec["steps"] == 15 and FakePipe.steps == 15 and rec["seconds"] == 3.0
    assert rec["GB/s"] == round(1000.0 * 15 / 3.0 / 1e9, 1)
    assert pipe.streams == 1 and pipe.fused is False and pipe.sync == "event"


def test_traffic_sources_cover_every_include(bench):
    """Each kernel's digest covers its .hip file and every header it
    includes, directly or through another header, so that a change to any
    of them invalidates the kernel's counter figures."""
    import re
    csrc = os.path.join(ROOT, "paper_2407_01614_amd", "csrc")

    def includes(name, seen):
        if name in seen:
            return seen
        seen.add(name)
        with open(os.path.join(csrc, name)) as f:
            for line in f:
                m = re.match(r'#include "([^"]+)"', line)
                if m:
                    includes(m.group(1), seen)
        return seen

    for kernel, sources in bench.TRAFFIC_SOURCES.items():
        need = includes(sources[0], set())
        assert need <= set(sources), (kernel, sorted(need - set(sources)))


def test_traffic_file_matches_current_sources(bench):
    """The committed counter figures are those of the sources as they are."""
    with open(os.path.join(ROOT, "profiles", "traffic.json")) as f:
        t = json.load(f)
    for kernel, v in t["kernels"].items():
        assert v["source_digest"] == bench.source_digest(bench.TRAFFIC_SOURCES[kernel]), kernel


def test_workloads_offered_fit_the_pipeline(bench):
    """--workload offers only configurations whose gather shards fit in the
    rank partition; the tiny one is refused with argparse's message."""
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "tiny"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "invalid choice" in r.stderr
