"""Host logic of bench.py (no GPU): the one-GPU guard, crossover interpolation, per-step statistics and the
rocprofv3 counter summary."""
import math
import os
import subprocess
import sys

import pytest

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, REPO)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(REPO, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_crossover_log_log_interpolation():
    # t_sparse / t_dense = (x / 8)^-1: sparse slower below x = 8, faster above, equal at x = 8 exactly
    pts = [(x, 1.0 / (x / 8.0), 1.0) for x in (1, 4, 16, 64)]
    assert bench._crossover(pts) == pytest.approx(8.0, rel=1e-12)
    # sparse always faster: no crossover
    assert bench._crossover([(x, 0.5, 1.0) for x in (1, 4, 16)]) is None


def test_spmm_algorithmic_counts():
    byt, flops = bench.spmm_algorithmic(4096, 1024, 8 * 10 ** 6)
    assert byt == 8 * 4096 * 1024 + 8 * 8 * 10 ** 6 + 8 * 4097 + 4 * 4096
    assert flops == 2.0 * 1024 * 8 * 10 ** 6


class _FakeEvent:
    """Stand-in for torch.cuda.Event on a clock that advances by a scripted duration per call."""

    clock = [0.0]

    def __init__(self, enable_timing=True):
        self.t = None

    def record(self):
        self.t = self.clock[0]

    def elapsed_time(self, other):
        return other.t - self.t


class _FakeTorch:
    class cuda:
        Event = _FakeEvent

        @staticmethod
        def synchronize():
            pass


@pytest.mark.parametrize("durations", [[3.0, 1.0, 2.0, 10.0, 4.0], [5.0, 1.0, 2.0, 8.0]])
def test_time_steps_mean_median_min(durations):
    _FakeEvent.clock = [0.0]
    it = iter(durations)

    def step():
        _FakeEvent.clock[0] += next(it)

    mean, median, lo = bench.time_steps(_FakeTorch, step, len(durations))
    s = sorted(durations)
    m = len(s) // 2
    want_median = s[m] if len(s) % 2 else 0.5 * (s[m - 1] + s[m])
    assert mean == pytest.approx(sum(durations) / len(durations))
    assert median == pytest.approx(want_median)
    assert lo == min(durations)


def _write_pmc(path, counter, kernel, values):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "p_counter_collection.csv"), "w") as f:
        f.write("Kernel_Name,Counter_Name,Counter_Value\n")
        for v in values:
            f.write(f'"{kernel}",{counter},{v}\n')
        f.write(f'"other_kernel",{counter},999999\n')


def test_summarize_pmc_scales_by_the_copy_probe(tmp_path):
    copy_bytes = 1 << 20
    k = "void sdnn::(anonymous namespace)::spmm_slots_kernel<false>(long, long)"
    cp = "__amd_rocclr_copyBuffer"
    _write_pmc(tmp_path / "f", "FETCH_SIZE", k, [100.0, 300.0])
    _write_pmc(tmp_path / "w", "WRITE_SIZE", k, [50.0])
    _write_pmc(tmp_path / "cf", "FETCH_SIZE", cp, [512.0])  # half of the 1024 KiB copied
    _write_pmc(tmp_path / "cw", "WRITE_SIZE", cp, [1024.0])
    out = tmp_path / "summary.txt"
    bench.summarize_pmc("spmm_slots_kernel", "test", [str(tmp_path / d) for d in ("f", "w", "cf", "cw")],
                        copy_bytes, ["cmd one", "cmd two"], str(out), ["spmm.hip", "common.h"])
    rec = dict(line.split(": ", 1) for line in out.read_text().splitlines() if ": " in line and " " not in
               line.split(": ", 1)[0])
    assert float(rec["fetch_scale"]) == pytest.approx(2.0)
    assert float(rec["write_scale"]) == pytest.approx(1.0)
    # (avg fetch 200 KiB x 2 + write 50 KiB x 1) x 1024 bytes
    assert int(rec["hbm_bytes_per_launch"]) == (200 * 2 + 50) * 1024
    assert rec["source_hash"] == bench._src_hash("spmm.hip", "common.h")
    assert "    cmd one" in out.read_text()


def test_summarize_counters_longest_dispatch(tmp_path):
    """--longest-dispatch keeps each kernel's longest dispatch of a run and drops the others."""
    d = tmp_path / "run"
    d.mkdir()
    with open(d / "x_counter_collection.csv", "w") as f:
        f.write("Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value,Start_Timestamp,End_Timestamp\n")
        f.write('1,"k(int)",SQ_WAVES,10,0,100\n')
        f.write('2,"k(int)",SQ_WAVES,99,0,5000\n')
        f.write('3,"k(int)",SQ_WAVES,20,0,200\n')
    out = tmp_path / "s.md"
    bench.summarize_counters([str(d)], "t", ["cmd"], str(out), longest=True)
    assert "| k | SQ_WAVES | 1 | 99 |" in out.read_text()
    bench.summarize_counters([str(d)], "t", ["cmd"], str(out))
    assert "| k | SQ_WAVES | 3 | 43 |" in out.read_text()


def test_source_hash_ignores_comments_only():
    """Counters stay current across comment edits and go stale on a change of code."""
    a = "int x = 1; // one\n/* a block\n   comment */ int y;\n"
    b = "int x = 1;   // another comment\nint y;"
    assert bench._code_only(a) == bench._code_only(b) == "int x = 1; int y;"
    assert bench._code_only(a) != bench._code_only("int x = 2; int y;")


def test_kernel_sources_name_the_file_that_defines_the_kernel():
    """A counter summary is current only while the file holding its kernel is unchanged."""
    csrc = os.path.join(os.path.dirname(bench.__file__), "paper_1708_02937_amd", "csrc")
    for kernel in ("spmm_blocked_kernel", "spmm_slots_kernel", "spmm_fanin_kernel", "spmm_narrow_kernel",
                   "gemm_dense_layer_kernel", "spgemm_pipe_kernel", "spgemm_small_kernel"):
        src = bench.kernel_sources(kernel)
        text = open(os.path.join(csrc, src[0]), encoding="utf-8").read()
        assert f"void {kernel}(" in text or f"void {kernel}<" in text or f" {kernel}(" in text, (kernel, src)


def test_kernel_split_and_roofline_from_profile_records():
    """The dominant kernel's roofline and HBM fields from profiling-log records: algorithmic bytes per launch
    (averaged over the launches' layers) divided by the average launch time."""
    from workloads import Layer, Problem
    import numpy as np

    n, batch = 1000, 256
    layers = [Layer(np.zeros(n + 1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.float32),
                    np.zeros(n, np.float32)) for _ in range(2)]
    layers[0].row_ptr[-1] = 3000  # only nnz is read
    layers[1].row_ptr[-1] = 5000
    p = Problem("t", n, 2, batch, math.inf, layers)
    recs = [(-1, "densify", 0.5), (0, "spmm_fanin_kernel", 2.0), (1, "spmm_fanin_kernel", 4.0), (-1, "pack", 1.0)]
    split = bench.kernel_split(recs)
    assert split["spmm_fanin_kernel"]["launches"] == 2 and split["spmm_fanin_kernel"]["avg_ms"] == 3.0
    roof = bench.kernel_roofline("spmm_fanin_kernel", split["spmm_fanin_kernel"], p)
    want_bytes = 8 * n * batch + 8 * 4000 + 8 * (n + 1) + 4 * n
    assert roof["bound"] == "hbm" and roof["algorithmic_bytes_per_launch"] == want_bytes
    assert roof["achieved"] == pytest.approx(round(want_bytes / 3e-3 / 1e9, 1))
    hbm = bench.hbm_fields(roof, 2 * want_bytes)
    assert hbm["effective"] == pytest.approx(want_bytes / 3e-3 / 1e9, abs=0.051)
    assert hbm["counter"] == pytest.approx(2 * want_bytes / 3e-3 / 1e9, abs=0.051)
    assert bench.hbm_fields(roof, None)["counter"] is None
