"""Host-side logic of bench.py that needs no GPU: the hash that decides
whether the committed HBM byte counters still describe the device code, and
the refusal of more than one GPU, the event pass's sample count and the
per-kernel statistics."""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_device_code_hash_tracks_the_kernels_only(tmp_path):
    text = open(bench.KERNEL_SRC).read()
    marker = "// " + "-" * 61 + " host side"
    a = text.index("namespace {")
    b = text.index(marker)
    base = tmp_path / "base.hip"
    base.write_text(text)
    h0 = bench.device_code_sha256(str(base))
    host_edit = tmp_path / "host.hip"
    host_edit.write_text(text[:b] + marker + "\n// host-side note"
                         + text[b + len(marker):])
    assert bench.device_code_sha256(str(host_edit)) == h0
    head_edit = tmp_path / "head.hip"
    head_edit.write_text("// file header note\n" + text)
    assert bench.device_code_sha256(str(head_edit)) == h0
    # a comment edited or added among the kernels, or blank lines, do not
    # count; a line of code does
    k = text.index("__device__", a)
    comment_edit = tmp_path / "comment.hip"
    comment_edit.write_text(text[:k] + "// a note on the kernels\n\n"
                            + text[k:])
    assert bench.device_code_sha256(str(comment_edit)) == h0
    kernel_edit = tmp_path / "kernel.hip"
    kernel_edit.write_text(text[:k] + "constexpr int kProbe = 1;\n"
                           + text[k:])
    assert bench.device_code_sha256(str(kernel_edit)) != h0


def test_traffic_is_reported_only_for_the_profiled_code(tmp_path, monkeypatch):
    text = open(bench.TRAFFIC_FILE).read()
    data = json.loads(text[text.index("{", text.index("Machine-readable")):])
    sha = bench.device_code_sha256()
    for stored, expect in ((sha, True), ("0" * 64, False)):
        data["device_code_sha256"] = stored
        f = tmp_path / f"traffic_{expect}.txt"
        f.write_text("counters\nMachine-readable:\n" + json.dumps(data))
        monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
        got = bench.measured_traffic("pack")
        if expect:
            assert got == data["llama3-8b-decode"]["pack"]["traffic_bytes"]
        else:
            assert got is None
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "missing.txt"))
    assert bench.measured_traffic("pack") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"),
                        "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_event_pass_has_enough_samples():
    """The per-kernel figures rest on at least MIN_KERNEL_SAMPLES launches
    however few steps are timed, and on every timed step's worth when more
    are."""
    for steps in (1, 5, 19, 20, 37, 200):
        n = len(bench._event_steps(steps))
        assert n == max(steps, bench.MIN_KERNEL_SAMPLES)
    assert bench.MIN_KERNEL_SAMPLES >= 20


def test_kernel_stats_sum_bytes_over_sum_time():
    """GB/s is total bytes over total time (not a mean of per-launch
    rates); mean, median and the p10/p90 pair are in microseconds."""
    st = bench._kernel_stats([1e9, 3e9], [1.0, 2.0])  # bytes, ms
    assert abs(st["GBps"] - 4e9 / 3e-3 / 1e9) < 1e-6
    assert st["us_mean"] == 1500.0 and st["us_median"] == 1500.0
    assert st["samples"] == 2 and st["bytes_mean"] == 2e9
    lo, hi = st["us_p10_p90"]
    assert 1000.0 < lo < hi < 2000.0
