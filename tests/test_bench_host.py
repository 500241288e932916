"""Host logic of bench.py that needs no GPU: the measured HBM traffic of the
roofline kernel is reported from its committed counter summary only for the
workload and kernel class it was measured on, and only while the sources it
was measured on are unchanged."""
import importlib.util
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_traffic_summary_value(bench, monkeypatch):
    # the machine-read value is the table's scaled FETCH_SIZE + WRITE_SIZE per
    # dispatch (KiB); with the current sources it is that value or, once they
    # have changed, None
    import re
    text = open(os.path.join(ROOT, bench.TRAFFIC_SUMMARY)).read()
    scaled = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        cal, scale, raw, out = re.search(r"^\| %s \| ([\d,.]+) KiB \| ([\d.]+) \| ([\d,.]+) KiB \| ([\d,]+) KiB \|" % c,
                                         text, re.M).groups()
        f = lambda s: float(s.replace(",", ""))
        assert abs(f(raw) * f(scale) - f(out)) <= 1.0, c
        scaled[c] = f(raw) * f(scale)
    want = int(re.search(r"^\s*traffic_bytes_per_launch:\s*(\d+)", text, re.M).group(1))
    assert abs(want - (scaled["FETCH_SIZE"] + scaled["WRITE_SIZE"]) * 1024) <= 1024
    assert bench.measured_traffic("1.5b", "attn") in (want, None)
    digest = re.search(r"^\s*sources_sha256:\s*(\S+)", text, re.M).group(1)
    monkeypatch.setattr(bench, "sources_sha256", lambda paths=None: digest)
    assert bench.measured_traffic("1.5b", "attn") == want


def test_traffic_only_for_its_workload_and_kernel(bench):
    assert bench.measured_traffic("7b", "attn") is None
    assert bench.measured_traffic("1.5b", "gemm_gu") is None


def test_traffic_dropped_when_sources_change(bench, monkeypatch):
    monkeypatch.setattr(bench, "sources_sha256", lambda paths=None: "0" * 64)
    assert bench.measured_traffic("1.5b", "attn") is None


def test_traffic_absent_summary(bench, monkeypatch):
    monkeypatch.setattr(bench, "TRAFFIC_SUMMARY", "profiles/no_such_summary.md")
    assert bench.measured_traffic("1.5b", "attn") is None


def test_more_than_one_gpu_is_refused():
    # the refusal comes before torch touches a device, so it runs anywhere
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_traffic_summary_ships_with_the_tree(bench):
    # the bench reads this summary at run time, so no pattern that keeps files
    # off the GPU machines may match it (tar-style: a pattern without a slash
    # matches the file name at any depth; './x' only from the top)
    import fnmatch
    ignore = os.path.join(ROOT, ".gpurunignore")
    if not os.path.exists(ignore):
        return
    rel = bench.TRAFFIC_SUMMARY
    for pat in (l.strip() for l in open(ignore)):
        if not pat or pat.startswith("#"):
            continue
        if pat.startswith("./"):
            p = pat[2:].rstrip("/")
            assert not (rel == p or rel.startswith(p + "/") or fnmatch.fnmatch(rel, p)), pat
        else:
            assert not fnmatch.fnmatch(os.path.basename(rel), pat) and not fnmatch.fnmatch(rel, pat), pat
