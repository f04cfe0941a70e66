"""CPU tests of bench.py's host-side helpers: the traffic figure read from a committed counter summary."""

import os

import bench


def _write_summary(root, config, source_hash, hbm_bytes):
    os.makedirs(os.path.join(root, "profiles"), exist_ok=True)
    with open(os.path.join(root, "profiles", f"fa_fwd_config{config}_hbm_traffic.txt"), "w") as f:
        f.write("# HBM traffic summary\n")
        f.write(f"kernel_source_sha256_16: {source_hash}\n")
        f.write("fetch_bytes_per_launch: 100\n")
        f.write("write_bytes_per_launch: 23\n")
        f.write(f"hbm_bytes_per_launch: {hbm_bytes}\n")


def test_traffic_read_when_the_summary_matches_the_kernel_source(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "0123456789abcdef")
    _write_summary(str(tmp_path), 3, "0123456789abcdef", 123)
    assert bench.traffic_from_profile(3) == 123.0


def test_traffic_null_when_the_kernel_changed_or_no_summary(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "0123456789abcdef")
    _write_summary(str(tmp_path), 3, "fedcba9876543210", 123)
    assert bench.traffic_from_profile(3) is None
    assert bench.traffic_from_profile(4) is None


def test_committed_summary_has_the_fields_bench_reads():
    path = os.path.join(bench.ROOT, "profiles", "fa_fwd_config3_hbm_traffic.txt")
    text = open(path).read()
    for key in ("kernel_source_sha256_16:", "hbm_bytes_per_launch:"):
        assert key in text
    recorded = [ln.split(":", 1)[1].strip() for ln in text.splitlines() if ln.startswith("kernel_source_sha256_16:")]
    if recorded == [bench.kernel_source_hash()]:
        assert bench.traffic_from_profile(3) > 0
