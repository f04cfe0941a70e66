"""CPU tests of bench.py's host-side helpers: the traffic figure read from a committed counter summary,
and the oracle timing (cpu_baseline) on whole heads and on the seeded row subset of long problems."""

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


def test_cpu_baseline_whole_heads_and_row_subset():
    import workloads as W

    small = W.small("cpu baseline small", Hq=4, Hkv=2, Sq=300, Sk=300, causal=True, seed=11)
    res = bench.cpu_baseline(small, *W.make_inputs(small), budget_s=0.0)
    # budget 0: exactly one key/value group (2 query heads) is timed, on every row
    assert res["rows_timed"] == 2 * 300 and "every row" in res["sample"]
    assert res["value"] > 0 and res["kind"] == "oracle" and res["cores"] >= 1
    assert res["extrapolated_s"] >= res["measured_s"] * 2 - 1e-3  # scaled by 4 heads / 2 timed
    long = W.small("cpu baseline long", Hq=1, Hkv=1, Sq=12000, Sk=12000, causal=True, seed=12)
    res = bench.cpu_baseline(long, *W.make_inputs(long), budget_s=0.0)
    rows = W.sample_rows(long, n=64)[0]
    assert res["rows_timed"] == len(rows) and "seeded subsets" in res["sample"]
    assert abs(res["extrapolated_s"] - res["measured_s"] * 12000 / len(rows)) <= 0.1 + 1e-3 * res["extrapolated_s"]


def test_code_hash_ignores_comments_and_layout_but_not_code():
    code = 'int f(int x) {\n  return x + 1;  // one more\n}\n/* block\n comment */ const char* s = "a // b /* c */";\n'
    same = '// header comment\nint f(int x)\n{\n    return x + 1;\n}\nconst char* s = "a // b /* c */";   /* x */\n'
    assert bench._code_tokens(code) == bench._code_tokens(same)
    # a change inside a string literal or to the code itself is seen
    assert bench._code_tokens(code) != bench._code_tokens(code.replace("a // b", "a // c"))
    assert bench._code_tokens(code) != bench._code_tokens(code.replace("x + 1", "x + 2"))
    assert len(bench.kernel_source_hash()) == 16
