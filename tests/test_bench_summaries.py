"""bench.py's reading of the committed rocprofv3 summaries (no GPU): the
kernel-source hash comes from the summary's header comment, and a summary
taken from other kernel sources is reported stale (traffic null)."""
import os

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_summary_header_hash_is_read(tmp_path):
    p = tmp_path / "s.txt"
    p.write_text("# title\n# command: x --y z:w\n# kernel_source_sha256_16: 0123456789abcdef\n"
                 "# note: a comment with a colon\ntraffic_bytes_per_launch: 42\n")
    kv = bench.read_summary(str(p))
    assert kv["kernel_source_sha256_16"] == "0123456789abcdef"
    assert kv["traffic_bytes_per_launch"] == "42"
    assert "note" not in kv and "command" not in kv


def test_committed_summaries_name_a_source_hash():
    d = os.path.join(ROOT, "profiles")
    for f in sorted(os.listdir(d)):
        if f.endswith(".txt"):
            kv = bench.read_summary(os.path.join(d, f))
            h = kv.get("kernel_source_sha256_16", "")
            assert len(h) == 16 and int(h, 16) >= 0, f


def test_traffic_follows_the_source_hash(tmp_path, monkeypatch):
    prof = tmp_path / "profiles"
    prof.mkdir()
    body = "traffic_bytes_per_launch: 1000\n"
    (prof / "traffic_k_8b_B256_seed2.txt").write_text("# kernel_source_sha256_16: 0000000000000000\n" + body)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_sha", lambda: "ffffffffffffffff")
    (prof / "traffic_k_8b_B256_seed3.txt").write_text("# kernel_source_sha256_16: ffffffffffffffff\n" + body)
    t, src = bench.measured_traffic("k", 256, 3)
    assert t == 1000 and src.endswith("seed3.txt")
    t, src = bench.measured_traffic("k", 256, 2)
    assert t is None and "stale" in src
    assert bench.measured_traffic("k", 256, 9) == (None, None)
