"""bench.py's lookup of committed HBM-traffic summaries: a record counts only
for the kernel sources it was taken with and for its own batch size."""

import bench


def _write(dirpath, name, value, sha):
    p = dirpath / "profiles"
    p.mkdir(exist_ok=True)
    (p / name).write_text(f"# x\n\n- traffic_bytes_per_launch: {value}\n"
                          f"- kernel_source_sha256: `{sha}`\n")


def test_record_matches_sources_and_batch(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "ffn_source_hash", lambda wdt: "h-" + wdt)
    _write(tmp_path, "verify_moe_c5_b64_traffic.md", 123, "h-q4g32")
    assert bench.recorded_traffic("c5", "q4g32", 64, 64) == 123
    assert bench.recorded_traffic("c5", "q4g32", 16, 64) is None
    # changed kernel sources: the record no longer applies
    monkeypatch.setattr(bench, "ffn_source_hash", lambda wdt: "other")
    assert bench.recorded_traffic("c5", "q4g32", 64, 64) is None


def test_unsuffixed_record_is_for_the_default_batch_only(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "ffn_source_hash", lambda wdt: "h")
    _write(tmp_path, "verify_moe_c2_traffic.md", 77, "h")
    assert bench.recorded_traffic("c2", "bf16", 16, 16) == 77
    assert bench.recorded_traffic("c2", "bf16", 8, 16) is None
    assert bench.recorded_traffic("c3", "bf16", 32, 32) is None


def test_malformed_record_is_ignored(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "ffn_source_hash", lambda wdt: "h")
    _write(tmp_path, "verify_moe_c2_traffic.md", "n/a", "h")
    assert bench.recorded_traffic("c2", "bf16", 16, 16) is None
