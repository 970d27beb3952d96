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


def test_code_hash_ignores_comments_but_not_code():
    a = b"int f(int x) {  // twice x\n  return 2 * x; /* doubled */\n}\n"
    b = b"int f(int x) {\n  /* a note\n     over two lines */ return 2 * x;\n}\n"
    c = b"int f(int x) {\n  return 3 * x;\n}\n"
    assert bench._code_only(a) == bench._code_only(b)
    assert bench._code_only(a) != bench._code_only(c)


def test_oracle_timing_repeats_until_the_time_or_the_cap(monkeypatch):
    calls = []
    monkeypatch.setattr(bench, "ORACLE_MIN_S", 0.05)
    monkeypatch.setattr(bench, "ORACLE_MAX_REPS", 7)
    reps, dt = bench.time_oracle(lambda: calls.append(1))
    assert reps == len(calls) == 7 and dt >= 0.0
    monkeypatch.setattr(bench, "ORACLE_MAX_REPS", 1000)
    import time
    reps, dt = bench.time_oracle(lambda: time.sleep(0.03))
    assert 2 <= reps <= 3 and dt >= 0.05


def test_int4_hash_covers_the_down_part_count(tmp_path, monkeypatch):
    # The K-part count of the int4 down projection sets how many partial sums
    # are written and read back, so it belongs to the int4 traffic record;
    # the bf16 kernels do not use it.
    import shutil
    src = tmp_path / "paper_2608_15018_amd" / "csrc"
    shutil.copytree(bench.os.path.join(bench.ROOT, "paper_2608_15018_amd", "csrc"), src)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    before = {w: bench.ffn_source_hash(w) for w in ("q4g32", "bf16")}
    kh = src / "kernels.h"
    text = kh.read_text()
    assert "0.02 * down / part" in text
    kh.write_text(text.replace("0.02 * down / part", "0.05 * down / part"))
    assert bench.ffn_source_hash("q4g32") != before["q4g32"]
    assert bench.ffn_source_hash("bf16") == before["bf16"]


def test_committed_traffic_records_match_the_kernel_sources():
    """Each committed HBM-traffic summary was taken with the kernel sources as
    they are now: bench.py reports its traffic only then, so a kernel change
    must come with new counter runs."""
    import glob
    import os
    import re
    recs = sorted(glob.glob(os.path.join(bench.ROOT, "profiles", "*_traffic.md")))
    assert recs, "no traffic records under profiles/"
    wdt_of = {"c2": "bf16", "c3": "bf16", "c4": "bf16", "c5": "q4g32"}
    stale = []
    for path in recs:
        name = os.path.basename(path)
        m = re.search(r"kernel_source_sha256: `([0-9a-f]{64})`", open(path).read())
        assert m, f"{name}: no kernel_source_sha256 line"
        if name.startswith("expand_"):
            want = bench.expand_source_hash()
        else:
            wl = re.match(r"verify_moe_(c\d)", name).group(1)
            want = bench.ffn_source_hash(wdt_of[wl])
        if m.group(1) != want:
            stale.append(name)
    assert not stale, f"traffic records taken with other kernel sources: {stale}"
