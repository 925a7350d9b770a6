"""bench.py's use of the committed counter records (profiles/counters.json):
a record is used only while the hash of its kernel's source file matches,
and runs with learnable features have keys of their own."""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_counters_key_separates_feature_runs():
    assert bench.counters_key("pascal", "bwd_message") == "pascal/bwd_message"
    assert bench.counters_key("pascal", "bwd_message", 2) == "pascal+features/bwd_message"


def test_records_carry_the_fields_the_bench_reads():
    with open(bench.COUNTERS) as f:
        recs = json.load(f)
    assert recs
    for key, rec in recs.items():
        for field in ("source_sha256_16", "bytes_per_launch", "valu_insts_per_launch"):
            assert field in rec, (key, field)
        src = os.path.join(os.path.dirname(bench.ITER_SRC), rec.get("source", "iter.hip"))
        assert os.path.exists(src), (key, src)


def test_a_record_is_used_only_on_its_own_source(tmp_path, monkeypatch):
    csrc = os.path.dirname(bench.ITER_SRC)
    recs = {
        "w/cur": {"source": "backward.hip",
                  "source_sha256_16": bench.source_hash(os.path.join(csrc, "backward.hip")),
                  "bytes_per_launch": 1, "valu_insts_per_launch": 2},
        "w/old": {"source": "backward.hip", "source_sha256_16": "0" * 16,
                  "bytes_per_launch": 1, "valu_insts_per_launch": 2},
        "w/iter": {"source_sha256_16": bench.source_hash(),
                   "bytes_per_launch": 1, "valu_insts_per_launch": 2},
        "w/gone": {"source": "no_such_file.hip", "source_sha256_16": "0" * 16,
                   "bytes_per_launch": 1, "valu_insts_per_launch": 2},
    }
    path = tmp_path / "counters.json"
    path.write_text(json.dumps(recs))
    monkeypatch.setattr(bench, "COUNTERS", str(path))
    assert bench.load_counters("w", "cur")["valu_insts_per_launch"] == 2
    assert bench.load_counters("w", "old") is None
    assert bench.load_counters("w", "iter") is not None      # no source named: iter.hip
    assert bench.load_counters("w", "gone") is None
    assert bench.load_counters("w", "missing") is None
    assert bench.load_counters("w", "cur", D=2) is None       # features: another key
