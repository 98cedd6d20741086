"""bench.py's counter bookkeeping on the host: FETCH_SIZE / WRITE_SIZE runs are
turned into HBM bytes per launch by scaling each counter with its reading for
the calibration copy, the entry is tied to the sha256 of the kernel's sources,
and a lookup returns nothing once those sources differ."""
import csv
import importlib.util
import json
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

HEADER = ["Correlation_Id", "Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]
# kernel names as rocprofv3 writes them (non-template kernels carry no "void")
COPY = ("(anonymous namespace)::copy_kernel(HIP_vector_type<unsigned int, 4u>*, "
        "HIP_vector_type<unsigned int, 4u> const*, unsigned long)")
SPLIT = ("void (anonymous namespace)::split_pv<4, false, (anonymous namespace)::KvBf16, true>"
         "((anonymous namespace)::SplitArgs)")
OTHER = "(anonymous namespace)::merge_splits((anonymous namespace)::MergeArgs)"


@pytest.fixture()
def bench(tmp_path, monkeypatch):
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    monkeypatch.setattr(mod, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    return mod


def write_csv(path, counter, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(HEADER)
        for i, (name, value) in enumerate(rows):
            w.writerow([i + 1, i + 1, name, counter, value])


def test_summarize_scales_each_counter_by_the_calibration_copy(bench, tmp_path):
    gib_kib = (1 << 30) / 1024.0
    # FETCH_SIZE reads half of what the copy moved, WRITE_SIZE all of it
    fetch = [(COPY, gib_kib / 2), (SPLIT, 500.0), (SPLIT, 520.0), (OTHER, 9e9)]
    write = [(COPY, gib_kib), (SPLIT, 3.0), (SPLIT, 5.0), (OTHER, 9e9)]
    write_csv(tmp_path / "f.csv", "FETCH_SIZE", fetch)
    write_csv(tmp_path / "w.csv", "WRITE_SIZE", write)
    bench.summarize_pmc(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "some_step")
    data = json.load(open(bench.TRAFFIC_FILE))
    e = data["some_step"]
    assert e["fetch_kib_raw"] == 510.0 and e["write_kib_raw"] == 4.0
    assert e["fetch_scale"] == 2.0 and e["write_scale"] == 1.0
    assert e["bytes_per_launch"] == (510 * 2 + 4) * 1024
    assert e["kernel_source_sha256"] == bench.kernel_source_sha("attention")
    # the lookup returns the bytes for the current sources only
    assert bench.load_traffic("some_step", bench.kernel_source_sha()) == (510 * 2 + 4) * 1024
    assert bench.load_traffic("some_step", "0" * 64) is None
    assert bench.load_traffic("another_step", bench.kernel_source_sha()) is None


def test_summarize_keeps_other_entries_and_replaces_its_own(bench, tmp_path):
    with open(bench.TRAFFIC_FILE, "w") as f:
        json.dump({"kept": {"kernel_source_sha256": "x", "bytes_per_launch": 1},
                   "some_step": {"kernel_source_sha256": "y", "bytes_per_launch": 2}}, f)
    gib_kib = (1 << 30) / 1024.0
    write_csv(tmp_path / "f.csv", "FETCH_SIZE", [(COPY, gib_kib), (SPLIT, 100.0)])
    write_csv(tmp_path / "w.csv", "WRITE_SIZE", [(COPY, gib_kib), (SPLIT, 1.0)])
    bench.summarize_pmc(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "some_step")
    data = json.load(open(bench.TRAFFIC_FILE))
    assert data["kept"] == {"kernel_source_sha256": "x", "bytes_per_launch": 1}
    assert data["some_step"]["bytes_per_launch"] == 101 * 1024


def test_summarize_refuses_ambiguous_kernel_names(bench, tmp_path):
    gib_kib = (1 << 30) / 1024.0
    other_split = SPLIT.replace("<4,", "<8,")
    write_csv(tmp_path / "f.csv", "FETCH_SIZE", [(COPY, gib_kib), (SPLIT, 1.0), (other_split, 2.0)])
    write_csv(tmp_path / "w.csv", "WRITE_SIZE", [(COPY, gib_kib), (SPLIT, 1.0)])
    with pytest.raises(SystemExit):
        bench.summarize_pmc(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "some_step")


def test_the_committed_traffic_file_matches_the_current_decode_sources(bench):
    """Every decode entry of profiles/traffic.json was taken on the kernel
    sources in the tree (else the bench reports its traffic as null)."""
    data = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    sha = bench.kernel_source_sha("attention")
    decode = {k: v for k, v in data.items() if not k.startswith("pack:")}
    assert decode
    stale = [k for k, v in decode.items() if v["kernel_source_sha256"] != sha]
    assert not stale, stale
