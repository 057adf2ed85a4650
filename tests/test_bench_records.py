"""CPU checks of bench.py's record lookups: the HBM-traffic and MFMA-busy figures come from
committed records only while the kernel sources hash as they did when the counters were taken."""
import json
import os

import pytest

import bench


@pytest.fixture
def fake_root(tmp_path, monkeypatch):
    csrc = tmp_path / "paper_2206_08720_amd" / "csrc"
    csrc.mkdir(parents=True)
    (csrc / "kernels_fcn.hip").write_text("// kernel source\n")
    (csrc / "shared.hpp").write_text("// shared header\n")
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    return tmp_path


def test_source_hash_covers_the_kernel_file_and_every_header(fake_root):
    h0 = bench.sources_sha16("kernels_fcn.hip")
    assert len(h0) == 16 and h0 == bench.sources_sha16("kernels_fcn.hip")
    hdr = fake_root / "paper_2206_08720_amd" / "csrc" / "shared.hpp"
    hdr.write_text("// shared header, changed\n")
    h1 = bench.sources_sha16("kernels_fcn.hip")
    assert h1 != h0
    (fake_root / "paper_2206_08720_amd" / "csrc" / "kernels_fcn.hip").write_text("// changed\n")
    assert bench.sources_sha16("kernels_fcn.hip") not in (h0, h1)


def test_traffic_record_is_used_only_for_its_kernel_at_its_sources(fake_root):
    assert bench.measured_traffic("w", "ntk_fcn") is None          # no record
    rec = {"kernel": "ntk_fcn", "kernel_source": "kernels_fcn.hip",
           "sources_sha256_16": bench.sources_sha16("kernels_fcn.hip"),
           "fetch_size_kib_per_launch": 100.0, "write_size_kib_per_launch": 10.0,
           "fetch_scale": 2.0, "write_scale": 1.0}
    (fake_root / "profiles" / "w_traffic.json").write_text(json.dumps(rec))
    assert bench.measured_traffic("w", "ntk_fcn") == (100.0 * 2.0 + 10.0) * 1024.0
    assert bench.measured_traffic("w", "dense_bwd") is None        # another kernel class
    (fake_root / "paper_2206_08720_amd" / "csrc" / "kernels_fcn.hip").write_text("// changed\n")
    assert bench.measured_traffic("w", "ntk_fcn") is None          # stale sources


def test_mfma_busy_record_is_used_only_at_its_sources(fake_root):
    cls = {"kernel_source": "kernels_fcn.hip", "sources_sha256_16": bench.sources_sha16("kernels_fcn.hip"),
           "mfma_busy": 0.93}
    (fake_root / "profiles" / "w_mfma_busy.json").write_text(json.dumps({"classes": {"ntk_fcn": cls}}))
    assert bench.measured_mfma_busy("w", "ntk_fcn") == 0.93
    assert bench.measured_mfma_busy("w", "gram") is None
    (fake_root / "paper_2206_08720_amd" / "csrc" / "shared.hpp").write_text("// changed\n")
    assert bench.measured_mfma_busy("w", "ntk_fcn") is None


def test_committed_records_name_their_workload_and_sources():
    """Every committed record carries a source hash and a class name bench.py knows."""
    prof = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "profiles")
    for f in sorted(os.listdir(prof)):
        if f.endswith("_traffic.json"):
            rec = json.load(open(os.path.join(prof, f)))
            assert rec["kernel"] in bench.STAGE_OF and len(rec["sources_sha256_16"]) == 16
            assert rec["fetch_scale"] > 0 and rec["write_scale"] > 0
        elif f.endswith("_mfma_busy.json"):
            rec = json.load(open(os.path.join(prof, f)))
            for name, cls in rec["classes"].items():
                assert name in bench.STAGE_OF and 0.0 <= cls["mfma_busy"] <= 1.0
                assert len(cls["sources_sha256_16"]) == 16
