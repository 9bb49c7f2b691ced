"""Host-side logic of bench.py: the kernel-source hash that keys the
committed HBM-counter summaries, and the lookup that reports their traffic
only while the kernel code is the one they were taken on."""
import json
import os
import shutil

import bench


def _copy_sources(tmp_path):
    for rel in bench.KERNEL_SOURCES:
        dst = tmp_path / rel
        dst.parent.mkdir(parents=True, exist_ok=True)
        shutil.copy(os.path.join(bench.ROOT, rel), dst)


def test_hash_ignores_comments_and_white_space(tmp_path, monkeypatch):
    _copy_sources(tmp_path)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h0 = bench.kernel_hash()
    p = tmp_path / bench.KERNEL_SOURCES[-1]
    src = p.read_text()
    p.write_text("// a reworded comment\n/* and a block\n   comment */\n" + src.replace("\n", "\n\n", 5))
    assert bench.kernel_hash() == h0


def test_hash_follows_the_code(tmp_path, monkeypatch):
    _copy_sources(tmp_path)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h0 = bench.kernel_hash()
    p = tmp_path / bench.KERNEL_SOURCES[0]
    p.write_text(p.read_text() + "\nconstexpr int kOneMore = 1;\n")
    assert bench.kernel_hash() != h0


def test_traffic_only_for_the_current_code(tmp_path, monkeypatch):
    _copy_sources(tmp_path)
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    t = {"fetch_kib_per_dispatch": 100.0, "fetch_scale": 2.0, "write_kib_per_dispatch": 50.0,
         "write_scale": 1.0, "kernel_sha": bench.kernel_hash()}
    (tmp_path / "profiles" / "w_traffic.json").write_text(json.dumps(t))
    assert bench.traffic_from_profile("w") == 1024.0 * (100.0 * 2.0 + 50.0)
    assert bench.traffic_from_profile("missing") is None
    t["kernel_sha"] = "0" * 16
    (tmp_path / "profiles" / "w_traffic.json").write_text(json.dumps(t))
    assert bench.traffic_from_profile("w") is None


def test_committed_summaries_match_the_sources():
    """Every committed traffic summary was taken on the current kernel code."""
    d = os.path.join(bench.ROOT, "profiles")
    names = [f[:-len("_traffic.json")] for f in os.listdir(d) if f.endswith("_traffic.json")]
    assert names
    for n in names:
        assert bench.traffic_from_profile(n) is not None, n
