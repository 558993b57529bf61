"""Host-side logic of bench.py: the one-GPU contract, the algorithmic byte counts behind the
roofline line, and the guard that drops stale HBM counters. No GPU is used."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_default_grid():
    # U Gauss-Legendre nodes and V azimuths integrate the product of two band-limited fields
    # (degree <= 2 lmax) times a harmonic of degree lmax exactly: 2U - 1 >= 3 lmax, V > 3 lmax
    for lmax in range(0, 25):
        U, V = bench.grid_dims(lmax)
        assert 2 * U - 1 >= 3 * lmax and V == 3 * lmax + 1
    assert bench.grid_dims(6) == (10, 19)


def test_headline_gather_bytes():
    # 10^4 receivers, 525,308 edges, lmax 6 (grid 10 x 19), R = 128, values-only receiver:
    # per edge one plane of sender values (128 x 190 floats), 7 radial coefficients per rank,
    # the unit vector and the sender index; per receiver the row pointer and Ta, Tb (2 x 128 x 49)
    per_edge = 4 * (128 * 190 + 128 * 7 + 3 + 1)
    per_recv = 4 * (1 + 2 * 128 * 49)
    want = 525308 * per_edge + 10000 * per_recv
    assert want == 53_494_871_040
    assert bench.receiver_bytes(6, 128, 10000, 525308, planes=1) == want
    # the paper's data flow reads three planes per sender
    assert (bench.receiver_bytes(6, 128, 10000, 525308)
            - bench.receiver_bytes(6, 128, 10000, 525308, planes=1)) == 525308 * 4 * 2 * 128 * 190
    # compulsory HBM bytes: every sender's plane once instead of once per edge
    comp = bench.compulsory_receiver_bytes(6, 128, 10000, 525308, planes=1)
    assert comp == (4 * 10000 * 128 * 190 + 525308 * 4 * (128 * 7 + 4) + 4 * 10001
                    + 4 * 10000 * 2 * 128 * 49)


def test_live_blocks():
    # Gaunt: equal slots -> even sector (block 0), mixed -> odd (1); curl the other way (3, 2)
    assert bench.live_blocks(False, False) == [0, 3]
    assert bench.live_blocks(False, True) == [0, 1, 2, 3]
    assert bench.live_blocks(True, True) == [0, 1, 2, 3]


def test_stale_traffic_counters_are_dropped(tmp_path, monkeypatch):
    rec = {"kernel_sha": bench.kernel_sha(), "bytes_per_launch": 123.0}
    (tmp_path / "traffic_w.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    assert bench.load_traffic("w") == 123.0
    rec["kernel_sha"] = "0" * 16
    (tmp_path / "traffic_w.json").write_text(json.dumps(rec))
    assert bench.load_traffic("w") is None
    assert bench.load_traffic("absent") is None


def test_kernel_sha_covers_the_device_sources(tmp_path, monkeypatch):
    src = tmp_path / "csrc"
    src.mkdir()
    (src / "a.hip").write_text("x")
    (src / "b.cpp").write_text("host only")
    monkeypatch.setattr(bench, "CSRC", str(src))
    h0 = bench.kernel_sha()
    (src / "b.cpp").write_text("host only, changed")
    assert bench.kernel_sha() == h0
    (src / "a.hip").write_text("y")
    assert bench.kernel_sha() != h0


@pytest.mark.parametrize("kind", ["both", "gaunt", "curl"])
def test_onsite_flops_scale(kind):
    # per (node, rank): the count doubles with the nodes and with the ranks
    a = bench.onsite_grid_flops(12, 128, 4096, kind)
    assert bench.onsite_grid_flops(12, 128, 8192, kind) == 2 * a
    assert bench.onsite_grid_flops(12, 256, 4096, kind) == 2 * a
