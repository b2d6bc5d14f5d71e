"""Host-side logic of bench.py: the one-GPU contract and the rule that a
committed HBM-counter summary is reported only for the kernel source it was
taken on (the scan file plus every header it includes)."""
import os
import shutil
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_before_any_device_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def _copy_sources(tmp_path):
    dst = tmp_path / "csrc"
    shutil.copytree(bench.CSRC, dst)
    return dst


def test_kernel_hash_follows_the_included_headers(tmp_path, monkeypatch):
    csrc = _copy_sources(tmp_path)
    monkeypatch.setattr(bench, "CSRC", str(csrc))
    h_tile, h_mq = bench.kernel_hash("dresd_kernels.hip"), bench.kernel_hash("dresd_scan_mq.hip")
    assert h_tile == bench.kernel_hash("dresd_kernels.hip") and h_tile != h_mq
    # a header both scans include changes both hashes
    with open(csrc / "dresd_device.h", "a") as f:
        f.write("\n// edit\n")
    assert bench.kernel_hash("dresd_kernels.hip") != h_tile
    assert bench.kernel_hash("dresd_scan_mq.hip") != h_mq
    h_tile2, h_mq2 = bench.kernel_hash("dresd_kernels.hip"), bench.kernel_hash("dresd_scan_mq.hip")
    # a source neither scan includes changes neither
    with open(csrc / "dresd_transform.hip", "a") as f:
        f.write("\n// edit\n")
    assert bench.kernel_hash("dresd_kernels.hip") == h_tile2
    assert bench.kernel_hash("dresd_scan_mq.hip") == h_mq2


def test_traffic_is_read_only_for_the_current_source(tmp_path, monkeypatch):
    csrc = _copy_sources(tmp_path)
    monkeypatch.setattr(bench, "CSRC", str(csrc))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    (tmp_path / "profiles").mkdir()
    path = tmp_path / "profiles" / "traffic_scan_w_B3.md"
    assert bench.read_traffic("w", 3, "single_tile") is None  # no summary
    h = bench.kernel_hash("dresd_kernels.hip")
    path.write_text("kernel_source_sha256_16: %s\nhbm_bytes_per_launch: 1.25e+09\n" % h)
    assert bench.read_traffic("w", 3, "single_tile") == 1.25e9
    assert bench.read_traffic("w", 3, "shared_key") is None  # another kernel's source
    # grouped launches run kernels of the same source file
    assert bench.read_traffic("w", 3, "single_tile_grouped") == 1.25e9
    with open(csrc / "dresd_kernels.hip", "a") as f:
        f.write("\n// edit\n")
    assert bench.read_traffic("w", 3, "single_tile") is None  # source changed since


def test_every_scan_kind_names_a_kernel_of_its_source():
    """Each kind the plan query reports maps to the source file whose hash
    gates its traffic summary and to a kernel defined in that file."""
    from paper_2502_15572_amd import SCAN_KINDS
    assert set(SCAN_KINDS.values()) == set(bench.SCAN_UNIT) == set(bench.SCAN_KERNEL_NAME)
    for kind in SCAN_KINDS.values():
        src = open(os.path.join(bench.CSRC, bench.SCAN_UNIT[kind])).read()
        assert " %s(ScanParams p)" % bench.SCAN_KERNEL_NAME[kind] in src, kind


def test_cpu_baseline_leg_parity_verdict():
    """The bench's parity verdict (query 0 against the oracle) passes the
    oracle's own answer and fails a wrong row."""
    import numpy as np
    import torch
    import oracle
    from datagen import WORKLOADS, generate, to_numpy_bits
    w = WORKLOADS["zipf33m_d128_f16"].scaled(5000)
    g = generate(w, "cpu")
    kb, dt = to_numpy_bits(g["keys"])
    q = g["queries"][:3]
    o = oracle.topk(kb, dt, q.numpy(), w.k, g["cont"].numpy())
    good = (torch.from_numpy(o[0]), torch.from_numpy(o[1]), torch.from_numpy(o[2]))
    base, par = bench.cpu_baseline_leg(g["keys"], g["cont"], q, w.k, good, time_it=False)
    assert base is None and par["verdict"] == "pass" and par["exact_order"]
    bad_idx = good[0].clone()
    outside = next(i for i in range(w.N) if i not in set(bad_idx[0].tolist()))
    bad_idx[0, 0] = outside
    _, par = bench.cpu_baseline_leg(g["keys"], g["cont"], q, w.k, (bad_idx,) + good[1:],
                                    time_it=False)
    assert par["verdict"] == "FAIL"
