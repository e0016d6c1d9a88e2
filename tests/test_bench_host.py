"""Host-side logic of bench.py (no GPU): the one-GPU guard, the use of the
recorded HBM-traffic summary only for the kernel sources and workload it was
taken on, the algorithmic byte counts per launch, and the CPU description."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}), ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_exits_with_a_message(argv, env):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv], capture_output=True, text=True,
                       env={**os.environ, **env}, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_traffic_is_used_only_for_matching_sources_and_workload(tmp_path, monkeypatch):
    prof = tmp_path / "profiles"
    prof.mkdir()
    rec = {"source_digest": bench.source_digest(), "workload_key": "c5",
           "kernels": {"qwd_encode": {"bytes_per_launch": 123}}}
    (prof / "hbm_traffic.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "source_digest", lambda: rec["source_digest"])
    assert bench.traffic_for("qwd_encode") == 123
    assert bench.traffic_for("qwd_encode", "c4") is None            # another workload
    assert bench.traffic_for("grad_quant") is None                  # no record for that kernel
    monkeypatch.setattr(bench, "source_digest", lambda: "another")  # kernel sources changed since
    assert bench.traffic_for("qwd_encode") is None
    (prof / "hbm_traffic.json").write_text("not json")
    assert bench.traffic_for("qwd_encode") is None


def test_source_digest_covers_device_sources_only(tmp_path, monkeypatch):
    csrc = tmp_path / "paper_2410_15526_amd" / "csrc"
    csrc.mkdir(parents=True)
    (csrc / "kernels.hpp").write_text("a")
    (csrc / "abi.cpp").write_text("x")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    d0 = bench.source_digest()
    (csrc / "abi.cpp").write_text("y")              # host-side argument checks only
    assert bench.source_digest() == d0
    (csrc / "kernels.hpp").write_text("b")
    assert bench.source_digest() != d0


def test_source_digest_ignores_comments_and_layout(tmp_path, monkeypatch):
    csrc = tmp_path / "paper_2410_15526_amd" / "csrc"
    csrc.mkdir(parents=True)
    k = csrc / "kernels.hpp"
    k.write_text("// header\nint f(int x) { return x + 1; }\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    d0 = bench.source_digest()
    k.write_text("// another header\n/* a block\n   comment */\nint f(int x)\n{\n    return x + 1; // same\n}\n")
    assert bench.source_digest() == d0
    k.write_text("int f(int x) { return x + 2; }\n")     # the code changed
    assert bench.source_digest() != d0


def test_algorithmic_bytes_per_launch():
    """The per-element byte counts of the kernels (reads + writes, group 128,
    bf16 model weights), checked against the c5 shard's launches."""
    pytest.importorskip("torch")
    from paper_2410_15526_amd.pipeline import HotPath
    n, g, P, Q = 1_625_292_800, 128, 8, 4
    info = HotPath.kernel_info(type("S", (), dict(n=n, group=g, qwd_group=g, P=P, Q=Q, M=n // P, m=n // P // Q,
                                                   prev_dtype="bf16"))())
    assert info["qwd_encode"].alg_bytes == n * (4 + 2 + 0.5) + 8 * n // g == 10_665_984_000
    assert info["qwd_decode"].alg_bytes == 7_415_398_400
    assert info["grad_quant"].alg_bytes == n * 5 + 4 * n // g == 8_177_254_400
    assert info["reduce_intra"].alg_bytes == 1_784_012_800
    assert info["reduce_inter"].alg_bytes == 311_091_200


def test_host_cpu_names_model_and_cores():
    s = bench.host_cpu()
    assert "cores available" in s and len(s) > len("cores available")


def test_all_cores_baseline_slices_the_sample(monkeypatch):
    """The all-cores oracle leg: whole-step slices of the sample, each a
    multiple of every group, block and chunk size, one thread per core."""
    pytest.importorskip("numpy")
    import synth
    w = synth.WORKLOADS["c5"]
    monkeypatch.setattr(bench.os, "sched_getaffinity", lambda pid: set(range(3)))
    r = bench.cpu_baseline_all_cores(w, 1 << 16, 0)
    assert r["cores"] == 3 and r["kind"] == "oracle" and r["value"] > 0
    per = int(r["sample"].split(" slices of ")[1].split(",")[0])
    assert per % (w.P * w.Q * max(w.group, w.hadamard_block, w.qwd_group)) == 0 and 3 * per <= 1 << 16


def test_read_write_split_and_additive_bound():
    """Reads per launch are the inputs each kernel must load; the additive
    bound lies between the write-only and the read-only rate and equals
    either one for a pure stream."""
    pytest.importorskip("torch")
    from paper_2410_15526_amd.pipeline import HotPath
    n, g, P, Q = 1_625_292_800, 128, 8, 4
    info = HotPath.kernel_info(type("S", (), dict(n=n, group=g, qwd_group=g, P=P, Q=Q, M=n // P, m=n // P // Q,
                                                   prev_dtype="bf16"))())
    assert info["qwd_encode"].read_bytes == 6 * n
    assert info["qwd_decode"].read_bytes == n // 2 + 8 * n // g + 2 * n
    assert info["grad_quant"].read_bytes == 4 * n
    assert info["reduce_intra"].read_bytes == n + 4 * n // g
    assert info["reduce_inter"].read_bytes == n // P // 2 + 4 * n // P // g
    c = {"read_GBps": 7000.0, "write_GBps": 6000.0}
    assert bench.rw_additive_GBps(10, 0, c) == pytest.approx(7000.0)
    assert bench.rw_additive_GBps(0, 10, c) == pytest.approx(6000.0)
    assert 6000.0 < bench.rw_additive_GBps(1, 1, c) < 7000.0
    assert bench.rw_additive_GBps(1, 1, c) == pytest.approx(2 / (1 / 7000 + 1 / 6000))


def test_workload_overrides():
    """Shape overrides replace the named workload's fields (and drop its extra sweeps)."""
    import argparse
    a = argparse.Namespace(workload="c4", n=1 << 20, group=64, hblock=0, P=4, Q=2, qwd_group=256,
                           model_weights="f32")
    w = bench.workload_from_args(a)
    assert (w.n, w.group, w.hadamard_block, w.P, w.Q, w.qwd_group, w.prev_dtype) == (1 << 20, 64, 0, 4, 2, 256, "f32")
    assert w.extra_groups == () and w.extra_qwd_groups == () and w.wid == 4
    b = argparse.Namespace(workload="c4", n=None, group=None, hblock=None, P=None, Q=None, qwd_group=None,
                           model_weights=None)
    import synth
    assert bench.workload_from_args(b) is synth.WORKLOADS["c4"]
