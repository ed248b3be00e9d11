"""bench.py on the CPU: the one-GPU guard, the counter lookup that fills
roofline.traffic, and the oracle baseline on a short sample (no GPU)."""

import hashlib
import json
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2608_25523_amd import workloads as W  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]


def test_traffic_only_from_counters_of_the_current_kernel_source(tmp_path, monkeypatch):
    src = tmp_path / "paper_2608_25523_amd" / "csrc"
    src.mkdir(parents=True)
    (src / "pfx_kernels.hip").write_bytes(b"// kernel source\n")
    (tmp_path / "profiles").mkdir()
    digest = hashlib.sha256(b"// kernel source\n").hexdigest()
    rec = {"kernel_source_sha256": digest, "decode": {"bytes_per_step": 123}, "extend": {"bytes_per_step": 456}}
    (tmp_path / "profiles" / "hbm_traffic.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.traffic_from_profile("decode") == 123
    assert bench.traffic_from_profile("extend") == 456
    assert bench.traffic_from_profile("other") is None
    (src / "pfx_kernels.hip").write_bytes(b"// kernel source, changed\n")
    assert bench.traffic_from_profile("decode") is None        # counters of another source
    (tmp_path / "profiles" / "hbm_traffic.json").unlink()
    assert bench.traffic_from_profile("decode") is None


def test_cpu_baseline_counts_unique_bytes():
    # One pass over the requests credits each its own suffix and an even
    # share of its agent's prefix: the shares add up to the step's U.
    b = W.config_batch(2)
    tau = b.num_kv_heads * b.head_dim * 4
    n_a = {int(a): int(np.sum(b.agent == a)) for a in set(b.agent.tolist())}
    shares = sum((int(b.suffix_len[r]) + int(b.prefix_len[int(b.agent[r])]) / n_a[int(b.agent[r])]) * tau
                 for r in range(len(b.agent)))
    assert abs(shares - b.unique_kv_bytes()) < 1e-6 * b.unique_kv_bytes()

    hv = W.host_values_fast(b, 2002)
    out = bench.cpu_baseline({"batch": b, "hv": hv}, W, seconds=0.5)
    assert out["kind"] == "oracle" and out["unit"] == "GB/s"
    assert out["value"] > 0 and out["cores"] >= 1
    assert "decode requests" in out["sample"]
