"""Host-side pieces of bench.py: the contract refusals and the oracle legs
(cpu_baseline) that sit beside the GPU figures. No GPU needed."""
import json
import subprocess
import sys
import os

import numpy as np
import torch

import bench
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0 and "one GPU" in (r.stdout + r.stderr)


def test_decode_point_oracle_leg():
    wl = workloads.decode_sweep("llada", 1, 0)
    r = bench.cpu_baseline(wl, 0.2, single_thread=False)
    assert r["kind"] == "oracle" and r["unit"] == "TFLOP/s" and r["value"] > 0 and r["cores"] >= 1
    assert "1 of 1 block decodes" in r["sample"] and "median of 3" in r["sample"]
    assert r["single_thread"] is None
    json.dumps(r)


def test_oracle_leg_single_thread_runs():
    wl = workloads.tiny_mixed(0)
    r = bench.cpu_baseline(wl, 0.3)
    names = [x["workload"] for x in r["single_thread"]]
    assert names == ["tiny_mixed", "llada_decode"]
    assert all(x["cores"] == 1 and x["value"] > 0 for x in r["single_thread"])
    assert r["cpu"] and r["cores"] == len(os.sched_getaffinity(0))
    json.dumps(r)


def test_kv_export_oracle_leg():
    # a small pool on the host stands in for the device pool: the leg copies
    # the sampled requests' pages and times the pure-Python export over them
    kv_len = np.array([40, 17, 33], np.int32)
    counts = (kv_len.astype(np.int64) + 15) // 16
    indptr = np.zeros(len(counts) + 1, np.int32)
    indptr[1:] = np.cumsum(counts)
    pool = int(indptr[-1]) * 2
    ids = np.random.default_rng(0).permutation(pool)[:indptr[-1]].astype(np.int32)
    k = torch.randn((pool, 2, 16, 64)).to(torch.bfloat16)
    v = torch.randn((pool, 2, 16, 64)).to(torch.bfloat16)
    r = bench.kv_cpu_baseline(k, v, kv_len, indptr, ids, 2, 64, 5.0)
    assert r["kind"] == "oracle" and r["unit"] == "GB/s" and r["value"] > 0
    assert "90 positions (3 of 3 requests)" in r["sample"]


def test_traffic_summaries_are_named_by_workload():
    """bench.py looks a workload's counter summary up by its --workload name:
    each profiles/traffic_<name>.json names that workload, which exists."""
    import glob
    import json
    import os

    import workloads
    files = glob.glob(os.path.join(os.path.dirname(bench.__file__), "profiles", "traffic_*.json"))
    assert files
    for f in files:
        stem = os.path.basename(f)[len("traffic_"):-len(".json")]
        with open(f) as fh:
            rec = json.load(fh)
        assert rec["workload"] == stem and callable(getattr(workloads, stem, None)), f
        assert rec["kernels"] and all("hbm_bytes_per_launch" in k for k in rec["kernels"].values())

