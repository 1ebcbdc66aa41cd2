"""bench.py's checks that need no GPU: the one-GPU refusal and the source hash that ties the
committed traffic records to the kernels they were measured on."""

import glob
import json
import os
import re
import shlex
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(args, **env):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=120,
                          env=dict(os.environ, **env))


def test_refuses_more_than_one_gpu():
    r = _run(["--gpus", "2"])
    assert r.returncode == 2 and "exactly one GPU" in r.stderr
    assert r.stdout == ""                   # no JSON line for a configuration it does not run


def test_refuses_a_multi_rank_launch():
    r = _run([], WORLD_SIZE="2")
    assert r.returncode == 2 and "exactly one GPU" in r.stderr


def test_kernel_source_hash():
    h = bench.kernel_source_hash()
    assert len(h) == 16 and int(h, 16) >= 0
    assert bench.kernel_source_hash() == h                            # stable
    assert bench.kernel_source_hash(bench.LMHEAD_SOURCES) != h        # covers the extra sources


def test_traffic_records_name_their_source_and_summary():
    # each record carries the hash of the sources it was measured on (bench.py reports the
    # traffic only while that hash matches) and points at a committed summary
    for name in ("hbm_traffic_cis_row_kernel.json", "hbm_traffic_lmhead.json"):
        rec = json.load(open(os.path.join(ROOT, "profiles", name)))
        recs = list(rec["bwd"].values()) if "bwd" in rec else [rec]
        for r in recs:
            assert len(r["source_hash"]) == 16
            assert os.path.isfile(os.path.join(ROOT, r["summary"]))


def test_profile_commands_run_committed_files():
    """Every command in a profile summary runs bench.py (a committed file) with options that
    bench.py accepts, directly after rocprofv3's `--`."""
    ap = bench.make_parser()
    found = 0
    for md in glob.glob(os.path.join(ROOT, "profiles", "*.md")):
        text = open(md).read()
        for block in re.findall(r"```\n(.*?)```", text, flags=re.S):
            for line in block.strip().splitlines():
                words = shlex.split(line)
                if words[0] == "rocprofv3":
                    words = words[words.index("--") + 1:]
                assert words[:2] == ["python3", "bench.py"], (md, line)
                ap.parse_args(words[2:])
                found += 1
    assert found >= 10


def test_rejects_option_combinations_before_device_work():
    # sequence operators run on the decoupled path only; the LM head runs one shape
    r = _run(["--op", "seq_tis"])
    assert r.returncode == 2 and "need --decoupled" in r.stderr and r.stdout == ""
    r = _run(["--lmhead", "--config", "1"])
    assert r.returncode == 2 and "MoE-rollout" in r.stderr and r.stdout == ""
    r = _run(["--config", "7"])
    assert r.returncode == 2 and r.stdout == ""


def test_cpu_baseline_on_a_tiny_host_batch():
    """The oracle timing leg on a small batch held in host memory: it runs, reports a rate,
    the worker count it used and the host's core count."""
    from workloads import make_batch
    b = make_batch(1, device="cpu", rows=64)
    rec = bench.cpu_baseline(b, b.V, target_s=0.2)
    assert rec["kind"] == "oracle" and rec["value"] > 0 and rec["equivalent_gbs"] > 0
    assert 1 <= rec["cores"] <= min(rec["host_cores"], bench.MAX_WORKERS)
    assert f"{rec['cores']} worker processes" in rec["sample"]


def test_cpu_baseline_lmhead_on_a_tiny_host_batch():
    import math

    from oracle import ops as X
    from workloads import make_lmhead_batch
    b = make_lmhead_batch(96, 200, 24, device="cpu", seed=2, c=1.0)
    prm = X.OpParams(op=X.OP_CIS, lam=b.lam, kappa=b.kappa, lo=0.0, hi=math.inf,
                     clip_low=0.2, clip_high=0.28, scale=b.scale)
    rec = bench.cpu_baseline_lmhead(b, prm, target_s=0.3)
    assert rec["kind"] == "oracle" and rec["value"] > 0 and rec["equivalent_tflops"] > 0
    assert 1 <= rec["cores"] <= rec["host_cores"]
