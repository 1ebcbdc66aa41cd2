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
