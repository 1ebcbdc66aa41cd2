"""Benchmark: fused CIS loss forward+backward on one MI355X.

Workload (default): the MoE-rollout batch, T = 16384 packed tokens, V = 151936, bf16 logits,
c = 1 (lambda = e - 1), kappa = 5e-3 (see workloads/synth.py). Inputs are generated on the GPU
before the timed region; a step is one call of the fused loss (every row: log-softmax, CIS
weight, loss term, gradient) through the C ABI with preallocated outputs.

Prints one JSON line. `roofline` refers to the fused row kernel: algorithmic bytes per launch
(read the logits once, write the gradient once, plus the per-token inputs and outputs) divided by
the average call time measured with HIP events on the stream the kernels run on (the call also
contains the tiny loss-reduction kernel, so this slightly understates the row kernel's rate).
`cpu_baseline` times the float64 CPU oracle on a bounded sample of the same rows, on the host's
cores, and also states its rate as the GB/s of the same algorithmic bytes per token.

    python bench.py [--steps K] [--warmup W] [--c C] [--mode bwd|fwd] [--config N]
                    [--op NAME] [--decoupled] [--no-cpu-baseline] [--no-copy-ceiling]

--op / --decoupled time the operator family and the decoupled PPO-clip path (the _ex entry
points; the decoupled call includes its weight pre-pass) on the same workload.

--lmhead times the loss behind the LM head instead (cis_lmhead_loss_bwd / _fwd): hidden states
[T, H] and a head weight [V, H] in bf16 (workloads/lmhead.py; H = 2048 by default), the logits
formed chunk by chunk on the matrix cores and never materialised for the whole batch. Its
`roofline` is the matrix-core bound: the three products' FLOPs (2 T V H each; one for the
forward) per call over the call time, against the bf16 dense peak.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
METRIC = "tokens/sec and achieved HBM GB/s, CIS loss fwd+bwd, V=151936, 1 MI355X"
PER_TOKEN_SCALAR_BYTES = 30   # ids 8 + mask 1 + l_infer 4 + A 4 in; l_train 4 + w 4 + trunc 1 + term 4 out


def kernel_source_hash(extra=()) -> str:
    h = hashlib.sha256()
    for f in ("paper_2609_32444_amd/csrc/cis_row.h", "paper_2609_32444_amd/csrc/cis_kernels.hip",
              "paper_2609_32444_amd/csrc/cis_kernels_ext.hip",
              "paper_2609_32444_amd/csrc/cis_api.cpp", "paper_2609_32444_amd/csrc/cis_internal.h",
              "paper_2609_32444_amd/csrc/cis_seg.h", *extra):
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def algorithmic_bytes(T_valid: int, T_invalid: int, V: int, esize: int, bwd: bool,
                      decoupled: bool = False) -> int:
    """Bytes the method must move per call: each valid row's logits once (and its gradient
    once), each invalid row's zero gradient, and the per-token inputs and outputs (the
    decoupled path also reads l_old). Implementation scratch (workspace) is not counted."""
    per_valid = esize * V * (2 if bwd else 1) + PER_TOKEN_SCALAR_BYTES + (4 if decoupled else 0)
    per_invalid = (esize * V if bwd else 0) + 9
    return T_valid * per_valid + T_invalid * per_invalid


OPS = {"cis": 0, "none": 1, "exact": 2, "tis": 3, "icepop": 4, "kpop": 5, "two_sided": 6,
       "qfixed": 7, "seq_tis": 8, "seq_mis": 9}
OP_BOUNDS = {"exact": (1e-6, 1e6), "tis": (0.0, 2.0), "icepop": (0.5, 5.0), "kpop": (0.0, 2.0),
             "seq_tis": (0.0, 2.0), "seq_mis": (0.5, 2.0)}   # Table tab:baselines


def hbm_traffic(mode: str, workload: str):
    """HBM bytes per launch from committed rocprofv3 counter passes, if they were taken on the
    current kernel source (else None)."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic_cis_row_kernel.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
        e = rec[mode][workload]
        if e.get("source_hash") != kernel_source_hash():
            return None
        return int(e["bytes_per_launch"])
    except Exception:
        return None


def lmhead_traffic():
    """HBM bytes per LM-head call (all of its kernels) from the committed counter passes, if
    they were taken on the current source (else None)."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic_lmhead.json")
    try:
        rec = json.load(open(path))
        if rec.get("source_hash") != kernel_source_hash(LMHEAD_SOURCES):
            return None
        return int(rec["bytes_per_call"])
    except Exception:
        return None


LMHEAD_SOURCES = ("paper_2609_32444_amd/csrc/cis_gemm.hip", "paper_2609_32444_amd/csrc/cis_gemm.h")


PROBE_MAX_ROW_BYTES = 19 * 1024 * 16   # the row-pattern probes hold one row per workgroup


def bandwidth_ceilings(rows: int, row_bytes: int, torch) -> dict:
    """Measured ceilings on this device (libcis_probe.so), in GB/s: the row kernel's access
    pattern as copy (equal read and write), read only and write only of rows x row_bytes, and
    the fastest equal read/write and read-only streams found on this part (4 KiB short-lived
    workgroups). Rows longer than the row-pattern probes hold are probed as pieces of the
    same total size."""
    while row_bytes > PROBE_MAX_ROW_BYTES and row_bytes % 32 == 0:
        rows, row_bytes = rows * 2, row_bytes // 2
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2609_32444_amd", "libcis_probe.so"))
    lib.cis_probe_bandwidth.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                        ctypes.c_void_p, ctypes.c_void_p]
    n = rows * row_bytes
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty(n, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1026, dtype=torch.int32, device="cuda")  # 1024 words + queue counter
    stream = torch.cuda.current_stream().cuda_stream
    grid = torch.cuda.get_device_properties(0).multi_processor_count
    out = {}
    for mode, name, moved in ((0, "copy", 2 * n), (1, "read", n), (2, "write", n),
                              (3, "copy_small_blocks", 2 * n), (4, "read_small_blocks", n)):
        if row_bytes > PROBE_MAX_ROW_BYTES and mode < 3:
            continue
        def go():
            rc = lib.cis_probe_bandwidth(mode, src.data_ptr(), dst.data_ptr(), rows, row_bytes,
                                         grid, sink.data_ptr(), stream)
            assert rc == 0, rc
        go(); go()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(5):
            go()
        e1.record()
        torch.cuda.synchronize()
        out[name] = moved / (e0.elapsed_time(e1) / 5 * 1e-3) / 1e9
    del src, dst
    return out


MAX_WORKERS = 16   # the host CPU share of one GPU on the measurement boxes


def host_cpu():
    """(cores this process may run on, /proc/cpuinfo model name and family/model numbers)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    info = {}
    try:
        for line in open("/proc/cpuinfo"):
            k, _, v = line.partition(":")
            k = k.strip()
            if k in ("model name", "cpu family", "model", "stepping") and k not in info:
                info[k] = v.strip()
            if len(info) == 4:
                break
    except OSError:
        pass
    model = info.get("model name", "")
    if "cpu family" in info:
        model += f" (family {info['cpu family']}, model {info.get('model', '?')}, " \
                 f"stepping {info.get('stepping', '?')})"
    return n, model


def cpu_baseline(b, V: int, target_s: float = 15.0):
    """The oracle as it stands (float64, with the gradient) on a sample of rows, in a process
    pool over the host cores (at most MAX_WORKERS); sized to roughly target_s of CPU time."""
    import multiprocessing as mp

    import numpy as np

    from oracle import cis as O

    host_cores, model = host_cpu()
    cores = max(1, min(host_cores, MAX_WORKERS))
    # probe one row to size the sample
    rows_all = np.nonzero(b.mask.cpu().numpy())[0]
    rng = np.random.default_rng(0)
    probe = rows_all[:9]
    import torch
    zp = O.Bf16Matrix(b.logits[torch.as_tensor(probe, device=b.logits.device)].contiguous()
                      .view(torch.int16).cpu().numpy().view(np.uint16))
    args = (b.ids[probe].cpu().numpy(), b.logp_infer[probe].cpu().double().numpy(),
            b.adv[probe].cpu().double().numpy(), None, b.lam, b.kappa, b.scale)
    O.cis_loss(zp, *args, rows=np.arange(1))           # warm-up row
    t0 = time.perf_counter()
    O.cis_loss(zp, *args, rows=np.arange(1, len(probe)))
    per_row = (time.perf_counter() - t0) / (len(probe) - 1)
    n = int(min(len(rows_all), max(cores * 4, target_s / max(per_row, 1e-6))))
    n = max(cores, (n // cores) * cores)
    rows = np.sort(rng.choice(rows_all, size=n, replace=False))
    bits = b.logits[torch.as_tensor(rows, device=b.logits.device)].contiguous() \
        .view(torch.int16).cpu().numpy().view(np.uint16)
    ids = b.ids.cpu().numpy()[rows]
    linf = b.logp_infer.cpu().double().numpy()[rows]
    adv = b.adv.cpu().double().numpy()[rows]
    global _BASE
    _BASE = (bits, ids, linf, adv, float(np.float32(b.lam)), float(np.float32(b.kappa)),
             float(np.float32(b.scale)))
    blocks = np.array_split(np.arange(n), cores)
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with ctx.Pool(cores) as pool:
        pool.map(_baseline_worker, blocks)
    dt = time.perf_counter() - t0
    # the oracle's rate in the HBM terms of the roofline: the same algorithmic bytes per token
    per_tok = algorithmic_bytes(1, 0, V, b.logits.element_size(), True)
    return {"value": n / dt, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "equivalent_gbs": n / dt * per_tok / 1e9,
            "sample": (f"all {n} valid rows of the batch" if n == len(rows_all) else
                       f"{n} random valid rows of the same batch")
                      + f", float64 oracle with gradient, {cores} worker processes "
                        f"(the pool is held to {MAX_WORKERS}; this process may run on "
                        f"{host_cores} cores), {dt:.1f} s wall ({per_row * n:.0f} s CPU est.)",
            "host_cores": host_cores,
            "cpu_model": model}


_BASE = None


def _baseline_worker(idx):
    from oracle import cis as O
    bits, ids, linf, adv, lam, kappa, scale = _BASE
    O.cis_loss(O.Bf16Matrix(bits[idx]), ids[idx], linf[idx], adv[idx], None, lam, kappa, scale,
               with_grad=True)
    return len(idx)


def cpu_baseline_lmhead(b, prm_ref, target_s: float = 40.0):
    """oracle.lmhead as it stands (float64: logits, loss, dL/dh and dL/dW of the sampled rows) on
    a sample of rows, one process whose matrix products use the host's BLAS threads (the
    per-row estimate from 64 rows overstates the cost of larger batches, so the sample aims at
    about a third of target_s)."""
    import numpy as np

    from oracle import lmhead as L

    cores, model = host_cpu()
    W = b.weight.float().cpu().double().numpy()
    h = b.hidden.float().cpu().double().numpy()
    ids = b.ids.cpu().numpy()
    linf = b.logp_infer.cpu().double().numpy()
    adv = b.adv.cpu().double().numpy()
    mask = b.mask.cpu().numpy()

    def run(rows):
        L.lmhead_cis_loss(h[rows], W, ids[rows], linf[rows], adv[rows], mask[rows], prm_ref,
                          with_grad=True, chunk=1024)

    rng = np.random.default_rng(0)
    run(np.arange(4))                       # warm-up: BLAS threads, page-in
    t0 = time.perf_counter()
    run(np.arange(4, 68))
    per_row = (time.perf_counter() - t0) / 64
    n = int(max(64, min(b.T, 8192, target_s / max(per_row, 1e-6))))
    rows = np.sort(rng.choice(b.T, size=n, replace=False))
    t0 = time.perf_counter()
    run(rows)
    dt = time.perf_counter() - t0
    # the oracle's rate in the terms of the roofline: the three products' FLOPs per token
    flops_per_tok = 3 * 2.0 * b.V * b.H
    threads = blas_threads(cores)
    return {"value": n / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "equivalent_tflops": n / dt * flops_per_tok / 1e12,
            "sample": f"{n} random rows of the same batch through oracle.lmhead (float64 logits, "
                      f"loss, dL/dh and dL/dW of those rows), one process, BLAS on {threads} "
                      f"threads ({cores} cores available), {dt:.1f} s wall",
            "host_cores": cores,
            "cpu_model": model}


def blas_threads(cores: int) -> int:
    """Threads numpy's BLAS runs on: OMP_NUM_THREADS / OPENBLAS_NUM_THREADS when set (the
    measurement boxes set them to the CPU share of one GPU), else the available cores."""
    for k in ("OPENBLAS_NUM_THREADS", "OMP_NUM_THREADS"):
        v = os.environ.get(k, "")
        if v.isdigit() and int(v) > 0:
            return min(int(v), cores)
    return cores


def bench_lmhead(args, torch, cis):
    """The loss behind the LM head (see the module docstring)."""
    import numpy as np

    from oracle import ops as X
    from workloads import make_lmhead_batch

    T, V = 16384, 151936
    H, chunk = args.hidden, args.chunk
    ext = args.op is not None or args.decoupled
    op = args.op or "cis"
    b = make_lmhead_batch(T, V, H, device="cuda", seed=2, c=args.c,
                          old_sd=0.3 if args.decoupled else None)
    bwd = args.mode == "bwd"
    lo, hi = OP_BOUNDS.get(op, (0.0, math.inf))
    prm = cis.params(OPS[op], lam=b.lam, kappa=b.kappa, lo=lo, hi=hi, scale=b.scale)
    lold = b.logp_old if args.decoupled else None
    offs = b.offsets if op.startswith("seq_") else None
    n_seq = 0 if offs is None else offs.numel() - 1
    rec = bool(args.recompute)
    ws = torch.empty(cis.lmhead_workspace_bytes(T, V, H, chunk, n_seq, bwd, rec), dtype=torch.uint8,
                     device="cuda")
    dh = torch.empty(T, H, dtype=torch.float32, device="cuda") if bwd else None
    dw = torch.empty(V, H, dtype=torch.float32, device="cuda") if bwd else None
    want = ("logp_train", "w", "acted", "terms")
    if bwd:
        def step():
            return cis.lmhead_loss_bwd(b.hidden, b.weight, b.ids, b.logp_infer, b.adv, b.mask,
                                       params=prm, logp_old=lold, seq_offsets=offs, chunk=chunk,
                                       dhidden=dh, dweight=dw, want=want, workspace=ws,
                                       recompute=rec)
    else:
        def step():
            return cis.lmhead_loss_fwd(b.hidden, b.weight, b.ids, b.logp_infer, b.adv, b.mask,
                                       params=prm, logp_old=lold, seq_offsets=offs, chunk=chunk,
                                       want=want, workspace=ws)
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    t_all0 = torch.cuda.Event(enable_timing=True)
    t_all1 = torch.cuda.Event(enable_timing=True)
    t_all0.record()
    for i in range(args.steps):
        starts[i].record()
        step()
        ends[i].record()
    t_all1.record()
    torch.cuda.synchronize()
    ms_per_step = t_all0.elapsed_time(t_all1) / args.steps
    per_call = sorted(s.elapsed_time(e) for s, e in zip(starts, ends))
    avg_call_ms = sum(per_call) / len(per_call)
    stats = cis.read_stats(ws)
    n_valid = stats["n_valid"]
    flops = (3 if bwd else 1) * 2.0 * T * V * H   # algorithmic: the recompute's 4th product is not
    tflops = flops / (avg_call_ms * 1e-3) / 1e12
    line = {
        "metric": f"tokens/sec, CIS loss {'fwd+bwd' if bwd else 'fwd'} through the LM head "
                  f"(H={H} -> V={V}), 1 MI355X",
        "value": n_valid / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # the dominant arithmetic: bf16 matrix-core products (float32 accumulation)
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"moe-rollout LM head T={T} V={V} H={H} bf16 chunk={chunk} "
                               f"c={args.c:g} {'fused fwd+bwd' if bwd else 'forward only'}"
                               + (f" op={op}" if ext else "")
                               + (" decoupled PPO-clip (0.2, 0.28)" if args.decoupled else "")
                               + (" logits recomputed (never stored)" if bwd and rec else "")
                               + (" logits never stored" if not bwd else ""),
                   "T": T, "V": V, "H": H, "chunk": chunk, "valid_tokens": n_valid,
                   "recompute": rec if bwd else None,
                   "lambda": b.lam, "kappa": b.kappa, "seed": b.meta["seed"]},
        "roofline": {
            "bound": "mfma",
            "achieved": tflops,
            "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": tflops / MFMA_BF16_PEAK_TFLOPS,
            "traffic": lmhead_traffic() if bwd and chunk == 4096 and H == 2048 and not ext
            and not rec else None,
            "traffic_scope": "HBM bytes per call, every kernel of the call (rocprofv3 counters)",
            "algorithmic_flops_per_call": flops,
            "avg_call_ms": avg_call_ms,
            "median_call_ms": per_call[len(per_call) // 2],
            "min_call_ms": per_call[0],
            "scope": "whole call (every kernel of the chunked pipeline) against the matrix-core "
                     "peak of its three products",
            "kernel_source": kernel_source_hash(LMHEAD_SOURCES),
        },
    }
    if ext:
        line["config"]["op"] = op
        line["config"]["decoupled"] = bool(args.decoupled)
        line["diagnostics"] = {k: stats[k] for k in ("n_trunc", "max_abs_logk", "trunc_excess")}
    if not args.no_cpu_baseline and not ext:
        f32 = lambda x: float(np.float32(x))  # noqa: E731
        prm_ref = X.OpParams(op=X.OP_CIS, lam=f32(b.lam), kappa=f32(b.kappa), lo=0.0,
                             hi=math.inf, clip_low=f32(0.2), clip_high=f32(0.28),
                             scale=f32(b.scale))
        line["cpu_baseline"] = cpu_baseline_lmhead(b, prm_ref)
    print(json.dumps(line), flush=True)


def make_parser() -> argparse.ArgumentParser:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--c", type=float, default=1.0)
    ap.add_argument("--mode", choices=("bwd", "fwd"), default="bwd")
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--op", choices=sorted(OPS), default=None,
                    help="operator of the weight (cis_loss_*_ex); default: the base CIS path")
    ap.add_argument("--decoupled", action="store_true",
                    help="the decoupled PPO-clip objective with l_old at a theta_old snapshot")
    ap.add_argument("--lmhead", action="store_true",
                    help="the loss behind the LM head (hidden [T, H] x weight [V, H], bf16)")
    ap.add_argument("--hidden", type=int, default=2048, help="--lmhead: hidden size H")
    ap.add_argument("--chunk", type=int, default=4096, help="--lmhead: rows per chunk")
    ap.add_argument("--recompute", action="store_true",
                    help="--lmhead backward: never store the logits (the product is formed twice)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-copy-ceiling", action="store_true")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a device copy of MIB mebibytes (counter calibration) and exit")
    return ap


def check_args(ap: argparse.ArgumentParser, args) -> None:
    """Rejects option combinations that bench.py does not run (exit status 2, before any
    device work)."""
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the CIS loss is measured on one MI355X "
              "(multi-GPU sharding is a design note only)", file=sys.stderr)
        sys.exit(2)
    if args.op in ("seq_tis", "seq_mis") and not args.decoupled:
        ap.error("sequence operators need --decoupled")
    if args.lmhead and args.config != 2:
        ap.error("--lmhead runs the MoE-rollout shape (--config 2)")
    if args.config not in (0, 1, 2, 3, 4):
        ap.error("--config is one of 0..4")


def main():
    ap = make_parser()
    args = ap.parse_args()
    check_args(ap, args)

    import torch

    import paper_2609_32444_amd as cis
    from workloads import make_batch

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_probe:
        n = args.copy_probe << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty(n, dtype=torch.uint8, device="cuda")
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_read": n, "copy_probe_bytes_written": n}), flush=True)
        return
    if args.lmhead:
        bench_lmhead(args, torch, cis)
        return
    b = make_batch(args.config, device="cuda", c=args.c)
    bwd = args.mode == "bwd"
    ext = args.op is not None or args.decoupled
    op = args.op or "cis"
    if ext:
        from workloads import old_logprobs, response_offsets
        lo, hi = OP_BOUNDS.get(op, (0.0, math.inf))
        prm = cis.params(OPS[op], lam=b.lam, kappa=b.kappa, lo=lo, hi=hi, scale=b.scale)
        lold = old_logprobs(b, sd=0.3) if args.decoupled else None
        offs = response_offsets(b.T, 256, 1536) if op.startswith("seq_") else None
        call = cis.LossCall(b.logits, b.ids, b.logp_infer, b.adv, b.mask, bwd=bwd, params=prm,
                            logp_old=lold, seq_offsets=offs)
    else:
        call = cis.LossCall(b.logits, b.ids, b.logp_infer, b.adv, b.mask, lam=b.lam,
                            kappa=b.kappa, scale=b.scale, bwd=bwd)
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        call.run()
    torch.cuda.synchronize()

    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    t_all0 = torch.cuda.Event(enable_timing=True)
    t_all1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_all0.record()
    for i in range(args.steps):
        starts[i].record()
        call.run()
        ends[i].record()
    t_all1.record()
    torch.cuda.synchronize()
    total_ms = t_all0.elapsed_time(t_all1)
    per_call = sorted(s.elapsed_time(e) for s, e in zip(starts, ends))
    avg_call_ms = sum(per_call) / len(per_call)
    ms_per_step = total_ms / args.steps

    stats = cis.read_stats(call.workspace)
    n_valid = stats["n_valid"]
    T, V = b.T, b.V
    esize = b.logits.element_size()
    alg = algorithmic_bytes(n_valid, T - n_valid, V, esize, bwd, args.decoupled)
    achieved_gbs = alg / (avg_call_ms * 1e-3) / 1e9
    tokens_per_s = n_valid / (ms_per_step * 1e-3)

    workload = f"{b.meta['name']} T={T} V={V} {'bf16' if esize == 2 else 'fp32'} c={args.c:g} " \
               f"kappa={b.kappa:g} {'fused fwd+bwd' if bwd else 'forward only'}"
    if ext:
        workload += f" op={op}" + (" decoupled PPO-clip (0.2, 0.28)" if args.decoupled else "")
    if not ext:
        traffic = hbm_traffic(args.mode, f"cfg{args.config}")
    elif op == "cis" and args.decoupled:
        traffic = hbm_traffic(args.mode, f"cfg{args.config}_decoupled")
    else:
        traffic = None
    line = {
        "metric": METRIC if bwd else METRIC.replace("fwd+bwd", "fwd"),
        "value": tokens_per_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # the arithmetic: float32 throughout (logits widened on load, gradients rounded on store)
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": workload, "T": T, "V": V, "valid_tokens": n_valid,
                   "storage": "bf16" if esize == 2 else "f32",
                   "lambda": b.lam, "kappa": b.kappa, "seed": b.meta["seed"]},
        "roofline": {
            "bound": "hbm",
            "achieved": achieved_gbs,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved_gbs / HBM_PEAK_GBS,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": alg,
            "avg_call_ms": avg_call_ms,
            "median_call_ms": per_call[len(per_call) // 2],
            "min_call_ms": per_call[0],
            "kernel_source": kernel_source_hash(),
        },
    }
    if not args.no_copy_ceiling:
        ceil = bandwidth_ceilings(T, ((V * esize + 15) // 16) * 16, torch)
        line["roofline"]["measured_ceiling_gbs"] = ceil
        if bwd:
            best = max(ceil.get("copy", 0.0), ceil["copy_small_blocks"])
            line["roofline"]["frac_of_measured_copy"] = achieved_gbs / best
            if "copy" in ceil:
                line["roofline"]["frac_of_row_pattern_copy"] = achieved_gbs / ceil["copy"]
        else:
            best = max(ceil.get("read", 0.0), ceil["read_small_blocks"])
            line["roofline"]["frac_of_measured_read"] = achieved_gbs / best
    if ext:
        line["config"]["op"] = op
        line["config"]["decoupled"] = bool(args.decoupled)
        line["diagnostics"] = {k: stats[k] for k in ("n_trunc", "max_abs_logk", "trunc_excess")}
    if not args.no_cpu_baseline and not ext:
        line["cpu_baseline"] = cpu_baseline(b, V)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
