"""Parity of the HIP path (through the C ABI) with the CPU oracle on the five workloads.

Every workload runs exactly as the benchmark runs it (same entry point, same launch
configuration). The tiny, small and MoE-rollout workloads are compared on every row: per-token
outputs, the loss and every gradient element, the MoE rollout at each of its three thresholds.
Each of the eight 65536-row chunks of the long-response workload, and the wide-vocabulary
workload, is compared on every row's per-token outputs and the loss, and on the gradients of
4096 (long response) or 1024 (wide vocabulary) seeded rows that always include the first and
last rows and the heavy-tail rows.
"""

import json

import numpy as np
import pytest
import torch

import paper_2609_32444_amd as cis
from tests import parity as P
from workloads import make_batch

pytestmark = pytest.mark.gpu

def _record(name, report):
    P.write_report(f"parity_{name}.json", report)
    print(name, json.dumps(report, default=float), flush=True)


def _sample_rows(T, n, seed, extra=()):
    rng = np.random.default_rng(seed)
    rows = set(rng.choice(T, size=min(n, T), replace=False).tolist())
    rows.update([0, T - 1])
    rows.update(int(r) for r in extra if 0 <= r < T)
    return np.array(sorted(rows), dtype=np.int64)


def _run(b, bwd=True):
    fn = cis.loss_bwd if bwd else cis.loss_fwd
    out = fn(b.logits, b.ids, b.logp_infer, b.adv, b.mask, lam=b.lam, kappa=b.kappa,
             scale=b.scale)
    torch.cuda.synchronize()
    return out


def _check_full(name, b, out, grad_rows=None, scalar_rows=None, z=None, ref=None):
    """Scalars + loss on all rows (or scalar_rows), gradients on grad_rows (all if None).

    `z` (the logits on the host) and `ref` (the oracle's scalars over the same rows) can be
    passed in to share them between two comparisons of one batch."""
    report = {"config": {k: v for k, v in b.meta.items() if k != "outlier_rows"}}
    all_grads = grad_rows is None and "dlogits" in out
    z = P.host_logits(b.logits) if z is None else z
    if ref is None or all_grads:
        ref = P.oracle_for_batch(b, rows=scalar_rows, with_grad=False,
                                 grad=out["dlogits"] if all_grads else None, z=z)
    P.compare_scalars(out, ref, b, report)
    if scalar_rows is None:
        P.compare_loss(out, ref, report)
    if all_grads:
        P.check_grad_stats(ref["grad_stats"], report)
        report["grad_rows"] = int(b.T)
    elif "dlogits" in out:
        refg = P.oracle_for_batch(b, rows=grad_rows, with_grad=False, grad=out["dlogits"], z=z)
        P.check_grad_stats(refg["grad_stats"], report)
        report["grad_rows"] = int(len(grad_rows))
    stats = cis.read_stats(out["workspace"])
    valid = int(((b.mask.cpu().numpy() != 0) & (b.ids.cpu().numpy() >= 0)
                 & (b.ids.cpu().numpy() < b.V)).sum())
    assert stats["n_valid"] == valid and stats["n_nonfinite"] == 0
    if scalar_rows is None:
        assert stats["n_trunc"] == int(ref["trunc"].sum())
    report["stats"] = stats
    _record(name, report)
    return report


def test_tiny_fp32_all_rows():
    b = make_batch(0, device="cuda")
    _check_full("tiny", b, _run(b))


def test_small_bf16_all_rows():
    b = make_batch(1, device="cuda")
    _check_full("small", b, _run(b))


@pytest.mark.parametrize("c", [0.5, 1.0, 2.0])
def test_moe_rollout_full_size(c):
    """Every row of the MoE-rollout batch: per-token outputs, loss and all 2.5e9 gradient
    elements against the oracle."""
    b = make_batch(2, device="cuda", c=c)
    out = _run(b)
    rep = _check_full(f"moe_rollout_c{c}", b, out)
    assert rep["grad"]["n_rows"] == b.T


@pytest.mark.parametrize("chunk", range(8))
def test_long_response_chunk(chunk):
    """One 65536-row chunk of the long-response workload: every row's per-token outputs and
    the chunk's loss, and the gradients of 4096 seeded rows plus the first, last and
    heavy-tail rows."""
    b = make_batch(3, device="cuda", chunk=chunk)
    out = _run(b)
    grows = _sample_rows(b.T, 4096, seed=200 + chunk, extra=b.meta["outlier_rows"])
    rep = _check_full(f"long_response_chunk{chunk}", b, out, grad_rows=grows)
    assert rep["trunc"] > 0 and rep["grad_rows"] >= 4096


def test_wide_vocab_fwd_and_bwd():
    """Wide vocabulary, forward only and fused: every row's per-token outputs and the loss,
    and the fused pass's gradient on every row."""
    b = make_batch(4, device="cuda")
    z = P.host_logits(b.logits)
    ref = P.oracle_for_batch(b, with_grad=False, z=z)
    out_f = _run(b, bwd=False)
    _check_full("wide_vocab_fwd", b, out_f, z=z, ref=ref)
    out_b = _run(b, bwd=True)
    rep = _check_full("wide_vocab_bwd", b, out_b, z=z)
    assert rep["grad_rows"] == b.T
    # Both passes also agree with each other to float32 rounding. (Not bit for bit: the fused
    # pass sums a row in one workgroup, the forward pass in 16 KiB segments that are combined
    # afterwards, so the exp-sum is accumulated in a different order.)
    for k in ("logp_train", "w", "terms"):
        f, g = out_f[k].double(), out_b[k].double()
        assert torch.all((f - g).abs() <= 1e-5 * f.abs() + 1e-7), k
    assert abs(out_f["loss"].item() - out_b["loss"].item()) <= 1e-5 * abs(out_f["loss"].item())


def test_determinism_moe_rollout():
    b = make_batch(2, device="cuda", c=1.0, rows=2048)
    o1 = _run(b)
    g1 = o1["dlogits"].clone()
    o2 = _run(b)
    assert torch.equal(g1.view(torch.int16), o2["dlogits"].view(torch.int16))
    for k in ("logp_train", "w", "trunc", "terms", "loss"):
        assert torch.equal(o1[k], o2[k]), k
    s1, s2 = cis.read_stats(o1["workspace"]), cis.read_stats(o2["workspace"])
    assert s1 == s2
