"""Parity helpers: run the CPU oracle on the same inputs as the HIP path and compare.

Tolerances (the readings used by every parity test):

* valid / bad-id flags and the zero rows of invalid tokens: bit-exact.
* truncation flags: bit-exact, except tokens whose oracle margin |Delta - log1p(lambda*phi)|
  is below 1e-5, where either flag is a correct result (the weight is continuous there).
* l_train: |gpu - ref| <= 1e-5 |ref| + 2e-6 (float32 log-sum-exp resolution).
* w: relative 1e-5.
* term: |gpu - ref| <= 1e-5 |ref| + 2e-6 |scale w A|; loss: <= 1e-5 sum_t |term_t| + 1e-6.
* float32 gradient: |g - g64| <= 2e-5 |g64| + 2^-126 (G_REL: the float32 evaluation of
  coef * exp(z - lse), whose argument and exponential carry a few 1e-6 relative).
* bf16 gradient: every element is the round-to-nearest-even bfloat16 of some value within
  that float32 tolerance of the float64 gradient: it equals the correctly rounded g64 except
  where g64 lies within 2e-5 |g64| of a rounding midpoint, where either neighbour is correct;
  values below 2^-126 may be flushed to zero. (bfloat16's unit roundoff 2^-8 exceeds the
  2e-3 relative bound, so the bound is taken against the best bfloat16 answer.) Reported
  beside it: the bit-equal fraction, the fraction within 2e-3 relative of g64, and per row
  ||g - g_ref|| / ||g_ref|| against g_ref = RNE(g64) over the elements outside the midpoint
  bands, which must be <= 2e-3 (it is 0 when the elementwise criterion holds; a row whose
  norm sits in one element near a midpoint can exceed 2e-3 over all elements while every
  element is a correct rounding, and that value is reported as well).
"""

from __future__ import annotations

import math
import multiprocessing as mp
import os

import numpy as np
import torch

from oracle import cis as O

F32_TINY = 2.0 ** -126
G_REL = 2e-5


def write_report(filename: str, report: dict) -> None:
    """Writes a test's comparison report as JSON into the directory named by the environment
    variable CIS_PARITY_REPORT_DIR; nothing is written when it is not set."""
    import json
    out = os.environ.get("CIS_PARITY_REPORT_DIR")
    if not out:
        return
    os.makedirs(out, exist_ok=True)
    rep = {k: v for k, v in report.items() if not str(k).startswith("_")}
    with open(os.path.join(out, filename), "w") as f:
        json.dump(rep, f, indent=1, default=str)


def host_logits(logits: torch.Tensor):
    """Host copy of device logits whose rows read exactly as float64: a Bf16Matrix of the
    bfloat16 bit patterns, or a float64 array for float32 logits."""
    if logits.dtype == torch.bfloat16:
        bits = logits.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        return O.Bf16Matrix(bits)
    return logits.cpu().double().numpy()


def f32(x: float) -> float:
    return float(np.float32(x))


# ------------------------------------------------------------------------------------------
# gradient comparison of one block of rows (runs inside the pool workers)
# ------------------------------------------------------------------------------------------
def grad_stats(g: np.ndarray, g64: np.ndarray, bf16: bool) -> dict:
    """Counts for the gradient criteria on a block of rows (both float64 arrays [n, V])."""
    st = {"n_el": int(g.size), "n_rows": int(g.shape[0])}
    nrm = np.linalg.norm(g64, axis=1)
    rel64 = np.linalg.norm(g - g64, axis=1) / np.where(nrm > 0, nrm, 1.0)
    st["max_row_rel_l2_vs_f64"] = float(rel64.max()) if rel64.size else 0.0
    st["zero_row_violations"] = int(np.sum(np.any(g[nrm == 0] != 0, axis=1)))
    if bf16:
        rnd = lambda x: O.bf16_bits_to_float64(O.round_float64_to_bf16_bits(x))  # noqa: E731
        slack = G_REL * np.abs(g64)
        lo, hi = rnd(g64 - slack), rnd(g64 + slack)
        ok = (g >= lo) & (g <= hi)
        flush = (np.abs(g64) < F32_TINY * (1.0 + G_REL)) & (np.abs(g) <= F32_TINY)
        ok |= flush
        st["out_of_tolerance"] = int((~ok).sum())
        rn = rnd(g64)
        st["bit_equal"] = int(np.sum(g == rn))
        st["midpoint_band"] = int(np.sum((lo != hi) & ~flush))
        st["within_2e-3_rel"] = int(np.sum(np.abs(g - g64) <= 2e-3 * np.abs(g64)))
        # per row, against the correctly rounded bfloat16 reference; entries below the float32
        # normal range (which may be flushed) are left out of both sides, and the criterion row
        # value also leaves out the midpoint bands
        keep = np.abs(g64) >= F32_TINY
        rnk = np.where(keep, rn, 0.0)
        nrn = np.linalg.norm(rnk, axis=1)
        den = np.where(nrn > 0, nrn, 1.0)
        rel_all = np.linalg.norm(np.where(keep, g, 0.0) - rnk, axis=1) / den
        st["max_row_rel_l2_all_elements"] = float(rel_all.max()) if rel_all.size else 0.0
        st["rows_over_2e-3_all_elements"] = int(np.sum(rel_all > 2e-3))
        out = keep & (lo == hi)
        rel = np.linalg.norm(np.where(out, g, 0.0) - np.where(out, rn, 0.0), axis=1) / den
    else:
        rel = rel64
        err = np.abs(g - g64)
        st["out_of_tolerance"] = int(np.sum(err > G_REL * np.abs(g64) + F32_TINY))
        st["max_rel"] = float(np.max(err / np.maximum(np.abs(g64), F32_TINY))) if g.size else 0.0
        st["bit_equal"] = int(np.sum(g == g64.astype(np.float32)))
        st["within_2e-3_rel"] = int(np.sum(err <= 2e-3 * np.abs(g64)))
    st["max_row_rel_l2"] = float(rel.max()) if rel.size else 0.0
    return st


def merge_grad_stats(parts) -> dict:
    out = {}
    for st in parts:
        for k, v in st.items():
            if k.startswith("max"):
                out[k] = max(out.get(k, 0.0), v)
            else:
                out[k] = out.get(k, 0) + v
    return out


# ------------------------------------------------------------------------------------------
# oracle over many rows (process pool; each worker runs the plain oracle on a block of rows)
# ------------------------------------------------------------------------------------------
_SHARED = {}


def _worker(args):
    rows, pos, with_grad = args
    d = _SHARED
    res = O.cis_loss(d["z"], d["ids"], d["linf"], d["adv"], d["mask"], d["lam"], d["kappa"],
                     d["scale"], with_grad=with_grad, rows=rows)
    gst = None
    if with_grad and d.get("gdev") is not None:
        fin = (res.flags & O.FLAG_NONFINITE) == 0
        gdev = d["gdev"]
        # gdev holds either every row of the batch or only the compared ones, in order
        at = pos if d["gdev_compared_only"] else rows
        g = O.bf16_bits_to_float64(gdev[at]) if gdev.dtype == np.uint16 else \
            gdev[at].astype(np.float64)
        gst = grad_stats(g[fin], res.grad[fin], gdev.dtype == np.uint16)
        res.grad = None
    return rows, res, gst


def _nproc() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


# Largest number of gradient elements a worker holds per block (each float64 array of a block
# is then at most 64 MB; the comparison keeps a handful of them alive).
_BLOCK_ELEMENTS = 1 << 23


def run_oracle(z, ids, linf, adv, mask, lam, kappa, scale, rows=None, with_grad=True,
               gdev=None, procs=None, gdev_compared_only=False) -> dict:
    """Oracle results for `rows` (all rows if None) as a dict of arrays indexed like rows.

    With `gdev` (the device gradient on the host: uint16 bf16 bits or float32, [T, V], or
    only the compared rows in the order of `rows` when gdev_compared_only) the workers compare
    gradients themselves and only the merged counts come back ("grad_stats"); otherwise the
    float64 gradient rows are returned under "grad".
    """
    T, V = z.shape
    rows = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    _SHARED.clear()
    _SHARED.update(z=z, ids=ids, linf=linf, adv=adv, mask=mask, lam=lam, kappa=kappa,
                   scale=scale, gdev=gdev, gdev_compared_only=gdev_compared_only)
    procs = _nproc() if procs is None else procs
    nblk = procs * 4
    if with_grad:
        nblk = max(nblk, -(-len(rows) * V // _BLOCK_ELEMENTS))
    pos = np.arange(len(rows))
    blocks = [(r, p) for r, p in zip(np.array_split(rows, max(1, min(len(rows), nblk))),
                                     np.array_split(pos, max(1, min(len(rows), nblk)))) if len(r)]
    if procs > 1 and len(blocks) > 1:
        ctx = mp.get_context("fork")
        with ctx.Pool(procs) as pool:
            parts = pool.map(_worker, [(r, p, with_grad) for r, p in blocks])
    else:
        parts = [_worker((r, p, with_grad)) for r, p in blocks]
    _SHARED.clear()
    out = {k: [] for k in ("logp_train", "w", "trunc", "term", "flags", "grad")}
    gsts = []
    for b, r, gst in parts:
        out["logp_train"].append(r.logp_train)
        out["w"].append(r.w)
        out["trunc"].append(r.trunc)
        out["term"].append(r.term)
        out["flags"].append(r.flags)
        if r.grad is not None:
            out["grad"].append(r.grad)
        if gst is not None:
            gsts.append(gst)
    res = {k: np.concatenate(v) for k, v in out.items() if v}
    res["rows"] = rows
    if gsts:
        res["grad_stats"] = merge_grad_stats(gsts)
    return res


def device_grad_host(g: torch.Tensor, V: int) -> np.ndarray:
    g = g[:, :V]
    if g.dtype == torch.bfloat16:
        return g.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    return g.contiguous().cpu().numpy()


def oracle_for_batch(b, rows=None, with_grad=True, grad=None, z=None) -> dict:
    """Oracle on batch `b`; pass the device gradient as `grad` to compare it in the workers.

    `z` is the batch's logits already on the host (host_logits), to reuse one copy for several
    comparisons. When `rows` is given, only those rows of `grad` are copied to the host.
    """
    z = host_logits(b.logits) if z is None else z
    mask = None if b.mask is None else b.mask.cpu().numpy()
    compared_only = grad is not None and rows is not None
    if grad is None:
        gdev = None
    elif compared_only:
        idx = torch.as_tensor(np.asarray(rows, dtype=np.int64), device=grad.device)
        gdev = device_grad_host(grad.index_select(0, idx), b.V)
    else:
        gdev = device_grad_host(grad, b.V)
    return run_oracle(z, b.ids.cpu().numpy(), b.logp_infer.cpu().double().numpy(),
                      b.adv.cpu().double().numpy(), mask, f32(b.lam), f32(b.kappa), f32(b.scale),
                      rows=rows, with_grad=with_grad or grad is not None, gdev=gdev,
                      gdev_compared_only=compared_only)


# ------------------------------------------------------------------------------------------
# comparison
# ------------------------------------------------------------------------------------------
def trunc_margin(ref: dict, linf: np.ndarray, lam: float, kappa: float) -> np.ndarray:
    """|Delta - log1p(lambda*phi)| of the oracle for each compared row (inf on invalid rows)."""
    rows = ref["rows"]
    lt = ref["logp_train"]
    one_m_p = -np.expm1(lt)
    phi = np.maximum(one_m_p, kappa)
    m = np.abs((lt - linf[rows]) - np.log1p(lam * phi))
    return np.where(ref["flags"] & O.FLAG_VALID, m, np.inf)


def compare_scalars(out: dict, ref: dict, b, report: dict) -> None:
    rows = ref["rows"]
    lam, kappa, scale = f32(b.lam), f32(b.kappa), f32(b.scale)
    linf = b.logp_infer.cpu().double().numpy()
    adv = b.adv.cpu().double().numpy()
    valid = (ref["flags"] & O.FLAG_VALID) > 0
    fin = valid & ((ref["flags"] & O.FLAG_NONFINITE) == 0)

    lt = out["logp_train"].cpu().double().numpy()[rows]
    w = out["w"].cpu().double().numpy()[rows]
    tr = out["trunc"].cpu().numpy()[rows].astype(bool)
    term = out["terms"].cpu().double().numpy()[rows]

    # invalid rows: exact zeros
    assert np.all(lt[~valid] == 0) and np.all(w[~valid] == 0) and np.all(term[~valid] == 0)
    assert not tr[~valid].any()

    with np.errstate(invalid="ignore"):
        err_lt = np.where(lt == ref["logp_train"], 0.0, np.abs(lt - ref["logp_train"]))[fin]
    assert np.all(err_lt <= 1e-5 * np.abs(ref["logp_train"][fin]) + 2e-6), \
        f"logp_train: max err {err_lt.max():.3g}"
    rel_w = (np.abs(w - ref["w"]) / np.maximum(np.abs(ref["w"]), 1e-300))[fin]
    assert np.all(rel_w <= 1e-5), f"w: max rel err {rel_w.max():.3g}"
    coefmag = np.abs(scale * ref["w"] * adv[rows])
    err_t = np.abs(term - ref["term"])[fin]
    assert np.all(err_t <= 1e-5 * np.abs(ref["term"][fin]) + 2e-6 * coefmag[fin]), \
        f"term: max err {err_t.max():.3g}"

    margin = trunc_margin(ref, linf, lam, kappa)
    differ = (tr != ref["trunc"]) & fin
    assert np.all(margin[differ] < 1e-5), \
        f"{int((differ & (margin >= 1e-5)).sum())} truncation flags differ outside the margin"
    report.update(rows=int(len(rows)), valid=int(valid.sum()), trunc=int(ref["trunc"].sum()),
                  trunc_in_margin_differ=int(differ.sum()),
                  max_rel_w=float(rel_w.max()) if rel_w.size else 0.0,
                  max_err_logp=float(err_lt.max()) if err_lt.size else 0.0)


def compare_loss(out: dict, ref_all: dict, report: dict) -> None:
    """Scalar loss against the oracle's fsum over all rows (ref_all must cover every row)."""
    L = float(out["loss"].item())
    terms = ref_all["term"]
    L64 = math.fsum(terms.tolist())
    bound = 1e-5 * float(np.sum(np.abs(terms))) + 1e-6
    assert abs(L - L64) <= bound, f"loss {L} vs {L64} (bound {bound:.3g})"
    report.update(loss=L, loss_ref=L64)


def check_grad_stats(st: dict, report: dict) -> None:
    assert st["out_of_tolerance"] == 0, f"{st['out_of_tolerance']} gradient elements out of tolerance"
    assert st["zero_row_violations"] == 0
    assert st["max_row_rel_l2"] <= 2e-3, f"row rel L2 {st['max_row_rel_l2']:.3g}"
    report["grad"] = dict(st, bit_equal_frac=st["bit_equal"] / max(st["n_el"], 1),
                          within_2e_3_frac=st["within_2e-3_rel"] / max(st["n_el"], 1))
