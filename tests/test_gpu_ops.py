"""The operator family, the decoupled PPO-clip path and the diagnostics on the GPU, against
oracle.ops (tolerances in tests/parity_ops.py): every operator at update ratio 1 and on the
decoupled path, the sequence operators over packed responses, cis_weights_ex on recorded
log-probabilities (with saturated probabilities), float32 logits, long rows, and the
decoupled path at the full MoE-rollout size on sampled rows."""

import math

import numpy as np
import pytest
import torch

import paper_2609_32444_amd as cis
from oracle import cis as O
from oracle import ops as X
from tests import parity as P
from tests import parity_ops as PO
from tests.parity_ops import make_params
from workloads import make_batch, make_random_batch, old_logprobs, response_offsets

pytestmark = pytest.mark.gpu
DEV = "cuda"

# (operator, bounds) at update ratio 1; bounds other than the paper's defaults put many tokens
# on both sides of them
TOKEN_OPS = [
    ("cis", X.OP_CIS, dict(lam=2.3, kappa=5e-3)),
    ("cis_lam0_kappa0", X.OP_CIS, dict(lam=0.0, kappa=0.0)),
    ("none", X.OP_NONE, {}),
    ("exact", X.OP_EXACT, dict(lo=1e-6, hi=1e6)),
    ("exact_narrow", X.OP_EXACT, dict(lo=0.4, hi=2.5)),
    ("tis", X.OP_TIS, dict(hi=2.0)),
    ("tis_1.13", X.OP_TIS, dict(hi=1.13)),
    ("icepop", X.OP_ICEPOP, dict(lo=0.5, hi=5.0)),
    ("icepop_narrow", X.OP_ICEPOP, dict(lo=0.8, hi=1.25)),
    ("kpop", X.OP_KPOP, dict(hi=2.0)),
    ("kpop_tight", X.OP_KPOP, dict(hi=0.05)),
    ("two_sided", X.OP_TWO_SIDED, dict(lam=2.3, kappa=5e-3)),
    ("qfixed", X.OP_QFIXED, dict(lam=math.e - 1)),
]
SEQ_OPS = [
    ("seq_tis", X.OP_SEQ_TIS, dict(hi=2.0)),
    ("seq_mis", X.OP_SEQ_MIS, dict(lo=0.5, hi=2.0)),
]


def f32(x):
    return float(np.float32(x))


def _dump(name, rep):
    P.write_report(f"parity_ops_{name}.json", rep)


def run_case(name, b, op, kw, logp_old=None, offsets=None, bwd=True, rows=None):
    prm_dev, prm_ref = make_params(op, kw, b.scale)
    fn = cis.loss_bwd_ex if bwd else cis.loss_fwd_ex
    out = fn(b.logits, b.ids, b.logp_infer, b.adv, b.mask, params=prm_dev, logp_old=logp_old,
             seq_offsets=offsets, V=b.V)
    torch.cuda.synchronize()
    ref = PO.run_ops_oracle(b, prm_ref, logp_old=logp_old, offsets=offsets, rows=rows,
                            grad=out["dlogits"] if bwd else None, acted=out["acted"])
    rep = {"case": name}
    PO.compare_ops(out, ref, b, prm_ref, rep, logp_old=logp_old, offsets=offsets,
                   check_loss=rows is None)
    if bwd:
        P.check_grad_stats(ref["grad_stats"], rep)
    if rows is None:
        PO.check_diagnostics(cis.read_stats(out["workspace"]), ref, rep["_differ"], rep)
    _dump(name, rep)
    return out, ref, rep


def small_batch(V=3001, T=96, dtype=torch.bfloat16, seed=1, delta_sd=1.5):
    epv = 8 if dtype == torch.bfloat16 else 4
    ld = (V + epv - 1) // epv * epv + epv
    return make_random_batch(T, V, dtype, DEV, seed=seed, delta_sd=delta_sd, mask_p=0.85, ld=ld)


@pytest.mark.parametrize("name,op,kw", TOKEN_OPS, ids=[t[0] for t in TOKEN_OPS])
def test_rate1_operator(name, op, kw):
    b = small_batch(seed=11 + op)
    _, ref, rep = run_case(f"rate1_{name}", b, op, kw)
    if name not in ("none", "exact", "kpop"):   # the others act on part of this batch
        assert rep["acted"] > 0


@pytest.mark.parametrize("name,op,kw", TOKEN_OPS + SEQ_OPS, ids=[t[0] for t in TOKEN_OPS + SEQ_OPS])
def test_decoupled_operator(name, op, kw):
    b = small_batch(seed=31 + op, T=160)
    lold = old_logprobs(b, sd=0.3, seed=op)
    offs = response_offsets(b.T, 3, 30, seed=op) if op in X.SEQ_OPS else None
    _, ref, rep = run_case(f"decoupled_{name}", b, op, kw, logp_old=lold, offsets=offs)
    valid = (ref["flags"] & O.FLAG_VALID) > 0
    # the update ratio spans both sides of the clip range, so the gate closes somewhere
    assert np.any(~ref["gate"][valid]) and np.any(ref["gate"][valid])


def test_rate1_cis_matches_base_entry_point_bitwise():
    b = small_batch(V=32768, T=64, seed=5)
    prm, _ = make_params(X.OP_CIS, dict(lam=b.lam, kappa=b.kappa), b.scale)
    a = cis.loss_bwd(b.logits, b.ids, b.logp_infer, b.adv, b.mask, lam=b.lam, kappa=b.kappa,
                     scale=b.scale, V=b.V)
    e = cis.loss_bwd_ex(b.logits, b.ids, b.logp_infer, b.adv, b.mask, params=prm, V=b.V)
    torch.cuda.synchronize()
    for k in ("logp_train", "w", "terms", "loss"):
        assert torch.equal(a[k], e[k]), k
    assert torch.equal(a["trunc"], e["acted"])
    assert torch.equal(a["dlogits"].view(torch.int16), e["dlogits"].view(torch.int16))
    sa, se = cis.read_stats(a["workspace"]), cis.read_stats(e["workspace"])
    assert sa == se


def test_forward_only_ex_matches_fused():
    b = small_batch(V=20000, T=64, seed=6)
    lold = old_logprobs(b, sd=0.3, seed=1)
    prm, _ = make_params(X.OP_TIS, dict(hi=2.0), b.scale)
    f = cis.loss_fwd_ex(b.logits, b.ids, b.logp_infer, b.adv, b.mask, params=prm, logp_old=lold,
                        V=b.V)
    g = cis.loss_bwd_ex(b.logits, b.ids, b.logp_infer, b.adv, b.mask, params=prm, logp_old=lold,
                        V=b.V)
    torch.cuda.synchronize()
    for k in ("w", "acted", "eps"):
        assert torch.equal(f[k], g[k]), k
    for k in ("logp_train", "terms"):
        d = (f[k].double() - g[k].double()).abs()
        assert torch.all(d <= 1e-5 * f[k].double().abs() + 2e-6), k


@pytest.mark.parametrize("V,dtype,op,kw", [
    (200003, torch.bfloat16, X.OP_TIS, dict(hi=2.0)),          # LDS-resident slots
    (262144, torch.bfloat16, X.OP_ICEPOP, dict(lo=0.5, hi=5.0)),  # streamed remainder
    (90001, torch.float32, X.OP_CIS, dict(lam=2.3, kappa=5e-3)),
    (4097, torch.float32, X.OP_KPOP, dict(hi=0.05)),
])
def test_decoupled_long_and_float32_rows(V, dtype, op, kw):
    b = small_batch(V=V, T=24, dtype=dtype, seed=V % 1000)
    lold = old_logprobs(b, sd=0.3, seed=2)
    run_case(f"decoupled_V{V}_{str(dtype)[6:]}", b, op, kw, logp_old=lold)


def test_decoupled_many_rows_per_workgroup():
    b = small_batch(V=4000, T=3000, seed=77)
    lold = old_logprobs(b, sd=0.3, seed=3)
    offs = response_offsets(b.T, 50, 400, seed=4)
    run_case("decoupled_seq_tis_T3000", b, X.OP_SEQ_TIS, dict(hi=2.0), logp_old=lold,
             offsets=offs)


def _recorded_logprobs(n, seed):
    g = np.random.default_rng(seed)
    lp = np.log(g.uniform(1e-4, 1.0, size=n))
    lq = lp - g.normal(0, 1.2, size=n)
    lq = np.minimum(lq, 0.0)
    # saturated and extreme tokens (App. D.5): p = 1, q = 1, both, tiny probabilities
    lp[:6] = [0.0, 0.0, -1e-9, -40.0, -0.3, 0.0]
    lq[:6] = [0.0, -2.0, 0.0, -0.1, -60.0, -1e-8]
    return lp.astype(np.float32), lq.astype(np.float32)


@pytest.mark.parametrize("name,op,kw", TOKEN_OPS + SEQ_OPS, ids=[t[0] for t in TOKEN_OPS + SEQ_OPS])
def test_weights_ex(name, op, kw):
    n = 5000
    lp, lq = _recorded_logprobs(n, seed=op)
    mask = (np.random.default_rng(op + 100).random(n) < 0.9).astype(np.uint8)
    offs = response_offsets(n, 1, 60, seed=op, device="cpu").numpy() if op in X.SEQ_OPS else None
    prm_dev, prm_ref = make_params(op, kw, 1.0)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    out = cis.weights_ex(t(lp), t(lq), t(mask), params=prm_dev,
                         seq_offsets=None if offs is None else t(offs))
    torch.cuda.synchronize()
    w = out["w"].cpu().double().numpy()
    acted = out["acted"].cpu().numpy().astype(bool)
    eps = out["eps"].cpu().double().numpy()
    lp64, lq64 = lp.astype(np.float64), lq.astype(np.float64)
    valid = mask.astype(bool)
    if op in X.SEQ_OPS:
        wr, ar, logK = X.seq_weights(op, lp64 - lq64, valid, offs, prm_ref)
        seg = np.searchsorted(offs, np.arange(n), side="right") - 1
        margin = np.minimum(np.abs(logK[seg] - math.log(prm_ref.hi)),
                            np.abs(logK[seg] - (math.log(prm_ref.lo) if prm_ref.lo > 0 else -np.inf)))
    else:
        wa = [X.token_weight(op, a, c, -math.expm1(a), prm_ref) if v else (0.0, False)
              for a, c, v in zip(lp64, lq64, valid)]
        wr = np.array([x[0] for x in wa])
        ar = np.array([x[1] for x in wa])
        margin = PO.op_margin(op, prm_ref, lp64 - lq64, lp64, lq64, -np.expm1(lp64))
    differ = (acted != ar) & valid
    assert np.all(margin[differ] < PO.margin_tol(op)), int(differ.sum())
    same = valid & ~differ
    err = np.abs(w[same] - wr[same])
    assert np.all(err <= 1e-5 * np.abs(wr[same]) + P.F32_TINY), err.max()
    assert np.all(w[~valid] == 0) and not acted[~valid].any() and np.all(eps[~valid] == 0)
    er = np.array([X.displacement(a, c, -math.expm1(a)) if v else 0.0
                   for a, c, v in zip(lp64, lq64, valid)])
    inf = np.isinf(er) | np.isinf(eps)
    assert np.array_equal(er[inf], eps[inf])
    assert np.all(np.abs(eps[~inf] - er[~inf]) <= 1e-4 * np.abs(er[~inf]) + 1e-5)
    st = cis.read_stats(out["workspace"])
    assert st["n_valid"] == int(valid.sum()) and st["loss"] == 0.0
    assert abs(st["n_trunc"] - int(ar[valid].sum())) <= int(differ.sum())
    mx = float(np.max(np.abs(lp64 - lq64)[valid]))
    assert abs(st["max_abs_logk"] - mx) <= 1e-6 * mx


def test_decoupled_full_size_moe_rollout():
    b = make_batch(2, device=DEV, c=1.0)
    lold = old_logprobs(b, sd=0.3, seed=9)
    # responses packed back to back with the batch's length range (256-1536 tokens)
    offs = response_offsets(b.T, 256, 1536, seed=2)
    rows = sample_rows(b.T, 192, seed=12)
    for name, op, kw in (("cis", X.OP_CIS, dict(lam=b.lam, kappa=b.kappa)),
                         ("seq_tis", X.OP_SEQ_TIS, dict(hi=2.0))):
        run_case(f"decoupled_full_{name}", b, op, kw, logp_old=lold,
                 offsets=offs if op in X.SEQ_OPS else None, rows=rows)


def sample_rows(T, n, seed):
    g = np.random.default_rng(seed)
    return np.unique(np.concatenate([[0, T - 1], g.choice(T, size=n, replace=False)]))
