"""The loss behind the LM head on the GPU (cis_lmhead_loss_fwd / _bwd) against oracle.lmhead.

Inputs come from workloads.make_lmhead_batch, whose hidden states and head weight make every
float32 partial sum of h W^T exact: the chunk's float32 logits equal the oracle's float64 ones,
so the per-row outputs, the loss and the diagnostics take the tolerances of tests/parity.py and
tests/parity_ops.py unchanged.

Gradients. The kernel rounds G = dL/dz (float32, within 2e-5 |G| + 2^-126 of the float64 G) to
bf16 as the operand of dL/dh = G W and dL/dW = G^T h, and accumulates in float32. Per element
of dL/dh (dL/dW likewise with |G|^T |h|):

    |gpu - ref| <= (2^-8 + 4e-5 + (8 sqrt(K) + n_add) 2^-24) (|G| |W|) + 1e-30

2^-8 is the unit roundoff of bf16 (8-bit significand, round to nearest even), 4e-5 covers the
float32 G, K is the contracted length (V for dL/dh, the rows of one dL/dW group for dL/dW) and
n_add the float32 additions of whole partial results (1 for dL/dh; the number of groups for
dL/dW, which is accumulated group by group). The accumulation term is the probabilistic bound of blocked
float32 summation (sqrt(K) u with a factor of 8) rather than the worst case K u, which at
K = 151936 would allow 0.9% and test nothing.
"""

import math

import numpy as np
import pytest
import torch

import paper_2609_32444_amd as cis
from oracle import lmhead as L
from oracle import ops as X
from tests import parity as P
from tests import parity_ops as PO
from tests.parity_ops import make_params
from workloads import make_lmhead_batch

pytestmark = pytest.mark.gpu
DEV = "cuda"
U32 = 2.0 ** -24
U16 = 2.0 ** -8


def f32(x):
    return float(np.float32(x))


def host(b):
    return (b.hidden.float().cpu().double().numpy(), b.weight.float().cpu().double().numpy())


def _dump(name, rep):
    P.write_report(f"parity_lmhead_{name}.json", rep)


def dw_group(chunk, T):
    """Rows per dL/dW product (cis_lmhead_loss_bwd in include/cis.h) and the number of them."""
    g = chunk * (16384 // chunk) if chunk % 8 == 0 and chunk < 16384 else chunk
    return min(g, T), (T + g - 1) // g


def grad_bound(Gabs_B, K, n_add):
    return (U16 + 4e-5 + (8.0 * math.sqrt(max(K, 1)) + n_add) * U32) * Gabs_B + 1e-30


def check_grad(name, gpu, ref, bound, rows_ok=None):
    err = np.abs(gpu - ref)
    if rows_ok is not None:
        err, ref, bound = err[rows_ok], ref[rows_ok], bound[rows_ok]
    bad = err > bound
    rel = np.linalg.norm(err) / max(np.linalg.norm(ref), 1e-300)
    if bad.any():
        i = np.unravel_index(int(np.argmax(err - bound)), err.shape)
        raise AssertionError(f"{name}: {int(bad.sum())} elements out of tolerance; worst at {i}: "
                             f"err {err[i]:.3g} bound {bound[i]:.3g} ref {ref[i]:.3g}")
    return {"max_err_over_bound": float(np.max(err / bound)) if err.size else 0.0,
            "rel_fro": float(rel)}


def ref_dict(res):
    return {"rows": np.arange(len(res.w)), "flags": res.flags, "logp_train": res.logp_train,
            "w": res.w, "term": res.term, "eps": res.eps, "logk": res.logk, "acted": res.acted,
            "rho": res.rho, "gate": res.gate}


def run_case(name, b, op=X.OP_CIS, kw=None, chunk=4096, decoupled=False, seq=False, bwd=True,
             recompute=False):
    kw = dict(lam=b.lam, kappa=b.kappa) if kw is None and op == X.OP_CIS else (kw or {})
    prm_dev, prm_ref = make_params(op, kw, b.scale)
    lold = b.logp_old if decoupled else None
    offs = b.offsets if seq else None
    if bwd:
        out = cis.lmhead_loss_bwd(b.hidden, b.weight, b.ids, b.logp_infer, b.adv, b.mask,
                                  params=prm_dev, logp_old=lold, seq_offsets=offs, chunk=chunk,
                                  recompute=recompute)
    else:
        out = cis.lmhead_loss_fwd(b.hidden, b.weight, b.ids, b.logp_infer, b.adv, b.mask,
                                  params=prm_dev, logp_old=lold, seq_offsets=offs, chunk=chunk)
    torch.cuda.synchronize()
    h, W = host(b)
    res = L.lmhead_cis_loss(h, W, b.ids.cpu().numpy(), b.logp_infer.cpu().double().numpy(),
                            b.adv.cpu().double().numpy(), b.mask.cpu().numpy(), prm_ref,
                            logp_old=None if lold is None else lold.cpu().double().numpy(),
                            offsets=None if offs is None else offs.cpu().numpy(),
                            with_grad=bwd, keep_grad=bwd)
    rep = {"case": name, "T": b.T, "V": b.V, "H": b.H, "chunk": chunk}
    ref = ref_dict(res)
    PO.compare_ops(out, ref, b, prm_ref, rep, logp_old=lold, offsets=offs)
    differ = rep.pop("_differ")
    stats = cis.read_stats(out["workspace"])
    PO.check_diagnostics(stats, ref, differ, rep)
    assert stats["n_valid"] == int(np.sum((res.flags & 1) > 0))
    if bwd:
        # rows whose acted flag or PPO gate may legitimately differ leave the gradient checks
        assert not differ.any(), "margin rows in a gradient case: pick another seed"
        if lold is not None:
            hi_c, lo_c = 1.0 + prm_ref.clip_high, 1.0 - prm_ref.clip_low
            near = (np.abs(res.rho - hi_c) <= 1e-5 * hi_c) | (np.abs(res.rho - lo_c) <= 1e-5 * lo_c)
            assert not near[(res.flags & 1) > 0].any(), "rows at the PPO clip edge: other seed"
        G = np.abs(res.grad)
        kdw, ngr = dw_group(chunk, b.T)
        dh = out["dhidden"].cpu().double().numpy()
        dW = out["dweight"].cpu().double().numpy()
        rep["dhidden"] = check_grad("dhidden", dh, res.dhidden, grad_bound(G @ np.abs(W), b.V, 1))
        rep["dweight"] = check_grad("dweight", dW, res.dW,
                                    grad_bound(G.T @ np.abs(h), kdw, ngr))
        inval = (res.flags & 1) == 0
        assert np.all(dh[inval] == 0), "dhidden rows of invalid tokens must be zero"
    _dump(name, rep)
    return out, res


SMALL = [
    # name, T, V, H, chunk, extra generator arguments
    ("one_chunk", 64, 1000, 64, 4096, {}),
    ("chunks_ragged", 300, 9001, 136, 128, {}),
    ("padded_H100", 200, 2053, 100, 64, dict(ld_h=104, ld_w=112)),
    ("masked", 257, 4099, 72, 128, dict(mask_p=0.7)),
    ("one_row", 1, 517, 2048, 4096, {}),
    ("vocab_1", 5, 1, 8, 4096, {}),
]


@pytest.mark.parametrize("recompute", [False, True], ids=["chunked_logits", "recompute"])
@pytest.mark.parametrize("name,T,V,H,chunk,gen", SMALL, ids=[c[0] for c in SMALL])
def test_lmhead_parity_small(name, T, V, H, chunk, gen, recompute):
    """Both backward modes: each chunk's float32 logits kept while G is formed, and the product
    formed again with an epilogue that writes G (the logits never stored)."""
    b = make_lmhead_batch(T, V, H, device=DEV, seed=11, min_len=16, max_len=96, **gen)
    run_case(name, b, chunk=chunk, recompute=recompute)


# ------------------------------------------------------------------------------------------
# General bf16 inputs: the logits' own float32 rounding, bounded from the inputs
# ------------------------------------------------------------------------------------------
U_ADD = 2.0 ** -23   # float32 unit roundoff, doubled to also cover a truncating adder


def _gamma(n):
    return n * U_ADD / (1.0 - n * U_ADD)


GENERAL = [
    # name, T, V, H, chunk
    ("vocab_151936", 128, 151936, 2048, 64),
    ("ragged_9001", 300, 9001, 2048, 128),
]


@pytest.mark.parametrize("recompute", [False, True], ids=["chunked_logits", "recompute"])
@pytest.mark.parametrize("name,T,V,H,chunk", GENERAL, ids=[g[0] for g in GENERAL])
def test_lmhead_general_bf16_inputs(name, T, V, H, chunk, recompute):
    """Hidden states N(0, 1) and head weights N(0, 4/(H-1)) rounded once to bf16, so the
    float32 logits h W^T carry their own dot-product rounding. The bounds follow from it:

    * each float32 logit is within E_v = gamma_H sum_k |h_k| |W_vk| of the exact one
      (gamma_n = n u / (1 - n u), u = 2^-23: any summation order, round-to-nearest or
      truncating additions); E = max_v E_v per row;
    * log-sum-exp moves by at most E, so l_train = z_y - lse by at most 2E; every
      probability, and 1 - p, by a factor within exp(+-2E): delta_p = expm1(2E);
    * w = min{k, 1 + lambda max(1 - p, kappa)} is then within delta_w = delta_p (+1e-5, the
      kernel's own float32 tolerance) relative; the truncation decision moves by at most 4E,
      so flags may differ where the oracle's margin is below 4E + 1e-5;
    * term = scale w A l_train and the loss follow by the product rule; G = coef (onehot - p)
      is within rho = delta_w (1 + delta_p) + delta_p relative per row, which widens the
      products' bounds of the module docstring by that factor.
    """
    b = make_lmhead_batch(T, V, H, device=DEV, seed=23, min_len=16, max_len=96, exact=False)
    prm_dev, prm_ref = make_params(X.OP_CIS, dict(lam=b.lam, kappa=b.kappa), b.scale)
    out = cis.lmhead_loss_bwd(b.hidden, b.weight, b.ids, b.logp_infer, b.adv, b.mask,
                              params=prm_dev, chunk=chunk, recompute=recompute)
    torch.cuda.synchronize()
    h, W = host(b)
    ids = b.ids.cpu().numpy()
    linf = b.logp_infer.cpu().double().numpy()
    adv = b.adv.cpu().double().numpy()
    res = L.lmhead_cis_loss(h, W, ids, linf, adv, b.mask.cpu().numpy(), prm_ref,
                            with_grad=True, keep_grad=True)
    valid = (res.flags & 1) > 0
    assert valid.all()
    E = _gamma(H) * (np.abs(h) @ np.abs(W).T).max(axis=1)
    dp = np.expm1(2.0 * E)
    dw = dp + 1e-5
    rho = dw * (1.0 + dp) + dp

    lt = out["logp_train"].cpu().double().numpy()
    w = out["w"].cpu().double().numpy()
    term = out["terms"].cpu().double().numpy()
    acted = out["acted"].cpu().numpy().astype(bool)
    lref, wref, tref = res.logp_train, res.w, res.term
    tol_l = 2.0 * E + 1e-5 * np.abs(lref) + 2e-6
    err_l = np.abs(lt - lref)
    assert np.all(err_l <= tol_l), f"l_train: worst err/bound {np.max(err_l / tol_l):.3g}"
    err_w = np.abs(w - wref)
    tol_w = dw * np.abs(wref) + P.F32_TINY
    assert np.all(err_w <= tol_w), f"w: worst err/bound {np.max(err_w / tol_w):.3g}"
    sA = np.abs(P.f32(b.scale) * adv)
    tol_t = sA * (dw * wref * np.abs(lref) + wref * (1.0 + dw) * tol_l) \
        + 1e-5 * np.abs(tref) + P.F32_TINY
    err_t = np.abs(term - tref)
    assert np.all(err_t <= tol_t), f"term: worst err/bound {np.max(err_t / tol_t):.3g}"
    one_m_p = -np.expm1(lref)
    margin = np.abs((lref - linf) - np.log1p(prm_ref.lam * np.maximum(one_m_p, prm_ref.kappa)))
    differ = acted != res.acted
    assert np.all(margin[differ] < 4.0 * E[differ] + 1e-5), "acted flags differ outside 4E"
    Lg, L64 = float(out["loss"].item()), res.loss
    assert abs(Lg - L64) <= float(np.sum(tol_t)) + 1e-5 * float(np.sum(np.abs(tref))) + 1e-6

    G = np.abs(res.grad)
    kdw, ngr = dw_group(chunk, b.T)
    dh = out["dhidden"].cpu().double().numpy()
    dW = out["dweight"].cpu().double().numpy()
    acc_h = (8.0 * math.sqrt(b.V) + 1) * U32
    acc_w = (8.0 * math.sqrt(kdw) + ngr) * U32
    ch = (1.0 + rho) * (U16 + 4e-5 + acc_h) + rho
    cw = (1.0 + rho) * (U16 + 4e-5 + acc_w) + rho
    rep = {"case": name, "T": T, "V": V, "H": H, "chunk": chunk,
           "max_E": float(E.max()), "max_err_logp_over_E": float(np.max(err_l / E)),
           "max_err_logp": float(err_l.max()), "acted_differ": int(differ.sum())}
    rep["dhidden"] = check_grad("dhidden", dh, res.dhidden,
                                ch[:, None] * (G @ np.abs(W)) + 1e-30)
    rep["dweight"] = check_grad("dweight", dW, res.dW, (cw[:, None] * G).T @ np.abs(h) + 1e-30)
    _dump(f"general_{name}_{'recompute' if recompute else 'chunked'}", rep)
    print(rep, flush=True)


def test_lmhead_products_with_more_tiles_than_cus():
    """Logits and dL/dW products of 314 tiles of 256 x 256 each (more than one per CU): their
    workgroups take tiles from the per-XCD work queues. The full comparison with the oracle, a
    ragged last tile in V, and a second call that must reproduce every output bit for bit
    (whichever workgroup takes a tile computes it the same way)."""
    b = make_lmhead_batch(512, 40000, 512, device=DEV, seed=13, min_len=16, max_len=96)
    out, _ = run_case("queued_products", b, chunk=512)
    prm, _ = make_params(X.OP_CIS, dict(lam=b.lam, kappa=b.kappa), b.scale)
    again = cis.lmhead_loss_bwd(b.hidden, b.weight, b.ids, b.logp_infer, b.adv, b.mask,
                                params=prm, chunk=512)
    torch.cuda.synchronize()
    for k in ("logp_train", "w", "acted", "terms", "eps", "loss", "dhidden", "dweight"):
        assert torch.equal(out[k], again[k]), k


@pytest.mark.parametrize("recompute", [False, True], ids=["chunked_logits", "recompute"])
def test_lmhead_queued_products_ragged_hidden(recompute):
    """H = 200 (three full 64-wide slabs and a masked one of 8) with a logits product of 314
    tiles: the queued products (with the stored chunk and pairs, or pairs then G) end their
    contraction on the masked slab, which is filled through registers. Against the oracle,
    and a second call reproduces every output bit for bit."""
    b = make_lmhead_batch(512, 40000, 200, device=DEV, seed=31, min_len=16, max_len=96)
    out, _ = run_case("queued_ragged_hidden", b, chunk=512, recompute=recompute)
    prm, _ = make_params(X.OP_CIS, dict(lam=b.lam, kappa=b.kappa), b.scale)
    again = cis.lmhead_loss_bwd(b.hidden, b.weight, b.ids, b.logp_infer, b.adv, b.mask,
                                params=prm, chunk=512, recompute=recompute)
    torch.cuda.synchronize()
    for k in ("logp_train", "w", "acted", "terms", "eps", "loss", "dhidden", "dweight"):
        assert torch.equal(out[k], again[k]), k


@pytest.mark.parametrize("recompute", [False, True], ids=["chunked_logits", "recompute"])
def test_lmhead_largest_vocabulary(recompute):
    """V = 2^22, the largest vocabulary the LM-head calls accept: float32 logit rows of 16 MB
    through the streamed row path (or 65536 pairs per row folded by the combine), a logits
    product of 16384 tiles, dL/dh split along V into 2^19-long contractions and dL/dW over all
    2^22 rows, every output against the oracle."""
    b = make_lmhead_batch(64, 1 << 22, 64, device=DEV, seed=17, min_len=16, max_len=32)
    run_case("max_vocab", b, chunk=64, recompute=recompute)


def test_lmhead_largest_chunk():
    """chunk = 2^16, the largest the LM-head calls accept, over a batch of exactly that many
    rows: one logits product of 65536 rows and one dL/dW group of K = 65536, against the
    oracle."""
    b = make_lmhead_batch(1 << 16, 1000, 64, device=DEV, seed=19, min_len=64, max_len=512)
    run_case("max_chunk", b, chunk=1 << 16)


def test_lmhead_largest_hidden_size():
    """H = 2^16, the largest hidden size the LM-head calls accept: logits contracted over 65536
    (1024 slabs), dL/dh and dL/dW 256 tiles wide. The per-token inputs come from a small batch;
    hidden and weight entries are {-1, 0, 1} * 2^-3, so every float32 partial sum of a logit is
    an integer multiple of 2^-6 below 2^17 in magnitude, exact, and the logits equal the
    oracle's float64 ones as with make_lmhead_batch."""
    import dataclasses
    T, V, H = 64, 1000, 1 << 16
    b0 = make_lmhead_batch(T, V, 64, device=DEV, seed=29, min_len=16, max_len=32)
    g = torch.Generator(device=DEV)
    g.manual_seed(30)
    h = (torch.randint(-1, 2, (T, H), generator=g, device=DEV).float() * 0.125).to(torch.bfloat16)
    W = (torch.randint(-1, 2, (V, H), generator=g, device=DEV).float() * 0.125).to(torch.bfloat16)
    b = dataclasses.replace(b0, hidden=h, weight=W)
    run_case("max_hidden", b, chunk=64)


def test_lmhead_forward_matches_backward_and_chunking():
    b = make_lmhead_batch(300, 9001, 136, device=DEV, seed=5, min_len=16, max_len=96)
    prm, _ = make_params(X.OP_CIS, dict(lam=b.lam, kappa=b.kappa), b.scale)
    args = (b.hidden, b.weight, b.ids, b.logp_infer, b.adv, b.mask)
    a = cis.lmhead_loss_bwd(*args, params=prm, chunk=128)
    c = cis.lmhead_loss_bwd(*args, params=prm, chunk=4096)
    f = cis.lmhead_loss_fwd(*args, params=prm, chunk=256)
    torch.cuda.synchronize()
    # chunks that are multiples of the 128-row tile give the same logits and per-row results
    for k in ("logp_train", "w", "acted", "terms", "eps", "loss"):
        assert torch.equal(a[k], c[k]), k
    assert torch.equal(a["dhidden"], c["dhidden"])
    # the forward-only kernel may sum a row in another order: float32 rounding apart
    for k in ("logp_train", "w", "terms"):
        assert torch.allclose(a[k], f[k], rtol=1e-5, atol=2e-6), k
    assert torch.equal(a["acted"], f["acted"])
    # both chunkings form dL/dW in one product over all 300 rows (one group)
    assert torch.equal(a["dweight"], c["dweight"])


TOKEN_OPS = [("icepop", X.OP_ICEPOP, dict(lo=0.5, hi=5.0)), ("tis", X.OP_TIS, dict(hi=2.0)),
             ("kpop", X.OP_KPOP, dict(hi=2.0)), ("two_sided", X.OP_TWO_SIDED, {})]


@pytest.mark.parametrize("name,op,kw", TOKEN_OPS, ids=[o[0] for o in TOKEN_OPS])
def test_lmhead_operators(name, op, kw):
    b = make_lmhead_batch(200, 3001, 64, device=DEV, seed=21, min_len=16, max_len=96,
                          delta_sd=0.5)
    run_case(f"op_{name}", b, op=op, kw=kw, chunk=128)


@pytest.mark.parametrize("name,op,kw,seq", [
    ("ppo_cis", X.OP_CIS, dict(lam=math.e - 1, kappa=5e-3), False),
    ("ppo_icepop", X.OP_ICEPOP, dict(lo=0.5, hi=5.0), False),
    ("ppo_seq_tis", X.OP_SEQ_TIS, dict(hi=2.0), True),
])
@pytest.mark.parametrize("recompute", [False, True], ids=["chunked_logits", "recompute"])
def test_lmhead_decoupled(name, op, kw, seq, recompute):
    b = make_lmhead_batch(300, 2001, 64, device=DEV, seed=31, min_len=16, max_len=80,
                          delta_sd=0.3, old_sd=0.2)
    run_case(name, b, op=op, kw=kw, chunk=128, decoupled=True, seq=seq, recompute=recompute)


def test_lmhead_forward_only_parity():
    b = make_lmhead_batch(150, 5003, 96, device=DEV, seed=41, min_len=16, max_len=96)
    run_case("fwd_only", b, chunk=64, bwd=False)


def test_lmhead_empty_batch_and_accumulation():
    b = make_lmhead_batch(96, 1000, 64, device=DEV, seed=51, min_len=16, max_len=48)
    prm, _ = make_params(X.OP_CIS, dict(lam=b.lam, kappa=b.kappa), b.scale)
    e = torch.empty(0, device=DEV)
    ei = torch.empty(0, dtype=torch.int64, device=DEV)
    h0 = b.hidden[:0]
    dW = torch.full((1000, 64), 3.0, device=DEV)
    out = cis.lmhead_loss_bwd(h0, b.weight, ei, e, e, None, params=prm, dweight=dW,
                              accumulate=True)
    torch.cuda.synchronize()
    assert torch.all(out["dweight"] == 3.0)
    out = cis.lmhead_loss_bwd(h0, b.weight, ei, e, e, None, params=prm, dweight=dW)
    torch.cuda.synchronize()
    assert torch.all(out["dweight"] == 0.0) and float(out["loss"].item()) == 0.0
    # accumulate: dW0 + the gradient (3 chunks of 32 rows, one dL/dW group)
    args = (b.hidden, b.weight, b.ids, b.logp_infer, b.adv, b.mask)
    dW0 = torch.randn(1000, 64, device=DEV) * 1e-3
    acc = cis.lmhead_loss_bwd(*args, params=prm, chunk=32, dweight=dW0.clone(),
                              accumulate=True)["dweight"]
    torch.cuda.synchronize()
    _, prm_ref = make_params(X.OP_CIS, dict(lam=b.lam, kappa=b.kappa), b.scale)
    h, W = host(b)
    res = L.lmhead_cis_loss(h, W, b.ids.cpu().numpy(), b.logp_infer.cpu().double().numpy(),
                            b.adv.cpu().double().numpy(), b.mask.cpu().numpy(), prm_ref,
                            keep_grad=True)
    d0 = dW0.cpu().double().numpy()
    bound = grad_bound(np.abs(res.grad).T @ np.abs(h), *dw_group(32, b.T)) + 4 * U32 * np.abs(d0)
    check_grad("dweight_accumulated", acc.cpu().double().numpy(), d0 + res.dW, bound)


def test_lmhead_empty_batch_zero_dweight_from_work_queues():
    """No rows and a head of 157 x 2 tiles of 256 x 256 (more than one per CU): dL/dW = 0 comes
    from a product with an empty contraction whose tiles are taken from the work queues."""
    W = torch.randn(40000, 512, device=DEV).to(torch.bfloat16)
    prm, _ = make_params(X.OP_CIS, dict(lam=1.0, kappa=0.005), -1.0)
    e = torch.empty(0, device=DEV)
    ei = torch.empty(0, dtype=torch.int64, device=DEV)
    h0 = torch.empty(0, 512, dtype=torch.bfloat16, device=DEV)
    for _ in range(2):
        dW = torch.full((40000, 512), 3.0, device=DEV)
        out = cis.lmhead_loss_bwd(h0, W, ei, e, e, None, params=prm, dweight=dW)
        torch.cuda.synchronize()
        assert torch.all(out["dweight"] == 0.0) and float(out["loss"].item()) == 0.0


# ------------------------------------------------------------------------------------------
# the full LM-head workload in the configuration the benchmark times
# ------------------------------------------------------------------------------------------
FULL_T, FULL_V, FULL_H, FULL_CHUNK = 16384, 151936, 2048, cis.LMHEAD_CHUNK


@pytest.mark.parametrize("recompute", [False, True], ids=["chunked_logits", "recompute"])
def test_lmhead_full_size_sampled(recompute):
    """T = 16384, V = 151936, H = 2048 in chunks of 4096 rows, both backward modes: sampled rows
    against the oracle
    (per-row outputs and dL/dh rows), and for dL/dW the properties that hold at any size:
    <dW, W> = sum_t <dh_t, h_t> (both are sum_t <G_t, z_t> for the same bf16 G), and each
    column of dW sums to sum_t (sum_v G_tv) h_t with sum_v G_tv = 0 up to G's bf16 rounding."""
    b = make_lmhead_batch(FULL_T, FULL_V, FULL_H, device=DEV, seed=2, c=1.0)
    prm_dev, prm_ref = make_params(X.OP_CIS, dict(lam=b.lam, kappa=b.kappa), b.scale)
    out = cis.lmhead_loss_bwd(b.hidden, b.weight, b.ids, b.logp_infer, b.adv, b.mask,
                              params=prm_dev, chunk=FULL_CHUNK, recompute=recompute)
    torch.cuda.synchronize()
    stats = cis.read_stats(out["workspace"])
    assert stats["n_valid"] == FULL_T and stats["n_bad_id"] == 0 and stats["n_nonfinite"] == 0
    terms = out["terms"].double()
    assert abs(stats["loss"] - float(terms.sum())) <= 1e-9 * float(terms.abs().sum())
    g = torch.Generator().manual_seed(3)
    rows = sorted(set(torch.randint(0, FULL_T, (6,), generator=g).tolist()) | {0, FULL_T - 1})
    h, W = host(b)
    res = L.lmhead_cis_loss(h[rows], W, b.ids.cpu().numpy()[rows],
                            b.logp_infer.cpu().double().numpy()[rows],
                            b.adv.cpu().double().numpy()[rows], b.mask.cpu().numpy()[rows],
                            prm_ref, keep_grad=True)
    rep = {"case": "full_size", "rows": rows}
    for k, kk in (("logp_train", "logp_train"), ("w", "w"), ("terms", "term")):
        dev = out[k].cpu().double().numpy()[rows]
        ref = getattr(res, kk)
        assert np.all(np.abs(dev - ref) <= 1e-5 * np.abs(ref) + 2e-6), (k, dev, ref)
    dh = out["dhidden"].cpu().double().numpy()
    rep["dhidden_rows"] = check_grad("dhidden", dh[rows], res.dhidden,
                                     grad_bound(np.abs(res.grad) @ np.abs(W), FULL_V, 1))
    # dW properties; |G_tv| <= |c_t| (1{v = y} + p_tv) bounds sum_v |G_tv| S_tv by
    # 2 |c_t| max_v S_tv <= 2 |c_t| ||h_t||_1 max|W|
    dW = out["dweight"].double()
    hd = b.hidden.double()
    Wd = b.weight.double()
    c = (b.scale * out["w"].double() * b.adv.double()).abs()
    lhs = float((dW * Wd).sum())
    rhs = float((out["dhidden"].double() * hd).sum())
    kdw, ngr = dw_group(FULL_CHUNK, FULL_T)
    gam = (8 * math.sqrt(FULL_V) + 8 * math.sqrt(kdw) + ngr + 2) * U32
    bound = gam * 2 * float((c * hd.abs().sum(1)).sum()) * float(Wd.abs().max())
    assert abs(lhs - rhs) <= bound, (lhs, rhs, bound)
    col = dW.sum(0)
    cbound = (2 * U16 + gam) * 2 * (c[:, None] * hd.abs()).sum(0) + 1e-30
    assert torch.all(col.abs() <= cbound)
    rep.update(trace_lhs=lhs, trace_rhs=rhs, trace_bound=bound,
               colsum_max_over_bound=float((col.abs() / cbound).max()))
    _dump(f"full_size_{'recompute' if recompute else 'chunked'}", rep)


def test_lmhead_full_size_few_valid_rows_dweight():
    """The same configuration with only a few valid rows: dL/dW is then a sum over those rows,
    which the oracle forms exactly; compared on sampled vocabulary rows (the sampled ids
    included)."""
    b = make_lmhead_batch(FULL_T, FULL_V, FULL_H, device=DEV, seed=4, c=1.0)
    keep = torch.tensor([3, 5000, 9001, FULL_T - 2], device=DEV)
    b.mask.zero_()
    b.mask[keep] = 1
    b.scale = -1.0 / 4
    prm_dev, prm_ref = make_params(X.OP_CIS, dict(lam=b.lam, kappa=b.kappa), b.scale)
    out = cis.lmhead_loss_bwd(b.hidden, b.weight, b.ids, b.logp_infer, b.adv, b.mask,
                              params=prm_dev, chunk=FULL_CHUNK)
    torch.cuda.synchronize()
    rows = keep.cpu().numpy()
    h, W = host(b)
    res = L.lmhead_cis_loss(h[rows], W, b.ids.cpu().numpy()[rows],
                            b.logp_infer.cpu().double().numpy()[rows],
                            b.adv.cpu().double().numpy()[rows], None, prm_ref, keep_grad=True)
    g = torch.Generator().manual_seed(9)
    vs = sorted(set(torch.randint(0, FULL_V, (60,), generator=g).tolist())
                | set(b.ids.cpu().numpy()[rows].tolist()) | {0, FULL_V - 1})
    dW = out["dweight"][vs].cpu().double().numpy()
    G = np.abs(res.grad)
    bound = grad_bound(G[:, vs].T @ np.abs(h[rows]), *dw_group(FULL_CHUNK, FULL_T))
    rep = {"case": "full_size_few_valid", "dweight_rows": check_grad("dweight", dW, res.dW[vs],
                                                                      bound)}
    dh = out["dhidden"].cpu().double().numpy()
    others = np.ones(FULL_T, dtype=bool)
    others[rows] = False
    assert np.all(dh[others] == 0)
    rep["dhidden_rows"] = check_grad("dhidden", dh[rows], res.dhidden,
                                     grad_bound(G @ np.abs(W), FULL_V, 1))
    _dump("full_size_few_valid", rep)
