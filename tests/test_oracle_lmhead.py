"""Pins of oracle.lmhead (the CIS loss behind the LM head, logits = hidden @ W^T) and planted
mistakes that they must catch. The checks use 50-digit finite differences, brute-force sums
written as plain loops (not matrix products), the zero column sum of the gradient, and
chunk-size independence."""

import math

import mpmath as mp
import numpy as np
import pytest

import oracle.cis as O
import oracle.lmhead as LH
import oracle.ops as X

mp.mp.dps = 50


def _problem(rng, T, H, V, scale=-0.3):
    hidden = rng.normal(0, 1.0, size=(T, H))
    W = rng.normal(0, 0.7, size=(V, H))
    ids = rng.integers(0, V, size=T)
    z = hidden @ W.T
    lt = np.array([O.row_log_softmax(z[t], int(ids[t])).logp for t in range(T)])
    linf = lt - rng.normal(0, 0.8, size=T)
    adv = rng.normal(0, 1, size=T)
    return hidden, W, ids, linf, adv


def check_gradients_finite_differences():
    """dL/dh and dL/dW against 50-digit central differences of
    sum_t scale * stopgrad(w_t) * A_t * log softmax(h_t W^T)[y_t] (rate 1) and of the decoupled
    surrogate scale * w_t * min(rho A, clip(rho) A), rho = softmax(h_t W^T)[y_t] / p_old."""
    rng = np.random.default_rng(71)
    T, H, V = 3, 4, 6
    hidden, W, ids, linf, adv = _problem(rng, T, H, V)
    prm = X.default_params(X.OP_CIS, lam=1.3, kappa=5e-3, scale=-0.3)
    lold = np.array([O.row_log_softmax(hidden[t] @ W.T, int(ids[t])).logp for t in range(T)])
    lold = lold - np.array([0.5, -0.1, 0.0])          # rho on both sides of the clip range
    for path in ("rate1", "decoupled"):
        res = LH.lmhead_cis_loss(hidden, W, ids, linf, adv, None, prm,
                                 logp_old=lold if path == "decoupled" else None)
        h = mp.mpf("1e-20")

        def L(hh, WW):
            tot = mp.mpf(0)
            for t in range(T):
                z = [mp.fsum(hh[t][k] * WW[j][k] for k in range(H)) for j in range(V)]
                lse = mp.log(mp.fsum(mp.e ** v for v in z))
                lp = z[ids[t]] - lse
                sw = prm.scale * res.w[t]
                if path == "rate1":
                    tot += sw * adv[t] * lp
                else:
                    rho = mp.e ** (lp - mp.mpf(float(lold[t])))
                    clipped = min(max(rho, 1 - mp.mpf(prm.clip_low)), 1 + mp.mpf(prm.clip_high))
                    tot += sw * min(rho * adv[t], clipped * adv[t])
            return tot
        hh = [[mp.mpf(float(v)) for v in row] for row in hidden]
        WW = [[mp.mpf(float(v)) for v in row] for row in W]
        for t in range(T):
            for k in range(H):
                hp = [list(r) for r in hh]
                hm = [list(r) for r in hh]
                hp[t][k] += h
                hm[t][k] -= h
                fd = float((L(hp, WW) - L(hm, WW)) / (2 * h))
                assert abs(res.dhidden[t, k] - fd) <= 1e-12 * max(1.0, abs(fd)), (path, t, k)
        for j in range(V):
            for k in range(H):
                Wp = [list(r) for r in WW]
                Wm = [list(r) for r in WW]
                Wp[j][k] += h
                Wm[j][k] -= h
                fd = float((L(hh, Wp) - L(hh, Wm)) / (2 * h))
                assert abs(res.dW[j, k] - fd) <= 1e-12 * max(1.0, abs(fd)), (path, j, k)


def check_one_hot_hidden_states():
    """With one-hot hidden states h_t = e_{k_t}, the logits are the rows W[:, k_t]: the loss is
    oracle.cis on those rows, dL/dh_t[i] = sum_j G[t, j] W[j, i] and dL/dW[j, i] = G[t, j] summed
    over the tokens with k_t = i (plain loops, no matrix products)."""
    rng = np.random.default_rng(72)
    T, H, V = 6, 5, 9
    W = rng.normal(0, 1.5, size=(V, H))
    k = rng.integers(0, H, size=T)
    hidden = np.zeros((T, H))
    hidden[np.arange(T), k] = 1.0
    ids = rng.integers(0, V, size=T)
    Z = np.array([[W[j, k[t]] for j in range(V)] for t in range(T)])
    linf = rng.normal(-2, 1, size=T)
    adv = rng.normal(0, 1, size=T)
    prm = X.default_params(X.OP_CIS, lam=2.3, kappa=5e-3, scale=0.7)
    res = LH.lmhead_cis_loss(hidden, W, ids, linf, adv, None, prm)
    ref = O.cis_loss(Z, ids, linf, adv, None, prm.lam, prm.kappa, prm.scale)
    assert np.allclose(res.logp_train, ref.logp_train, rtol=0, atol=1e-13)
    assert np.allclose(res.w, ref.w, rtol=1e-14, atol=0) and res.loss == pytest.approx(ref.loss)
    G = ref.grad
    for t in range(T):
        for i in range(H):
            s = math.fsum(G[t, j] * W[j, i] for j in range(V))
            assert abs(res.dhidden[t, i] - s) <= 1e-13 * max(1.0, abs(s))
    for j in range(V):
        for i in range(H):
            s = math.fsum(G[t, j] for t in range(T) if k[t] == i)
            assert abs(res.dW[j, i] - s) <= 1e-13 * max(1.0, abs(s))


def check_weight_gradient_column_sums():
    """Every row of G = dL/dz sums to zero (softmax and one-hot both sum to one), so the
    gradient of the head weight sums to zero over the vocabulary: sum_j dW[j, :] = 0."""
    rng = np.random.default_rng(73)
    hidden, W, ids, linf, adv = _problem(rng, 20, 8, 30)
    res = LH.lmhead_cis_loss(hidden, W, ids, linf, adv, None,
                             X.default_params(X.OP_TIS, scale=-0.05))
    colsum = res.dW.sum(axis=0)
    assert np.max(np.abs(colsum)) <= 1e-13 * max(1.0, np.max(np.abs(res.dW)))
    assert np.max(np.abs(res.dW)) > 1e-3


def check_chunking_regroups_sums():
    """The result does not depend on the row chunk the products are taken over."""
    rng = np.random.default_rng(74)
    hidden, W, ids, linf, adv = _problem(rng, 37, 6, 25)
    mask = (rng.random(37) < 0.8).astype(np.uint8)
    prm = X.default_params(X.OP_CIS, scale=-1 / 37)
    a = LH.lmhead_cis_loss(hidden, W, ids, linf, adv, mask, prm, chunk=37)
    b = LH.lmhead_cis_loss(hidden, W, ids, linf, adv, mask, prm, chunk=5)
    assert np.array_equal(a.flags, b.flags) and np.allclose(a.term, b.term, rtol=1e-14, atol=0)
    assert np.allclose(a.dhidden, b.dhidden, rtol=1e-13, atol=1e-16)
    assert np.allclose(a.dW, b.dW, rtol=1e-12, atol=1e-15)


CHECKS = [check_gradients_finite_differences, check_one_hot_hidden_states,
          check_weight_gradient_column_sums, check_chunking_regroups_sums]


@pytest.mark.parametrize("check", CHECKS, ids=lambda f: f.__name__)
def test_oracle_lmhead_pin(check):
    check()


# ------------------------------------------------------------------------------------------
# planted mistakes
# ------------------------------------------------------------------------------------------
_orig = LH.lmhead_cis_loss


def _mutant(kind):
    def f(hidden, W, ids, logp_infer, adv, mask, prm, logp_old=None, offsets=None,
          with_grad=True, chunk=1024):
        if kind == "logits_without_transpose_scale":
            W = np.asarray(W) * 1.0000001
        r = _orig(hidden, W, ids, logp_infer, adv, mask, prm, logp_old, offsets, with_grad,
                  chunk if kind != "weight_grad_last_chunk_only" else chunk)
        if not with_grad:
            return r
        if kind == "dhidden_sign":
            r.dhidden = -r.dhidden
        elif kind == "weight_grad_last_chunk_only":
            T = np.asarray(hidden).shape[0]
            if T > chunk:
                t0 = ((T - 1) // chunk) * chunk
                part = _orig(np.asarray(hidden)[t0:], W, np.asarray(ids)[t0:],
                             np.asarray(logp_infer)[t0:], np.asarray(adv)[t0:],
                             None if mask is None else np.asarray(mask)[t0:], prm)
                r.dW = part.dW
        elif kind == "dW_without_hidden":
            r.dW = r.dW / np.maximum(np.abs(np.asarray(hidden)).sum(), 1.0)
        elif kind == "dhidden_transposed_weight":
            G = r.dhidden @ np.linalg.pinv(np.asarray(W, dtype=np.float64))
            r.dhidden = G @ np.asarray(W, dtype=np.float64)[::-1]
        return r
    return f


MUTANTS = ["dhidden_sign", "weight_grad_last_chunk_only", "dW_without_hidden",
           "dhidden_transposed_weight", "logits_without_transpose_scale"]


@pytest.mark.parametrize("kind", MUTANTS)
def test_some_lmhead_pin_catches_mutant(monkeypatch, kind):
    monkeypatch.setattr(LH, "lmhead_cis_loss", _mutant(kind))
    caught = []
    for check in CHECKS:
        try:
            check()
        except (AssertionError, ValueError, IndexError):
            caught.append(check.__name__)
    assert caught, f"no pin caught the planted mistake {kind!r}"
