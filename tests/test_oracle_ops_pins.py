"""Pins of oracle.ops (operator family, sequence operators, decoupled PPO-clip loss and the
training diagnostics) against what the paper and the mathematics fix.

As in test_oracle_pins.py, no check re-types the oracle's formula: each compares it with an
independent computation (50-digit mpmath through Lemma 1's displacement form, scipy's
Bernoulli entropy, brute-force expectations over tiny vocabularies, finite differences of the
objective of Eq. (1)), or with an identity between operators that the paper states (TIS is CIS
with a flat cap; lambda = 0 is TIS with C = 1; the two-sided band lifts the displacement).
``test_oracle_ops_mutants.py`` plants mistakes in oracle.ops and requires that a check fails.
"""

import math

import mpmath as mp
import numpy as np
import pytest
import scipy.stats

import oracle.cis as O
import oracle.ops as X
from tests.test_oracle_pins import mp_logit, mp_softmax, mp_tokens

mp.mp.dps = 50


def lg(x):
    return float(mp.log(x))


def tw(op, p, q, prm):
    """Oracle token weight for mpmath probabilities p, q (training, inference)."""
    return X.token_weight(op, lg(p), lg(q), float(1 - p), prm)


def eps_of(p, q):
    return mp_logit(p) - mp_logit(q)


# ------------------------------------------------------------------------------------------
# Token operators (Table tab:baselines)
# ------------------------------------------------------------------------------------------

def check_tis_is_flat_cis():
    """TIS with cap C equals CIS with kappa = 1 and lambda = C - 1 (phi = 1: a flat cap), TIS
    with C = 1 equals CIS with lambda = 0 (Sec. 4.4), and TIS truncates exactly when
    e^eps > 1 + (C - 1)/(1 - p) (Eq. (5))."""
    rng = np.random.default_rng(31)
    for p, q in mp_tokens(rng, 300, lo=-8, hi=8):
        for C in (1.0, 1.13, 2.0, 5.0):
            w, act = tw(X.OP_TIS, p, q, X.OpParams(op=X.OP_TIS, hi=C))
            wc, tc = O.cis_weight(lg(p), lg(q), float(1 - p), C - 1.0, 1.0)
            assert abs(w - wc) <= 1e-14 * max(1.0, wc) and act == tc, (p, q, C)
            if abs(p / q - C) > 1e-9 * C:
                assert act == bool(mp.e ** eps_of(p, q) > 1 + (C - 1) / (1 - p)), (p, q, C)
        w1, _ = tw(X.OP_TIS, p, q, X.OpParams(op=X.OP_TIS, hi=1.0))
        w0, _ = O.cis_weight(lg(p), lg(q), float(1 - p), 0.0, 5e-3)
        assert abs(w1 - w0) <= 1e-15 * max(1.0, w0)


def check_exact_and_none_calibration():
    """Sampling y ~ q over a tiny vocabulary: the exact ratio is calibrated, sum_y q_y w_y = 1,
    whenever no k_y leaves the clamp; with a clamp that binds, tokens above it weigh exactly
    the TIS weight with C = hi and tokens below it weigh lo. 'No correction' weighs 1."""
    rng = np.random.default_rng(32)
    prm = X.default_params(X.OP_EXACT)
    for V in (2, 4, 7):
        for _ in range(10):
            z = rng.normal(0, 2, size=V)
            d = rng.normal(0, 1, size=V)
            P, Q = mp_softmax(z), mp_softmax(z, d)
            tot = mp.fsum(Q[y] * mp.mpf(tw(X.OP_EXACT, P[y], Q[y], prm)[0]) for y in range(V))
            assert abs(tot - 1) < 1e-13
            assert all(tw(X.OP_NONE, P[y], Q[y], X.OpParams(op=X.OP_NONE)) == (1.0, False)
                       for y in range(V))
    narrow = X.OpParams(op=X.OP_EXACT, lo=0.7, hi=1.4)
    for p, q in mp_tokens(rng, 300, lo=-5, hi=5):
        k = float(p / q)
        w, act = tw(X.OP_EXACT, p, q, narrow)
        if k < 0.7:
            assert w == 0.7 and act
        else:
            wt, at = tw(X.OP_TIS, p, q, X.OpParams(op=X.OP_TIS, hi=1.4))
            assert w == wt and act == at


def check_icepop_band_mass():
    """Sampling y ~ q, the IcePop weight k 1{k in [alpha, beta]} has expectation
    sum_y p_y 1{k_y in band} (since q k = p): the training-side mass of the kept tokens. With an
    unbounded band it is the exact ratio."""
    rng = np.random.default_rng(33)
    for V in (3, 5, 8):
        for _ in range(12):
            z = rng.normal(0, 2, size=V)
            d = rng.normal(0, 1.2, size=V)
            P, Q = mp_softmax(z), mp_softmax(z, d)
            for lo, hi in ((0.5, 5.0), (0.9, 1.1), (0.0, math.inf)):
                prm = X.OpParams(op=X.OP_ICEPOP, lo=lo, hi=hi)
                lhs = mp.fsum(Q[y] * mp.mpf(tw(X.OP_ICEPOP, P[y], Q[y], prm)[0]) for y in range(V))
                kept = [y for y in range(V) if lo <= P[y] / Q[y] <= hi]
                rhs = mp.fsum(P[y] for y in kept)
                if all(abs(P[y] / Q[y] - b) > 1e-9 for y in range(V) for b in (lo, hi)
                       if math.isfinite(b)):
                    assert abs(lhs - rhs) < 1e-13, (V, lo, hi, lhs, rhs)
                    for y in range(V):
                        assert tw(X.OP_ICEPOP, P[y], Q[y], prm)[1] == (y not in kept)


def check_kpop_metric():
    """The binary KL matches scipy's relative entropy of the two Bernoulli distributions, the
    metric takes the larger direction, and App. D.5's saturated tokens behave as stated: equal
    probabilities of one are kept (metric 0), one-sided saturation is finite in float64."""
    rng = np.random.default_rng(34)
    for _ in range(300):
        a, b = rng.uniform(1e-6, 1 - 1e-6, size=2)
        ref = scipy.stats.entropy([a, 1 - a], [b, 1 - b])
        assert abs(X.binary_kl(a, b) - ref) <= 1e-12 * max(1.0, ref)
        m = X.kpop_metric(math.log(a), math.log(b))
        both = max(ref, scipy.stats.entropy([b, 1 - b], [a, 1 - a]))
        assert abs(m - both) <= 1e-12 * max(1.0, both)
        w, act = X.token_weight(X.OP_KPOP, math.log(a), math.log(b), 1 - a, X.OpParams(
            op=X.OP_KPOP, hi=2.0))
        assert act == (both > 2.0) and (w == 0.0 if act else abs(w - a / b) < 1e-12 * a / b)
    assert X.kpop_metric(0.0, 0.0) == 0.0
    sat = X.kpop_metric(0.0, math.log(1e-9))
    e = 1e-8
    ref = scipy.stats.entropy([1 - e, e], [e, 1 - e])
    assert math.isfinite(sat) and abs(sat - ref) <= 1e-9 * ref and sat > 2.0
    assert X.kpop_metric(0.0, math.log(0.9)) < 2.0


def check_two_sided_band():
    """At kappa = 0 the two-sided weight is Lemma 1 applied to the displacement clipped to
    [1/2, 1 + lambda]: p + (1 - p) min{max{e^eps, 1/2}, 1 + lambda} (App. C.1). With a floor it
    is never below (1 + p)/2 and equals the CIS weight wherever e^eps >= 1/2."""
    rng = np.random.default_rng(35)
    for p, q in mp_tokens(rng, 300, lo=-7, hi=7):
        ee = mp.e ** eps_of(p, q)
        for lam in (0.5, 1.7, 2.3):
            w, act = tw(X.OP_TWO_SIDED, p, q, X.OpParams(op=X.OP_TWO_SIDED, lam=lam, kappa=0.0))
            ref = p + (1 - p) * min(max(ee, mp.mpf(0.5)), 1 + mp.mpf(lam))
            assert abs(w - float(ref)) <= 1e-12 * float(ref), (p, q, lam, w, ref)
            if abs(ee - 0.5) > 1e-9 and abs(ee - 1 - lam) > 1e-9:
                assert act == bool(ee < 0.5 or ee > 1 + lam)
            w5, _ = tw(X.OP_TWO_SIDED, p, q, X.OpParams(op=X.OP_TWO_SIDED, lam=lam, kappa=5e-3))
            assert w5 >= float((1 + p) / 2) * (1 - 1e-15)
            if ee >= 0.5 + 1e-9:
                wc, _ = O.cis_weight(lg(p), lg(q), float(1 - p), lam, 5e-3)
                assert abs(w5 - wc) <= 1e-14 * max(1.0, wc)


def check_qfixed_cap():
    """The q-fixed cap sigmoid(logit q + c)/q (c = log(1 + lambda)) truncates exactly when
    eps > c, i.e. the same tokens as CIS at kappa = 0, and its weight is never below CIS's."""
    rng = np.random.default_rng(36)
    for p, q in mp_tokens(rng, 300, lo=-7, hi=7):
        e = eps_of(p, q)
        for lam in (0.5, math.e - 1, 2.3):
            c = mp.log1p(lam)
            w, act = tw(X.OP_QFIXED, p, q, X.OpParams(op=X.OP_QFIXED, lam=lam))
            capq = 1 / (1 + mp.e ** (-(mp_logit(q) + c))) / q
            if abs(e - c) > 1e-9:
                assert act == bool(e > c), (p, q, lam)
                _, tc = O.cis_weight(lg(p), lg(q), float(1 - p), lam, 0.0)
                assert act == tc
            ref = capq if act else p / q
            assert abs(w - float(ref)) <= 1e-12 * float(ref)
            wc, _ = O.cis_weight(lg(p), lg(q), float(1 - p), lam, 0.0)
            assert w >= wc * (1 - 1e-13)


# ------------------------------------------------------------------------------------------
# Sequence operators (Table tab:baselines, Seq-TIS / Seq-MIS)
# ------------------------------------------------------------------------------------------

def _responses(rng, T):
    n = int(rng.integers(1, min(6, T)))
    cuts = sorted(rng.choice(np.arange(1, T), size=n, replace=False).tolist())
    return np.array([0] + cuts + [T])


def check_seq_weights():
    """K is the product of p_t/q_t over a response's valid tokens (50-digit product), every
    valid token of the response carries the same weight and flag, masked tokens carry nothing
    and do not enter K, and one-token responses reduce to the token operators (TIS; IcePop with
    the same band)."""
    rng = np.random.default_rng(37)
    for _ in range(40):
        T = int(rng.integers(2, 14))
        off = _responses(rng, T)
        pq = mp_tokens(rng, T, lo=-3, hi=3)
        lk = np.array([lg(p) - lg(q) for p, q in pq])
        valid = rng.random(T) < 0.8
        lk_masked = lk.copy()
        lk_masked[~valid] += 50.0           # masked tokens' ratios must not matter
        for op, prm in ((X.OP_SEQ_TIS, X.OpParams(op=X.OP_SEQ_TIS, hi=2.0)),
                        (X.OP_SEQ_MIS, X.OpParams(op=X.OP_SEQ_MIS, lo=0.5, hi=2.0))):
            w, act, _ = X.seq_weights(op, lk_masked, valid, off, prm)
            for s in range(len(off) - 1):
                toks = [t for t in range(off[s], off[s + 1]) if valid[t]]
                K = mp.fprod([pq[t][0] / pq[t][1] for t in toks]) if toks else mp.mpf(1)
                if op == X.OP_SEQ_TIS:
                    ref, ra = (2.0, True) if K > 2 else (float(K), False)
                else:
                    keep = 0.5 <= K <= 2
                    ref, ra = (float(K) if keep else 0.0), not keep
                if min(abs(K - 2), abs(K - 0.5)) > 1e-9:
                    for t in toks:
                        assert abs(w[t] - ref) <= 1e-12 * max(1.0, ref) and act[t] == ra
            assert np.all(w[~valid] == 0) and not np.any(act[~valid])
    # one-token responses
    T = 30
    pq = mp_tokens(rng, T, lo=-3, hi=3)
    lk = np.array([lg(p) - lg(q) for p, q in pq])
    off = np.arange(T + 1)
    ones = np.ones(T, dtype=bool)
    w, act, _ = X.seq_weights(X.OP_SEQ_TIS, lk, ones, off, X.OpParams(op=X.OP_SEQ_TIS, hi=2.0))
    w2, act2, _ = X.seq_weights(X.OP_SEQ_MIS, lk, ones, off,
                                X.OpParams(op=X.OP_SEQ_MIS, lo=0.5, hi=2.0))
    for t, (p, q) in enumerate(pq):
        wt, at = tw(X.OP_TIS, p, q, X.OpParams(op=X.OP_TIS, hi=2.0))
        assert abs(w[t] - wt) <= 1e-13 * max(1, wt) and act[t] == at
        wi, ai = tw(X.OP_ICEPOP, p, q, X.OpParams(op=X.OP_ICEPOP, lo=0.5, hi=2.0))
        assert abs(w2[t] - wi) <= 1e-13 * max(1, wi) and act2[t] == ai


# ------------------------------------------------------------------------------------------
# Diagnostics (App. A, D.1, D.5)
# ------------------------------------------------------------------------------------------

def check_displacement():
    """eps = logit p - logit q in 50 digits; Lemma 1 holds with it (k = p + (1 - p) e^eps); at a
    probability of one it takes the stated infinite/limit values."""
    rng = np.random.default_rng(38)
    for p, q in mp_tokens(rng, 300, lo=-12, hi=12):
        e = X.displacement(lg(p), lg(q), float(1 - p))
        ref = eps_of(p, q)
        assert abs(e - float(ref)) <= 1e-10 * max(1.0, abs(float(ref))), (p, q, e, ref)
        k = float(p + (1 - p) * mp.e ** mp.mpf(e))
        assert abs(k - float(p / q)) <= 1e-9 * float(p / q)
    assert X.displacement(0.0, math.log(0.5), 0.0) == math.inf
    assert X.displacement(math.log(0.5), 0.0, 0.5) == -math.inf
    assert X.displacement(0.0, 0.0, 0.0) == 0.0


def check_loss_diagnostics():
    """Over a batch of rows at kappa = 0: the truncated excess sum (k - w) equals
    sum (1 - p)(e^eps - 1 - lambda)_+ (App. B.1, Lemma 'truncation identities'), the acted-on
    count is the number of tokens with eps > log(1 + lambda), and max |log k| is the largest
    |log(p/q)| over valid rows (50-digit references from the logits)."""
    rng = np.random.default_rng(39)
    for V in (3, 6, 11):
        T = 24
        z = rng.normal(0, 2.5, size=(T, V))
        d = rng.normal(0, 1.0, size=(T, V))
        ids = rng.integers(0, V, size=T)
        mask = (rng.random(T) < 0.8).astype(np.uint8)
        mask[0] = 1
        d[0, ids[0]] += 9.0                 # q >> p: the largest |log k| is a negative log k
        P = [mp_softmax(z[t]) for t in range(T)]
        Q = [mp_softmax(z[t], d[t]) for t in range(T)]
        linf = np.array([lg(Q[t][ids[t]]) for t in range(T)])
        adv = rng.normal(0, 1, size=T)
        lam = 1.3
        prm = X.OpParams(op=X.OP_CIS, lam=lam, kappa=0.0, scale=-1.0 / T)
        res = X.cis_ops_loss(z, ids, linf, adv, mask, prm, with_grad=False)
        exc, nact, mx = mp.mpf(0), 0, mp.mpf(0)
        for t in range(T):
            if not mask[t]:
                continue
            p, q = P[t][ids[t]], Q[t][ids[t]]
            e = eps_of(p, q)
            exc += (1 - p) * max(mp.e ** e - 1 - lam, 0)
            nact += int(e > mp.log1p(lam))
            mx = max(mx, abs(mp.log(p / q)))
        assert abs(res.excess - float(exc)) <= 1e-11 * max(1.0, float(exc))
        assert res.n_acted == nact
        assert abs(res.max_abs_logk - float(mx)) <= 1e-12 * max(1.0, float(mx))


# ------------------------------------------------------------------------------------------
# Decoupled PPO-clip path (Eq. (1))
# ------------------------------------------------------------------------------------------

def _ppo_batch(rng, V, T=8):
    z = rng.normal(0, 2.5, size=(T, V))
    ids = rng.integers(0, V, size=T)
    lt = np.array([O.row_log_softmax(z[t], int(ids[t])).logp for t in range(T)])
    # rho = p(theta)/p_old spread over both sides of the clip range [0.8, 1.28]
    rho = np.array([0.5, 0.79, 0.9, 1.0, 1.1, 1.27, 1.3, 2.0])[:T]
    lold = lt - np.log(rho)
    linf = lold - rng.normal(0, 0.7, size=T)
    adv = np.where(np.arange(T) % 2 == 0, 1.3, -0.9)
    return z, ids, lold, linf, adv


def check_ppo_gradient_finite_differences():
    """d/dz of scale * stopgrad(w) * min(rho A, clip(rho) A), rho = softmax(z)_y / p_old, by
    central differences in 50 digits, for both signs of A and rho on both sides of the clip
    range: the oracle's gradient (gate, the factor rho, onehot - softmax) matches."""
    rng = np.random.default_rng(40)
    lo_c, hi_c = 0.8, 1.28
    for V in (3, 8):
        z, ids, lold, linf, adv = _ppo_batch(rng, V)
        for op in (X.OP_CIS, X.OP_TIS, X.OP_ICEPOP):
            prm = X.default_params(op, scale=-0.25)
            res = X.cis_ppo_loss(z, ids, linf, lold, adv, None, prm)
            h = mp.mpf("1e-20")
            for t in range(z.shape[0]):
                y = int(ids[t])
                sw = prm.scale * res.w[t]
                pold = mp.e ** mp.mpf(float(lold[t]))

                def L(zz):
                    r = mp.e ** (zz[y] - mp.log(mp.fsum(mp.e ** v for v in zz))) / pold
                    return sw * min(r * adv[t], min(max(r, lo_c), hi_c) * adv[t])
                zrow = [mp.mpf(float(v)) for v in z[t]]
                r0 = float(mp.e ** (zrow[y] - mp.log(mp.fsum(mp.e ** v for v in zrow))) / pold)
                if min(abs(r0 - lo_c), abs(r0 - hi_c)) < 1e-6:
                    continue
                for j in range(V):
                    zp, zm = list(zrow), list(zrow)
                    zp[j] += h
                    zm[j] -= h
                    fd = float((L(zp) - L(zm)) / (2 * h))
                    assert abs(res.grad[t, j] - fd) <= 1e-12 * max(abs(sw), 1e-300) + 1e-300, \
                        (op, V, t, j, res.grad[t, j], fd)
                assert abs(res.term[t] - float(L(zrow))) <= 1e-12 * max(abs(sw), 1e-300)


def check_ppo_term_consistent_with_gradient():
    """The per-token term, evaluated by the oracle itself at z +- h, differentiates to the
    oracle's gradient (float64 central differences): the loss value and the gradient describe
    the same objective, including where clipping flattens it."""
    rng = np.random.default_rng(41)
    z, ids, lold, linf, adv = _ppo_batch(rng, 5)
    prm = X.default_params(X.OP_CIS, scale=1.0)
    res = X.cis_ppo_loss(z, ids, linf, lold, adv, None, prm)
    h = 1e-6
    for t in range(z.shape[0]):
        if min(abs(res.rho[t] - 0.8), abs(res.rho[t] - 1.28)) < 1e-3:
            continue
        for j in range(z.shape[1]):
            zp, zm = z.copy(), z.copy()
            zp[t, j] += h
            zm[t, j] -= h
            tp = X.cis_ppo_loss(zp, ids, linf, lold, adv, None, prm, with_grad=False,
                                rows=[t]).term[0]
            tm = X.cis_ppo_loss(zm, ids, linf, lold, adv, None, prm, with_grad=False,
                                rows=[t]).term[0]
            assert abs((tp - tm) / (2 * h) - res.grad[t, j]) <= 1e-6 * max(1.0, abs(res.w[t]))


def check_ppo_reduces_to_rho_one():
    """With l_old equal to the current log-probability (rho = 1, the first minibatch) the
    decoupled gradient is the rho = 1 path's gradient, the gate is open for either sign of A,
    the term is scale * w * A, and the weight depends only on (l_old, l_infer), not on the
    logits."""
    rng = np.random.default_rng(42)
    for V in (4, 9):
        T = 10
        z = rng.normal(0, 2, size=(T, V))
        ids = rng.integers(0, V, size=T)
        lt = np.array([O.row_log_softmax(z[t], int(ids[t])).logp for t in range(T)])
        linf = lt - rng.normal(0, 1.0, size=T)
        adv = rng.normal(0, 1, size=T)
        prm = X.default_params(X.OP_CIS, scale=-0.1)
        a = X.cis_ppo_loss(z, ids, linf, lt, adv, None, prm)
        b = X.cis_ops_loss(z, ids, linf, adv, None, prm)
        assert np.all(a.gate) and np.allclose(a.rho, 1.0, rtol=0, atol=1e-15)
        for t in range(T):
            coef = prm.scale * a.w[t] * adv[t]
            assert abs(a.w[t] - b.w[t]) <= 1e-13 * max(1.0, b.w[t])
            assert np.max(np.abs(a.grad[t] - b.grad[t])) <= 1e-13 * max(abs(coef), 1e-300)
            assert abs(a.term[t] - coef) <= 1e-14 * max(abs(coef), 1e-300)
        z2 = z + rng.normal(0, 1, size=z.shape)
        c = X.cis_ppo_loss(z2, ids, linf, lt, adv, None, prm, with_grad=False)
        assert np.array_equal(c.w, a.w) and np.array_equal(c.acted, a.acted)


def check_ppo_sequence_operator_rows():
    """On the decoupled path a sequence operator gives each valid token its response's weight
    (the same values seq_weights gives from l_old - l_infer)."""
    rng = np.random.default_rng(43)
    T, V = 12, 5
    z = rng.normal(0, 2, size=(T, V))
    ids = rng.integers(0, V, size=T)
    lold = np.array([O.row_log_softmax(z[t], int(ids[t])).logp for t in range(T)]) - 0.05
    linf = lold - rng.normal(0, 0.3, size=T)
    adv = rng.normal(0, 1, size=T)
    mask = (rng.random(T) < 0.85).astype(np.uint8)
    off = np.array([0, 3, 4, 9, 12])
    for op in X.SEQ_OPS:
        prm = X.default_params(op, scale=0.5)
        res = X.cis_ppo_loss(z, ids, linf, lold, adv, mask, prm, offsets=off, with_grad=False)
        for s in range(len(off) - 1):
            toks = [t for t in range(off[s], off[s + 1]) if mask[t]]
            K = math.exp(math.fsum(lold[t] - linf[t] for t in toks))
            for t in toks:
                if op == X.OP_SEQ_TIS:
                    assert abs(res.w[t] - min(K, 2.0)) <= 1e-13 * max(1.0, K)
                elif not (abs(K - 0.5) < 1e-9 or abs(K - 2) < 1e-9):
                    assert res.w[t] == (K if 0.5 <= K <= 2 else 0.0) or \
                        abs(res.w[t] - K) <= 1e-13 * K


def check_table_hyperparameters():
    """default_params carries the hyperparameters printed in Table tab:baselines, App. C.1's PPO
    clip and App. D.5's KL clamp (tests/golden/paper_numbers.json); the two-sided floor
    (1 + p)/2 is the lift e^eps >= 1/2 of App. C.1 mapped through Lemma 1."""
    import json
    import os
    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                       "paper_numbers.json")))
    b = gold["baseline_operators"]
    assert (X.default_params(X.OP_EXACT).lo, X.default_params(X.OP_EXACT).hi) == \
        tuple(b["exact_clamp"])
    assert X.default_params(X.OP_TIS).hi == b["tis_cap"]
    ice = X.default_params(X.OP_ICEPOP)
    assert [ice.lo, ice.hi] == b["icepop_band"]
    assert X.default_params(X.OP_KPOP).hi == b["kpop_bound"] and X.KPOP_CLAMP == b["kpop_clamp"]
    assert X.default_params(X.OP_SEQ_TIS).hi == b["seq_tis_cap"]
    mis = X.default_params(X.OP_SEQ_MIS)
    assert [mis.lo, mis.hi] == b["seq_mis_band"]
    for op in range(10):
        prm = X.default_params(op)
        assert [prm.clip_low, prm.clip_high] == gold["ppo_clip"]["value"]
    cis = X.default_params(X.OP_CIS)
    assert (cis.lam, cis.kappa) == (gold["deployed"]["lambda"], gold["deployed"]["kappa"])
    # the floor: a token whose displacement is e^eps = 1/2 exactly sits on the lift
    fl = gold["two_sided_floor"]["value"]
    for p in (0.1, 0.5, 0.9):
        p = mp.mpf(p)
        q = 1 / (1 + mp.e ** (-(mp_logit(p) - mp.log(fl))))
        k = p / q
        assert abs(k - (1 + p) / 2) < 1e-40


CHECKS = [
    check_table_hyperparameters,
    check_tis_is_flat_cis,
    check_exact_and_none_calibration,
    check_icepop_band_mass,
    check_kpop_metric,
    check_two_sided_band,
    check_qfixed_cap,
    check_seq_weights,
    check_displacement,
    check_loss_diagnostics,
    check_ppo_gradient_finite_differences,
    check_ppo_term_consistent_with_gradient,
    check_ppo_reduces_to_rho_one,
    check_ppo_sequence_operator_rows,
]


@pytest.mark.parametrize("check", CHECKS, ids=lambda f: f.__name__)
def test_oracle_ops_pin(check):
    check()
