"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these checks re-types the oracle's own formula: each compares it with an independent
computation (50-digit mpmath from the definitions, torch's float64 log_softmax, finite
differences, brute-force enumeration over tiny vocabularies), with an identity or invariant the
paper proves, or with a number the paper prints (tests/golden/paper_numbers.json).

Every ``check_*`` function raises AssertionError on failure; ``test_oracle_mutants.py`` plants
plausible mistakes in the oracle and requires that some check fails for each.
"""

import json
import math
import os

import mpmath as mp
import numpy as np
import pytest

import oracle.cis as O

mp.mp.dps = 50
HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = json.load(open(os.path.join(HERE, "golden", "paper_numbers.json")))


# ------------------------------------------------------------------------------------------
# independent reference arithmetic (mpmath, straight from the definitions)
# ------------------------------------------------------------------------------------------

def mp_softmax(z, d=None):
    """softmax(z + d) in 50 digits; z and d are added exactly (not in float64)."""
    if d is None:
        d = [0.0] * len(z)
    ez = [mp.e ** (mp.mpf(float(v)) + mp.mpf(float(dv))) for v, dv in zip(z, d)]
    tot = mp.fsum(ez)
    return [v / tot for v in ez]


def mp_logit(p):
    return mp.log(p) - mp.log(1 - p)


def mp_tokens(rng, n, lo=-6.0, hi=6.0):
    """(p, q) pairs as mpmath numbers from log-odds drawn uniformly, plus both log-probs."""
    out = []
    for _ in range(n):
        lp, lq = rng.uniform(lo, hi, size=2)
        p = 1 / (1 + mp.e ** (-mp.mpf(float(lp))))
        q = 1 / (1 + mp.e ** (-mp.mpf(float(lq))))
        out.append((p, q))
    return out


def oracle_w_from_pq(p, q, lam, kappa):
    """Oracle weight for a token whose training/inference probabilities are p, q (mpmath)."""
    ltr = float(mp.log(p))
    linf = float(mp.log(q))
    one_minus_p = float(1 - p)
    return O.cis_weight(ltr, linf, one_minus_p, lam, kappa)


LAMS = [0.0, 0.5, math.expm1(1.0), 2.3, 6.0]
KAPPAS = [0.0, 5e-3, 0.1, 1.0]


# ------------------------------------------------------------------------------------------
# P1/P2/P6: Eq. (4) and Lemma B.2 (eq:app_clipped_ratio, eq:app_clipped_excess)
# ------------------------------------------------------------------------------------------

def check_clipped_ratio_identity():
    """kappa = 0: min{k, 1+lam(1-p)} = p + (1-p) min{e^eps, 1+lam} with eps = logit p - logit q,
    and k - w = (1-p)(e^eps - 1 - lam)_+ (Eq. (4); App. B.1, Lemma 'truncation identities')."""
    rng = np.random.default_rng(11)
    for p, q in mp_tokens(rng, 300):
        eps = mp_logit(p) - mp_logit(q)
        k = p / q
        for lam in LAMS:
            w, tr = oracle_w_from_pq(p, q, lam, 0.0)
            rhs = p + (1 - p) * min(mp.e ** eps, 1 + mp.mpf(lam))
            assert abs(w - float(rhs)) <= 1e-12 * max(1.0, float(rhs)), (p, q, lam, w, rhs)
            excess = (1 - p) * max(mp.e ** eps - 1 - lam, 0)
            assert abs((float(k) - w) - float(excess)) <= 1e-11 * max(1.0, float(k)), \
                (p, q, lam, float(k) - w, excess)
            # truncation happens exactly when the displacement exceeds log(1+lam)
            if abs(eps - mp.log1p(lam)) > 1e-9:
                assert tr == bool(eps > mp.log1p(lam)), (p, q, lam, tr, eps)


def check_untruncated_weight_is_exact_ratio():
    """eps <= log(1+lam) => w = k for every floor kappa (the floor only loosens the cap;
    App. B.4 eq:app_floor_order)."""
    rng = np.random.default_rng(12)
    for p, q in mp_tokens(rng, 300):
        eps = mp_logit(p) - mp_logit(q)
        k = float(p / q)
        for lam in LAMS:
            if eps <= mp.log1p(lam) - 1e-12:
                for kappa in KAPPAS:
                    w, tr = oracle_w_from_pq(p, q, lam, kappa)
                    assert not tr and abs(w - k) <= 1e-13 * max(1.0, k), (p, q, lam, kappa, w, k)


# ------------------------------------------------------------------------------------------
# P3: the closed form sigmoid(logit(q)+c)/q at kappa = 0
# ------------------------------------------------------------------------------------------

def check_closed_form_cap():
    """With c = log(1+lam) the bound on the log-odds displacement, holding q fixed gives the
    ratio bound capq = sigmoid(logit q + c)/q. At kappa = 0 the oracle truncates exactly the
    tokens with k > capq, never returns more than capq, and capq -> 1 as q -> 1; the paper's
    cap 1 + lam(1-p) is nonincreasing in p and -> 1 as p -> 1 (Sec. 3.3, Eq. (4))."""
    rng = np.random.default_rng(13)
    for p, q in mp_tokens(rng, 300):
        k = p / q
        for lam in LAMS[1:]:
            c = mp.log1p(lam)
            capq = 1 / (1 + mp.e ** (-(mp_logit(q) + c))) / q
            w, tr = oracle_w_from_pq(p, q, lam, 0.0)
            if abs(k - capq) > 1e-9 * capq:
                assert tr == bool(k > capq), (p, q, lam)
            assert w <= float(capq) * (1 + 1e-12), (p, q, lam, w, capq)
    for lam in LAMS[1:]:
        c = mp.log1p(lam)
        caps = [1 / (1 + mp.e ** (-(mp_logit(mp.mpf(q)) + c))) / mp.mpf(q)
                for q in (0.9, 0.99, 0.999999)]
        assert caps[0] > caps[1] > caps[2] > 1 and caps[2] - 1 < 1e-4 * lam
        # the paper's cap, evaluated through the oracle with k very large
        prev = math.inf
        for one_minus_p in [0.9, 0.5, 0.1, 1e-2, 1e-4, 1e-8]:
            w, _ = O.cis_weight(math.log1p(-one_minus_p), -700.0, one_minus_p, lam, 0.0)
            assert w <= prev and w >= 1.0
            prev = w
        assert prev - 1.0 < 1e-7 * lam


# ------------------------------------------------------------------------------------------
# P4/P5: one-sidedness and the floor corollary (App. B.1 eq:app_one_sided; App. B.4)
# ------------------------------------------------------------------------------------------

def check_one_sided_and_floor_bounds():
    """w <= k always; w = k whenever k <= 1; eps <= 0 => p < k <= 1; w <= 1 + lam;
    f_lam <= f_{lam,kappa} <= k (Corollary 'Effect of the numerical floor')."""
    rng = np.random.default_rng(14)
    for p, q in mp_tokens(rng, 400, lo=-9, hi=9):
        k = float(p / q)
        eps = mp_logit(p) - mp_logit(q)
        if eps <= 0:
            assert float(p) < k * (1 + 1e-15) and k <= 1 + 1e-15
        for lam in LAMS:
            w0, _ = oracle_w_from_pq(p, q, lam, 0.0)
            for kappa in KAPPAS:
                w, _ = oracle_w_from_pq(p, q, lam, kappa)
                assert w <= k * (1 + 1e-14)
                if k <= 1:
                    assert abs(w - k) <= 1e-13 * k + 1e-300
                assert w <= 1 + lam + 1e-12
                assert w0 <= w * (1 + 1e-14) + 1e-300


# ------------------------------------------------------------------------------------------
# P7: special cases that reduce to other operators
# ------------------------------------------------------------------------------------------

def check_special_cases():
    """lam = 0 is TIS with C = 1 (Sec. 4.4); lam -> inf recovers the exact ratio (Sec. 3.3,
    after Theorem 2); kappa = 1 gives the fixed cap C = 1 + lam; the fixed-cap equivalence
    k <= C <=> e^eps <= 1 + (C-1)/(1-p) (Eq. (5), App. B.1 eq:app_fixed_cap)."""
    rng = np.random.default_rng(15)
    for p, q in mp_tokens(rng, 300, lo=-8, hi=8):
        k = float(p / q)
        w, _ = oracle_w_from_pq(p, q, 0.0, 5e-3)
        assert abs(w - min(k, 1.0)) <= 1e-14 * max(1.0, k)
        w, _ = oracle_w_from_pq(p, q, 1e300, 5e-3)
        assert abs(w - k) <= 1e-13 * k
        for lam in LAMS:
            w, _ = oracle_w_from_pq(p, q, lam, 1.0)
            assert abs(w - min(k, 1 + lam)) <= 1e-13 * max(1.0, k)
        eps = O.log_odds_displacement(float(mp.log(p)), float(mp.log(q)))
        for C in (1.0, 1.13, 2.0, 5.0):
            lhs = k <= C
            rhs = math.exp(eps) <= 1 + (C - 1) / float(1 - p)
            if abs(k - C) > 1e-9 * C:
                assert lhs == rhs, (p, q, C)


# ------------------------------------------------------------------------------------------
# P8: numbers printed in the paper
# ------------------------------------------------------------------------------------------

def check_paper_numbers():
    lam = GOLD["deployed"]["lambda"]
    kappa = GOLD["deployed"]["kappa"]
    # Sec. 4.3: the CIS cap exceeds the TIS cap C = 2 exactly for p < 0.565
    p_star = GOLD["cap_looser_than_tis2_below_p"]["value"]
    lo, hi = 0.0, 1.0
    for _ in range(80):                         # bisection on the oracle's cap
        mid = 0.5 * (lo + hi)
        w, _ = O.cis_weight(math.log(mid), -700.0, 1.0 - mid, lam, kappa)
        if w > 2.0:
            lo = mid
        else:
            hi = mid
    assert round(lo, GOLD["cap_looser_than_tis2_below_p"]["printed_digits"]) == p_star
    # App. D.5: below the floor the cap is 1 + lam*kappa ~ 1.01
    for one_minus_p in (4e-3, 1e-4, 1e-9):
        w, tr = O.cis_weight(math.log1p(-one_minus_p), -700.0, one_minus_p, lam, kappa)
        assert tr and round(w, GOLD["floor_cap"]["printed_digits"]) == GOLD["floor_cap"]["value"]
    # Sec. 3.3: below the floor the displacement threshold is e^eps <= 1 + lam*kappa/(1-p)
    for one_minus_p in (4e-3, 1e-3, 1e-5):
        p = 1 - mp.mpf(one_minus_p)
        bound = 1 + lam * kappa / one_minus_p
        for fac in (0.999, 1.001):
            eps = mp.log(bound * fac)
            q = 1 / (1 + mp.e ** (-(mp_logit(p) - eps)))
            _, tr = oracle_w_from_pq(p, q, lam, kappa)
            assert tr == (fac > 1), (one_minus_p, fac)
    # Sec. 4.4: lam = 0 is TIS with C = 1
    for k_log in (-0.3, 0.0, 0.4, 3.0):
        w, _ = O.cis_weight(-0.5, -0.5 - k_log, 1 - math.exp(-0.5), 0.0, kappa)
        assert abs(w - min(math.exp(k_log), 1.0)) < 1e-15


# ------------------------------------------------------------------------------------------
# P9/P10: brute force over tiny vocabularies (Lemma 1; calibration and unbiasedness)
# ------------------------------------------------------------------------------------------

def check_brute_force_lemma1():
    """For V <= 8 and every sampled y: exp(l_train - l_infer) = p/q = p + (1-p) e^eps with
    eps = -delta_y + log sum_{j!=y} w_j e^{delta_j} (App. B.1 eq:app_eps_def), and the oracle's
    log-odds displacement equals that eps."""
    rng = np.random.default_rng(16)
    for V in (2, 3, 5, 8):
        for _ in range(12):
            z = rng.normal(0, 3, size=V)
            d = rng.normal(0, 1, size=V)
            P = mp_softmax(z)
            Q = mp_softmax(z, d)
            for y in range(V):
                rs = O.row_log_softmax(z, y)
                assert abs(rs.logp - float(mp.log(P[y]))) < 1e-13 * max(1, abs(float(mp.log(P[y]))))
                assert abs(rs.one_minus_p - float(1 - P[y])) < 1e-13 * float(1 - P[y])
                denom = mp.fsum(mp.e ** mp.mpf(float(z[j])) for j in range(V) if j != y)
                eps = -mp.mpf(float(d[y])) + mp.log(mp.fsum(
                    mp.e ** mp.mpf(float(z[j])) / denom * mp.e ** mp.mpf(float(d[j]))
                    for j in range(V) if j != y))
                linf = float(mp.log(Q[y]))
                k_or, _ = O.cis_weight(rs.logp, linf, rs.one_minus_p, 1e300, 0.0)
                k_mp = P[y] / Q[y]
                assert abs(k_or - float(k_mp)) < 1e-12 * float(k_mp)
                assert abs(k_mp - (P[y] + (1 - P[y]) * mp.e ** eps)) < mp.mpf('1e-40') * k_mp
                eps_or = O.log_odds_displacement(rs.logp, linf)
                assert abs(eps_or - float(eps)) < 1e-11 * max(1.0, abs(float(eps)))


def check_brute_force_expectations():
    """Sampling y ~ q: sum_y q_y k_y = 1 (the calibration identity of App. C.4);
    sum_y q_y k_y (e_y - p) = 0 (exact correction is unbiased for the softmax score, Sec. 4.3);
    and at kappa = 0, sum_y q_y (k_y - w_y) = sum_y q_y (1 - p_y)(e^eps_y - 1 - lam)_+."""
    rng = np.random.default_rng(17)
    for V in (2, 4, 7):
        for _ in range(10):
            z = rng.normal(0, 2.5, size=V)
            d = rng.normal(0, 1.5, size=V)
            P = mp_softmax(z)
            Q = mp_softmax(z, d)
            lam = 1.3
            tot = mp.mpf(0)
            score = [mp.mpf(0)] * V
            lhs = mp.mpf(0)
            rhs = mp.mpf(0)
            for y in range(V):
                rs = O.row_log_softmax(z, y)
                linf = float(mp.log(Q[y]))
                k, _ = O.cis_weight(rs.logp, linf, rs.one_minus_p, 1e300, 0.0)
                w, _ = O.cis_weight(rs.logp, linf, rs.one_minus_p, lam, 0.0)
                tot += Q[y] * k
                for j in range(V):
                    score[j] += Q[y] * k * ((1 if j == y else 0) - P[j])
                lhs += Q[y] * (k - w)
                eps = mp_logit(P[y]) - mp_logit(Q[y])
                rhs += Q[y] * (1 - P[y]) * max(mp.e ** eps - 1 - lam, 0)
            assert abs(tot - 1) < 1e-13
            assert max(abs(s) for s in score) < 1e-13
            assert abs(lhs - rhs) < 1e-12


# ------------------------------------------------------------------------------------------
# P11: the gradient, by finite differences with the weight frozen (stop-gradient)
# ------------------------------------------------------------------------------------------

def check_gradient_finite_differences():
    """d/dz of scale * stopgrad(w) * A * log softmax(z)_y, by central differences in 50-digit
    arithmetic; rows of the gradient sum to zero; g_y = coef (1 - p_y), g_j = -coef p_j."""
    rng = np.random.default_rng(18)
    for V in (3, 8, 16):
        T = 4
        z = rng.normal(0, 3, size=(T, V))
        ids = rng.integers(0, V, size=T)
        linf = rng.normal(-1.5, 1.0, size=T)
        adv = rng.normal(0, 1, size=T)
        scale = -1.0 / T
        lam, kappa = 1.7, 5e-3
        res = O.cis_loss(z, ids, linf, adv, None, lam, kappa, scale, with_grad=True)
        h = mp.mpf("1e-20")
        for t in range(T):
            y = int(ids[t])
            coef = scale * res.w[t] * adv[t]

            def L(zz):
                return coef * (mp.mpf(float(zz[y]) if not isinstance(zz[y], mp.mpf) else zz[y])
                               - mp.log(mp.fsum(mp.e ** v for v in zz)))
            zrow = [mp.mpf(float(v)) for v in z[t]]
            for j in range(V):
                zp = list(zrow)
                zm = list(zrow)
                zp[j] += h
                zm[j] -= h
                fd = (L(zp) - L(zm)) / (2 * h)
                assert abs(res.grad[t, j] - float(fd)) <= 1e-13 * max(abs(coef), 1e-300) + 1e-300, \
                    (V, t, j, res.grad[t, j], fd)
            assert abs(math.fsum(res.grad[t])) <= 1e-15 * max(1.0, abs(coef))
            # the loss term itself: coef * log p_y
            lp = float(zrow[y] - mp.log(mp.fsum(mp.e ** v for v in zrow)))
            assert abs(res.term[t] - coef * lp) <= 1e-14 * abs(coef * lp) + 1e-300


# ------------------------------------------------------------------------------------------
# P12: log-softmax equals an independent library routine
# ------------------------------------------------------------------------------------------

def check_log_softmax_library():
    import torch
    rng = np.random.default_rng(19)
    for V in (1, 2, 1000, 151936):
        z = rng.normal(0, 3, size=V)
        if V > 10:
            z[:: 97] -= 40.0
        ref = torch.log_softmax(torch.from_numpy(z), dim=0).numpy()
        for y in {0, V - 1, V // 2, int(np.argmax(z))}:
            rs = O.row_log_softmax(z, y)
            assert abs(rs.logp - ref[y]) <= 1e-12 * max(1.0, abs(ref[y]))
            if V > 1:
                exact_comp = -math.expm1(float(ref[y])) if ref[y] < -1e-3 else None
                if exact_comp is not None:
                    assert abs(rs.one_minus_p - exact_comp) <= 1e-11 * exact_comp


def check_complement_mass_near_one():
    """1 - p keeps relative accuracy when p -> 1 (where 1 - exp(log p) would cancel)."""
    V = 50
    for gap in (20.0, 30.0, 35.0):
        z = np.zeros(V)
        z[3] = gap
        rs = O.row_log_softmax(z, 3)
        exact = (V - 1) * mp.e ** (-gap) / (1 + (V - 1) * mp.e ** (-gap))
        assert abs(rs.one_minus_p - float(exact)) <= 1e-14 * float(exact)


# ------------------------------------------------------------------------------------------
# P13: a toy row, end to end, against 50-digit arithmetic
# ------------------------------------------------------------------------------------------

def check_toy_row():
    z = [2.0, -1.0, 0.5, 0.0]
    y, linf, A, scale = 0, -0.9, 1.0, -1.0
    lam, kappa = math.e - 1, 0.0
    res = O.cis_loss(np.array([z]), np.array([y]), np.array([linf]), np.array([A]), None,
                     lam, kappa, scale)
    P = mp_softmax(z)
    k = P[y] / mp.e ** mp.mpf(linf)
    cap = 1 + mp.mpf(lam) * (1 - P[y])
    w = min(k, cap)
    assert k > cap and bool(res.trunc[0])
    assert abs(res.logp_train[0] - float(mp.log(P[y]))) < 1e-15
    assert abs(res.w[0] - float(w)) < 1e-15
    coef = scale * w * A
    assert abs(res.loss - float(coef * mp.log(P[y]))) < 1e-15
    g = [-coef * P[j] for j in range(4)]
    g[y] = coef * (1 - P[y])
    assert np.max(np.abs(res.grad[0] - np.array([float(v) for v in g]))) < 1e-15


def check_masks_and_invalid_ids():
    rng = np.random.default_rng(20)
    T, V = 6, 5
    z = rng.normal(size=(T, V))
    ids = np.array([0, 4, 5, -1, 2, 3])
    mask = np.array([1, 1, 1, 1, 0, 1], dtype=np.uint8)
    res = O.cis_loss(z, ids, np.full(T, -1.0), np.ones(T), mask, 1.0, 5e-3, -1.0)
    assert list(res.flags & O.FLAG_VALID) == [1, 1, 0, 0, 0, 1]
    assert list((res.flags & O.FLAG_BAD_ID) > 0) == [False, False, True, True, False, False]
    for t in (2, 3, 4):
        assert res.w[t] == 0 and res.term[t] == 0 and not res.grad[t].any()


CHECKS = [
    check_clipped_ratio_identity,
    check_untruncated_weight_is_exact_ratio,
    check_closed_form_cap,
    check_one_sided_and_floor_bounds,
    check_special_cases,
    check_paper_numbers,
    check_brute_force_lemma1,
    check_brute_force_expectations,
    check_gradient_finite_differences,
    check_log_softmax_library,
    check_complement_mass_near_one,
    check_toy_row,
    check_masks_and_invalid_ids,
]


@pytest.mark.parametrize("check", CHECKS, ids=[c.__name__ for c in CHECKS])
def test_oracle_pin(check):
    check()


def test_cis_weights_array_form_matches_row_form():
    """Algorithm 1 on arrays (p from the given log-probability) against the row form."""
    rng = np.random.default_rng(21)
    n = 500
    lt = -np.abs(rng.normal(0, 2, n)) * rng.choice([1e-9, 1e-4, 1, 3], n)
    li = lt - rng.normal(0, 1.0, n)
    mask = rng.random(n) > 0.2
    w, tr = O.cis_weights(lt, li, mask, 2.3, 5e-3)
    for i in range(n):
        if not mask[i]:
            assert w[i] == 0 and not tr[i]
            continue
        p = mp.e ** mp.mpf(float(lt[i]))
        k = mp.e ** (mp.mpf(float(lt[i])) - mp.mpf(float(li[i])))
        cap = 1 + mp.mpf(2.3) * max(1 - p, mp.mpf(5e-3))
        assert abs(w[i] - float(min(k, cap))) <= 1e-14 * float(min(k, cap))
