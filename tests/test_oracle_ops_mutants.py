"""Plant plausible mistakes in oracle.ops (on the CPU) and require that a pin catches each.

Each mutant replaces one function of oracle.ops for the duration of the test; the pins of
test_oracle_ops_pins.py must then fail (or raise) somewhere.
"""

import math

import numpy as np
import pytest

import oracle.ops as X
from tests.test_oracle_ops_pins import CHECKS

_tw = X.token_weight
_kl = X.binary_kl
_seq = X.seq_weights
_disp = X.displacement
_gate = X.ppo_gate
_sur = X.ppo_surrogate
_coef = X.ppo_coef
_fin = X._finish


def _token_mutant(kind):
    def f(op, lp, lq, one_minus_p, prm):
        k = math.exp(lp - lq) if lp - lq < 709 else math.inf
        q, omq = math.exp(lq), -math.expm1(lq)
        if kind == "two_sided_floor_minus" and op == X.OP_TWO_SIDED:
            w, tr = _tw(X.OP_CIS, lp, lq, one_minus_p, prm)
            floor = 0.5 * one_minus_p
            return (floor, True) if w < floor else (w, tr)
        if kind in ("qfixed_exp_plus_c", "qfixed_uses_p") and op == X.OP_QFIXED:
            c = math.log1p(prm.lam)
            if kind == "qfixed_uses_p":
                q, omq = 1.0 - one_minus_p, one_minus_p
            capq = 1.0 / (q + omq * math.exp(c if kind == "qfixed_exp_plus_c" else -c))
            return (capq, True) if k > capq else (k, False)
        if kind == "icepop_inverted" and op == X.OP_ICEPOP:
            keep = not (prm.lo <= k <= prm.hi)
            return (k if keep else 0.0), not keep
        if kind == "exact_no_lower_clamp" and op == X.OP_EXACT:
            return min(k, prm.hi), k > prm.hi
        if kind == "tis_inverse_ratio" and op == X.OP_TIS:
            k = 1.0 / k
            return (prm.hi, True) if k > prm.hi else (k, False)
        if kind == "tis_not_truncating" and op == X.OP_TIS:
            return k, False
        return _tw(op, lp, lq, one_minus_p, prm)
    return f


def _kl_no_clamp(a, b):
    return a * math.log(a / b) + (1.0 - a) * math.log((1.0 - a) / (1.0 - b))


def _kpop_one_direction(lp, lq):
    return X.binary_kl(math.exp(lp), math.exp(lq))


def _seq_mutant(kind):
    def f(op, logk, valid, offsets, prm):
        if kind == "seq_includes_masked":
            return _seq(op, logk, np.ones_like(valid, dtype=bool), offsets, prm)
        if kind == "seq_geometric_mean":
            off = np.asarray(offsets)
            lk = np.array(logk, dtype=np.float64)
            for s in range(len(off) - 1):
                n = max(1, int(np.sum(valid[off[s]:off[s + 1]])))
                lk[off[s]:off[s + 1]] /= n
            return _seq(op, lk, valid, offsets, prm)
        return _seq(op, logk, valid, offsets, prm)
    return f


def _disp_mutant(kind):
    def f(lp, lq, one_minus_p):
        if kind == "eps_sign":
            return -_disp(lp, lq, one_minus_p)
        return lp - lq                      # eps_without_complement
    return f


def _gate_mutant(kind):
    def f(rho, A, cl, ch):
        if kind == "gate_same_side":
            return A != 0.0 and rho <= 1.0 + ch
        return A != 0.0                     # gate_always
    return f


def _sur_mutant(kind):
    def f(rho, A, cl, ch):
        clipped = min(max(rho, 1.0 - cl), 1.0 + ch)
        if kind == "surrogate_max":
            return max(rho * A, clipped * A)
        return rho * A                      # surrogate_unclipped
    return f


def _coef_without_rho(sw, A, rho, gate):
    return sw * A if gate else 0.0


def _fin_mutant(kind):
    def f(n, V, sel, logp, w, acted, term, flags, logk, eps, gate, rho, grad):
        r = _fin(n, V, sel, logp, w, acted, term, flags, logk, eps, gate, rho, grad)
        valid = (flags & X.FLAG_VALID) > 0
        if kind == "excess_sign":
            r.excess = -r.excess
        elif kind == "max_logk_signed":
            r.max_abs_logk = float(np.max(logk[valid])) if np.any(valid) else 0.0
        elif kind == "acted_counts_masked":
            r.n_acted = int(np.sum(acted))  + int(np.sum(~valid))
        return r
    return f


MUTANTS = (
    [("token_weight", k, _token_mutant(k)) for k in
     ("two_sided_floor_minus", "qfixed_exp_plus_c", "qfixed_uses_p", "icepop_inverted",
      "exact_no_lower_clamp", "tis_inverse_ratio", "tis_not_truncating")]
    + [("binary_kl", "kl_no_clamp", _kl_no_clamp),
       ("kpop_metric", "kpop_one_direction", _kpop_one_direction)]
    + [("seq_weights", k, _seq_mutant(k)) for k in ("seq_includes_masked", "seq_geometric_mean")]
    + [("displacement", k, _disp_mutant(k)) for k in ("eps_sign", "eps_without_complement")]
    + [("ppo_gate", k, _gate_mutant(k)) for k in ("gate_same_side", "gate_always")]
    + [("ppo_surrogate", k, _sur_mutant(k)) for k in ("surrogate_max", "surrogate_unclipped")]
    + [("ppo_coef", "coef_without_rho", _coef_without_rho)]
    + [("_finish", k, _fin_mutant(k)) for k in
       ("excess_sign", "max_logk_signed", "acted_counts_masked")]
)


@pytest.mark.parametrize("target,kind,fn", MUTANTS, ids=[m[1] for m in MUTANTS])
def test_some_ops_pin_catches_mutant(monkeypatch, target, kind, fn):
    monkeypatch.setattr(X, target, fn)
    caught = []
    for check in CHECKS:
        try:
            check()
        except (AssertionError, ValueError, ZeroDivisionError, OverflowError, IndexError):
            caught.append(check.__name__)
    assert caught, f"no pin caught the planted mistake {kind!r}"
