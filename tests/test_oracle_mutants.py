"""Plant plausible mistakes in the oracle (on the CPU) and require that a pin catches each.

This shows that the pins in test_oracle_pins.py constrain every part of the oracle: a dropped
term, a swapped operand, a wrong index or sign, a wrong reduction. Each mutant replaces one
oracle function for the duration of the test only.
"""

import math

import numpy as np
import pytest

import oracle.cis as O
from tests.test_oracle_pins import CHECKS

_orig_weight = O.cis_weight
_orig_row = O.row_log_softmax
_orig_loss = O.cis_loss


def _weight_mutant(kind):
    def w(lt, li, one_minus_p, lam, kappa):
        delta = (li - lt) if kind == "swapped_logprobs" else (lt - li)
        if math.isnan(delta):
            return math.nan, False
        k = math.inf if delta > 709 else math.exp(delta)
        if kind == "dropped_confidence_factor":
            phi = 1.0
        elif kind == "floor_as_min":
            phi = min(one_minus_p, kappa)
        elif kind == "floor_on_cap":
            phi = one_minus_p
        else:
            phi = max(one_minus_p, kappa)
        cap = 1.0 + lam * phi
        if kind == "floor_on_cap":
            cap = max(cap, 1.0 + kappa)
        if kind == "two_sided_lift":
            p = 1.0 - one_minus_p
            return max(min(k, cap), (1 + p) / 2), k > cap
        if kind == "cap_on_logratio":
            return min(delta, math.log(cap)), delta > math.log(cap)
        tr = k > cap
        return (cap if tr else k), tr
    return w


def _row_mutant(kind):
    def r(z, y):
        rs = _orig_row(z, y)
        z = np.asarray(z, dtype=np.float64)
        if kind == "complement_includes_y":
            rs.one_minus_p = 1.0
        elif kind == "lse_is_max":
            rs.logp = float(z[y]) - rs.m
        elif kind == "gather_off_by_one":
            rs.logp = float(z[(y + 1) % z.shape[0]]) - rs.lse
        elif kind == "complement_by_cancellation":
            rs.one_minus_p = 1.0 - math.exp(rs.logp)
        elif kind == "complement_by_subtraction":
            rs.one_minus_p = (rs.s - math.exp(float(z[y]) - rs.m)) / rs.s if rs.s else math.nan
            rs.one_minus_p = float(np.float32(rs.one_minus_p))
        return rs
    return r


def _loss_mutant(kind):
    def f(logits, ids, logp_infer, adv, mask, lam, kappa, scale, with_grad=True, rows=None):
        if kind == "mask_ignored":
            mask = None
        res = _orig_loss(logits, ids, logp_infer, adv, mask, lam, kappa, scale, with_grad, rows)
        if kind == "gradient_sign" and res.grad is not None:
            res.grad = -res.grad
        if kind == "gradient_without_onehot" and res.grad is not None:
            for i, t in enumerate(range(len(ids)) if rows is None else rows):
                y = int(ids[t])
                if 0 <= y < res.grad.shape[1] and res.flags[i] & O.FLAG_VALID:
                    coef = scale * res.w[i] * adv[t]
                    res.grad[i, y] -= coef
        if kind == "weight_not_applied":
            for i, t in enumerate(range(len(ids)) if rows is None else rows):
                if res.flags[i] & O.FLAG_VALID and res.w[i] != 0:
                    res.term[i] /= res.w[i]
                    if res.grad is not None:
                        res.grad[i] /= res.w[i]
            res.loss = math.fsum(res.term.tolist())
        return res
    return f


MUTANTS = (
    [("cis_weight", k, _weight_mutant(k)) for k in
     ("swapped_logprobs", "dropped_confidence_factor", "floor_as_min", "floor_on_cap",
      "two_sided_lift", "cap_on_logratio")]
    + [("row_log_softmax", k, _row_mutant(k)) for k in
       ("complement_includes_y", "lse_is_max", "gather_off_by_one",
        "complement_by_cancellation", "complement_by_subtraction")]
    + [("cis_loss", k, _loss_mutant(k)) for k in
       ("mask_ignored", "gradient_sign", "gradient_without_onehot", "weight_not_applied")]
)


@pytest.mark.parametrize("target,kind,fn", MUTANTS, ids=[m[1] for m in MUTANTS])
def test_some_pin_catches_mutant(monkeypatch, target, kind, fn):
    monkeypatch.setattr(O, target, fn)
    caught = []
    for check in CHECKS:
        try:
            check()
        except (AssertionError, ValueError, ZeroDivisionError, OverflowError, IndexError) as e:
            caught.append(check.__name__)
    assert caught, f"no pin caught the planted mistake {kind!r}"
