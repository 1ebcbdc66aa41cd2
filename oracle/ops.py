"""Plain float64 CPU oracle for the operator family, the decoupled PPO-clip loss and the
training diagnostics around the CIS token loss.

TEST INFRASTRUCTURE ONLY (like ``oracle.cis``): only the test suite, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py`` may import it; the HIP library shares nothing with it.

What it restates (arXiv 2609.32444):

* Sec. 2.1, Eq. (1) (``eq:objective``): the token objective k_t * min(rho_t A_t, clip(rho_t) A_t)
  with the update ratio rho_t = pi_train(y_t; theta) / p_t, where p_t is the training-side
  probability at the rollout snapshot theta_old, q_t the inference-side one, k_t = p_t / q_t, and
  clip restricting rho to [1 - c_low, 1 + c_high]. App. C.1 "Recipe": c_low = 0.2, c_high = 0.28.
* App. C.1 "Operators" and Table ``tab:baselines``: the weight that each arm puts on the token
  loss, detached from the gradient:
    none            1
    exact ratio     k, clamped to [1e-6, 1e6]
    TIS             min(k, C), C = 2
    IcePop          k * 1{alpha <= k <= beta}, [alpha, beta] = [0.5, 5]
    KPop-dagger     k * 1{max(KL_B(p||q), KL_B(q||p)) <= phi}, float64, phi = 2
    Seq-TIS         min(K, C) on every token of a response, K = prod_t k_t, C = 2
    Seq-MIS         K * 1{alpha <= K <= beta} on every token of a response, [0.5, 2]
    CIS             min{k, 1 + lambda * max(1 - p, kappa)} (Algorithm 1)
* App. C.1 "Operators", two-sided band (ablation table): the displacement is also lifted from
  below to e^eps >= 1/2, which by Lemma 1 (k = p + (1 - p) e^eps) gives the weight
  max{min{k, 1 + lambda*phi}, (1 + p)/2}.
* App. D.5 "The KL mask and probability saturation": KL_B(p||q) = p log(p/q) +
  (1-p) log((1-p)/(1-q)), both directions, p and q clamped to [1e-8, 1 - 1e-8], in float64.
* The q-fixed cap: holding q fixed instead of p, a displacement threshold eps <= c maps through
  Lemma 1 to k <= 1 / (q + (1 - q) e^{-c}); here c = log(1 + lambda), so at kappa = 0 it truncates
  exactly the tokens that CIS truncates.
* App. D.1 (training statistics table and dynamics figure) and App. D.5: the diagnostics
  "fraction of tokens acted on" (whole responses for Seq-TIS/Seq-MIS), "largest |log k_t| in the
  batch", the truncated excess sum_t (k_t - f_t), and the per-token displacement
  eps_t = logit p_t - logit q_t computed from the two log-probabilities (App. A).

Readings where the paper is silent (each is a parameter of the tests, not hidden here):

* "Acted on" means the operator changed the token's weight: truncated (CIS, TIS, exact above
  its upper clamp, q-fixed, Seq-TIS), masked (IcePop, KPop, Seq-MIS), clamped from below
  (exact), or lifted (two-sided band).
* Band and clamp edges are inclusive (a token with k = beta is kept), caps are strict (k = C is
  not truncated), matching the strict CIS truncation flag of ``oracle.cis``.
* The truncated excess is sum over valid tokens of (k_t - w_t), accumulated in float64. For the
  masking operators this is the masked weight; for the two-sided band it includes the (negative)
  lift.
* eps_t is +inf when only p_t = 1, -inf when only q_t = 1, and log k_t when both are 1 (the
  log(1-p) - log(1-q) part is taken as 0 when 1-p == 1-q).
* The decoupled path's gradient follows PPO's min: it flows through rho*A where that term is the
  smaller one (A > 0: rho <= 1 + c_high; A < 0: rho >= 1 - c_low; ties count as unclipped) and is
  zero elsewhere. Its loss value is scale * w * min(rho A, clip(rho) A).
* In the decoupled path p_t comes from the given log-probability at theta_old, and 1 - p_t is
  -expm1(l_old). In the rho = 1 path p_t comes from the same logits (complement mass), as in
  ``oracle.cis``.
* Sequence operators need every token's k before any gradient, so they are defined on the
  decoupled path only (k_t from the two recorded log-probabilities); a response is the token
  range [off[s], off[s+1]) of CSR offsets, and only its valid tokens enter K.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

from .cis import FLAG_BAD_ID, FLAG_NONFINITE, FLAG_TRUNC, FLAG_VALID, cis_weight, row_log_softmax

__all__ = [
    "OP_CIS", "OP_NONE", "OP_EXACT", "OP_TIS", "OP_ICEPOP", "OP_KPOP", "OP_TWO_SIDED",
    "OP_QFIXED", "OP_SEQ_TIS", "OP_SEQ_MIS", "SEQ_OPS", "OpParams", "default_params",
    "binary_kl", "kpop_metric", "token_weight", "seq_weights", "displacement",
    "ppo_surrogate", "ppo_gate", "ppo_coef", "OpsResult", "cis_ops_loss", "cis_ppo_loss",
]

OP_CIS, OP_NONE, OP_EXACT, OP_TIS, OP_ICEPOP, OP_KPOP, OP_TWO_SIDED, OP_QFIXED, OP_SEQ_TIS, \
    OP_SEQ_MIS = range(10)
SEQ_OPS = (OP_SEQ_TIS, OP_SEQ_MIS)

KPOP_CLAMP = 1e-8


@dataclass
class OpParams:
    """Operator and loss parameters. ``lo``/``hi`` are the exact-ratio clamp, the TIS/Seq-TIS cap
    (hi), the IcePop/Seq-MIS band, or the KPop bound phi (hi), depending on ``op``."""
    op: int = OP_CIS
    lam: float = 2.3
    kappa: float = 5e-3
    lo: float = 0.0
    hi: float = math.inf
    clip_low: float = 0.2
    clip_high: float = 0.28
    scale: float = 1.0


def default_params(op: int, **kw) -> OpParams:
    """The hyperparameters of Table ``tab:baselines`` (and App. C.1's PPO clip) for ``op``."""
    base = {
        OP_CIS: dict(lam=2.3, kappa=5e-3),
        OP_NONE: dict(),
        OP_EXACT: dict(lo=1e-6, hi=1e6),
        OP_TIS: dict(hi=2.0),
        OP_ICEPOP: dict(lo=0.5, hi=5.0),
        OP_KPOP: dict(hi=2.0),
        OP_TWO_SIDED: dict(lam=2.3, kappa=5e-3),
        OP_QFIXED: dict(lam=2.3),
        OP_SEQ_TIS: dict(hi=2.0),
        OP_SEQ_MIS: dict(lo=0.5, hi=2.0),
    }[op]
    base.update(kw)
    return OpParams(op=op, **base)


def _exp(x: float) -> float:
    if math.isnan(x):
        return math.nan
    return math.inf if x > 709.0 else math.exp(x)


# --------------------------------------------------------------------------------------------
# KPop-dagger's metric (App. D.5)
# --------------------------------------------------------------------------------------------

def binary_kl(a: float, b: float) -> float:
    """KL(Bern(a) || Bern(b)) in float64 with both probabilities clamped to [1e-8, 1 - 1e-8]."""
    a = min(max(a, KPOP_CLAMP), 1.0 - KPOP_CLAMP)
    b = min(max(b, KPOP_CLAMP), 1.0 - KPOP_CLAMP)
    return a * math.log(a / b) + (1.0 - a) * math.log((1.0 - a) / (1.0 - b))


def kpop_metric(logp_p: float, logp_q: float) -> float:
    """max(KL_B(p||q), KL_B(q||p)) with p = e^{l_p}, q = e^{l_q}; a NaN input gives 0."""
    p, q = _exp(logp_p), _exp(logp_q)
    if math.isnan(p) or math.isnan(q):
        return 0.0
    return max(binary_kl(p, q), binary_kl(q, p))


# --------------------------------------------------------------------------------------------
# Token-level operators (Table tab:baselines, App. C.1)
# --------------------------------------------------------------------------------------------

def token_weight(op: int, logp_p: float, logp_q: float, one_minus_p: float,
                 prm: OpParams) -> tuple[float, bool]:
    """(w, acted) of a token-level operator from the training-side log-probability l_p (with
    its complement 1 - p) and the inference-side log-probability l_q."""
    if op in SEQ_OPS:
        raise ValueError("sequence operators act on whole responses (seq_weights)")
    logk = logp_p - logp_q
    k = _exp(logk)
    if op == OP_CIS:
        return cis_weight(logp_p, logp_q, one_minus_p, prm.lam, prm.kappa)
    if op == OP_NONE:
        return 1.0, False
    if math.isnan(k):
        return math.nan, False
    if op == OP_EXACT:
        return min(max(k, prm.lo), prm.hi), (k < prm.lo or k > prm.hi)
    if op == OP_TIS:
        return (prm.hi, True) if k > prm.hi else (k, False)
    if op == OP_ICEPOP:
        keep = prm.lo <= k <= prm.hi
        return (k if keep else 0.0), not keep
    if op == OP_KPOP:
        keep = kpop_metric(logp_p, logp_q) <= prm.hi
        return (k if keep else 0.0), not keep
    if op == OP_TWO_SIDED:
        w, tr = cis_weight(logp_p, logp_q, one_minus_p, prm.lam, prm.kappa)
        floor = 1.0 - 0.5 * one_minus_p          # (1 + p) / 2
        return (floor, True) if w < floor else (w, tr)
    if op == OP_QFIXED:
        c = math.log1p(prm.lam)
        q, one_minus_q = _exp(logp_q), -math.expm1(logp_q)
        capq = 1.0 / (q + one_minus_q * math.exp(-c))
        return (capq, True) if k > capq else (k, False)
    raise ValueError(f"unknown operator {op}")


def seq_weights(op: int, logk: np.ndarray, valid: np.ndarray, offsets: np.ndarray,
                prm: OpParams) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Seq-TIS / Seq-MIS over the responses [off[s], off[s+1]): (w [T], acted [T], logK [S]).

    log K_s is the float64 sum (math.fsum) of log k_t over the response's valid tokens; every
    valid token of response s gets the response's weight and flag, invalid tokens get 0/False.
    """
    if op not in SEQ_OPS:
        raise ValueError("not a sequence operator")
    off = np.asarray(offsets, dtype=np.int64)
    T = logk.shape[0]
    if off[0] != 0 or off[-1] != T or np.any(np.diff(off) < 0):
        raise ValueError("offsets must rise from 0 to T")
    w = np.zeros(T)
    acted = np.zeros(T, dtype=bool)
    logK = np.zeros(off.shape[0] - 1)
    for s in range(off.shape[0] - 1):
        a, b = int(off[s]), int(off[s + 1])
        idx = [t for t in range(a, b) if valid[t]]
        lk = math.fsum(float(logk[t]) for t in idx) if idx else 0.0
        logK[s] = lk
        K = _exp(lk)
        if op == OP_SEQ_TIS:
            ws, act = (prm.hi, True) if K > prm.hi else (K, False)
        else:
            keep = prm.lo <= K <= prm.hi
            ws, act = (K if keep else 0.0), not keep
        for t in idx:
            w[t] = ws
            acted[t] = act
    return w, acted, logK


# --------------------------------------------------------------------------------------------
# Diagnostics (App. A, D.1, D.5)
# --------------------------------------------------------------------------------------------

def displacement(logp_p: float, logp_q: float, one_minus_p: float) -> float:
    """eps = logit p - logit q = (l_p - l_q) - (log(1 - p) - log(1 - q)), with the conventions
    of the module docstring when a probability is 1."""
    one_minus_q = -math.expm1(logp_q)
    logk = logp_p - logp_q
    if one_minus_p == one_minus_q:
        return logk
    if one_minus_p <= 0.0:
        return math.inf
    if one_minus_q <= 0.0:
        return -math.inf
    return logk - (math.log(one_minus_p) - math.log(one_minus_q))


@dataclass
class OpsResult:
    logp_train: np.ndarray   # [n] float64 (0 on invalid rows)
    w: np.ndarray            # [n] weight on the token loss (0 on invalid rows)
    acted: np.ndarray        # [n] bool
    term: np.ndarray         # [n] float64 per-token loss
    flags: np.ndarray        # [n] uint8 FLAG_* bits (FLAG_TRUNC = acted)
    logk: np.ndarray         # [n] log k_t (0 on invalid rows)
    eps: np.ndarray          # [n] displacement (0 on invalid rows)
    gate: np.ndarray         # [n] bool: the gradient flows (decoupled path; valid rows)
    rho: np.ndarray          # [n] update ratio (1 on the rho = 1 path)
    loss: float              # fsum of term
    n_acted: int
    max_abs_logk: float      # over valid rows (0 when there are none)
    excess: float            # fsum over valid rows of (k - w)
    grad: np.ndarray | None  # [n, V] or None
    diag: dict = field(default_factory=dict)


# --------------------------------------------------------------------------------------------
# PPO clipping of the update ratio (Eq. (1); App. C.1 "Recipe")
# --------------------------------------------------------------------------------------------

def ppo_surrogate(rho: float, A: float, clip_low: float, clip_high: float) -> float:
    """min(rho A, clip(rho) A) with clip(rho) = min(max(rho, 1 - c_low), 1 + c_high)."""
    clipped = min(max(rho, 1.0 - clip_low), 1.0 + clip_high)
    return min(rho * A, clipped * A)


def ppo_gate(rho: float, A: float, clip_low: float, clip_high: float) -> bool:
    """Whether d/drho of the surrogate is A (the unclipped branch is the minimum) rather than 0."""
    return (A > 0.0 and rho <= 1.0 + clip_high) or (A < 0.0 and rho >= 1.0 - clip_low)


def ppo_coef(scale_w: float, A: float, rho: float, gate: bool) -> float:
    """Coefficient of (onehot - softmax) in the gradient: scale*w*A*rho where the gate is on."""
    return scale_w * A * rho if gate else 0.0


def _finish(n, V, sel, logp, w, acted, term, flags, logk, eps, gate, rho, grad) -> OpsResult:
    valid = (flags & FLAG_VALID) > 0
    loss = math.fsum(term.tolist()) if np.all(np.isfinite(term)) else float(np.sum(term))
    n_acted = int(np.sum(acted & valid))
    lk = np.abs(logk[valid])
    max_abs = float(np.max(lk)) if lk.size else 0.0
    ks = [(_exp(float(logk[i])) - float(w[i])) for i in range(n) if valid[i]]
    excess = math.fsum(ks) if all(math.isfinite(x) for x in ks) else float(np.sum(ks))
    return OpsResult(logp, w, acted, term, flags, logk, eps, gate, rho, loss, n_acted, max_abs,
                     excess, grad)


def _row_valid(ids, mask, t, V):
    y = int(ids[t])
    on = True if mask is None else bool(mask[t])
    return on, (on and 0 <= y < V)


def cis_ops_loss(logits, ids, logp_infer, adv, mask, prm: OpParams, with_grad: bool = True,
                 rows=None) -> OpsResult:
    """The rho = 1 path of ``oracle.cis.cis_loss`` with any token-level operator: p_t from the
    same logits, term = scale * w * A * log p, gradient scale * w * A * (onehot - softmax)."""
    if prm.op in SEQ_OPS:
        raise ValueError("sequence operators need the recorded training log-probabilities")
    T, V = logits.shape
    sel = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    n = sel.shape[0]
    logp, w, term, logk, eps = (np.zeros(n) for _ in range(5))
    acted = np.zeros(n, dtype=bool)
    gate = np.zeros(n, dtype=bool)
    rho = np.ones(n)
    flags = np.zeros(n, dtype=np.uint8)
    grad = np.zeros((n, V)) if with_grad else None
    for i, t in enumerate(sel):
        on, valid = _row_valid(ids, mask, t, V)
        if not valid:
            flags[i] = FLAG_BAD_ID if on else 0
            continue
        y = int(ids[t])
        z = np.asarray(logits[t], dtype=np.float64)
        rs = row_log_softmax(z, y)
        lq = float(logp_infer[t])
        wt, act = token_weight(prm.op, rs.logp, lq, rs.one_minus_p, prm)
        f = FLAG_VALID | (FLAG_TRUNC if act else 0)
        if not math.isfinite(rs.lse) or math.isnan(wt):
            f |= FLAG_NONFINITE
        flags[i], logp[i], w[i], acted[i] = f, rs.logp, wt, act
        logk[i] = rs.logp - lq
        eps[i] = displacement(rs.logp, lq, rs.one_minus_p)
        gate[i] = True
        coef = prm.scale * wt * float(adv[t])
        term[i] = 0.0 if coef == 0.0 else coef * rs.logp
        if with_grad:
            with np.errstate(invalid="ignore", over="ignore"):
                g = -coef * np.exp(z - rs.lse)
            g[y] = coef * rs.one_minus_p
            grad[i] = g
    return _finish(n, V, sel, logp, w, acted, term, flags, logk, eps, gate, rho, grad)


def cis_ppo_loss(logits, ids, logp_infer, logp_old, adv, mask, prm: OpParams, offsets=None,
                 with_grad: bool = True, rows=None) -> OpsResult:
    """The decoupled path of Eq. (1): weight from (l_old, l_infer), PPO-clipped update ratio
    rho = exp(l_train - l_old); per-token term scale * w * min(rho A, clip(rho) A) and its
    gradient scale * w * A * rho * (onehot - softmax) where the unclipped branch is the min."""
    T, V = logits.shape
    valid_all = np.array([_row_valid(ids, mask, t, V)[1] for t in range(T)], dtype=bool)
    lold = np.asarray(logp_old, dtype=np.float64)
    linf = np.asarray(logp_infer, dtype=np.float64)
    if prm.op in SEQ_OPS:
        if offsets is None:
            raise ValueError("sequence operators need response offsets")
        sw, sact, _ = seq_weights(prm.op, lold - linf, valid_all, offsets, prm)
    sel = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    n = sel.shape[0]
    logp, w, term, logk, eps = (np.zeros(n) for _ in range(5))
    acted = np.zeros(n, dtype=bool)
    gate = np.zeros(n, dtype=bool)
    rho = np.ones(n)
    flags = np.zeros(n, dtype=np.uint8)
    grad = np.zeros((n, V)) if with_grad else None
    for i, t in enumerate(sel):
        on, valid = _row_valid(ids, mask, t, V)
        if not valid:
            flags[i] = FLAG_BAD_ID if on else 0
            continue
        y = int(ids[t])
        z = np.asarray(logits[t], dtype=np.float64)
        rs = row_log_softmax(z, y)
        lo_, lq = float(lold[t]), float(linf[t])
        one_minus_p_old = -math.expm1(lo_)
        if prm.op in SEQ_OPS:
            wt, act = float(sw[t]), bool(sact[t])
        else:
            wt, act = token_weight(prm.op, lo_, lq, one_minus_p_old, prm)
        r = _exp(rs.logp - lo_)
        A = float(adv[t])
        f = FLAG_VALID | (FLAG_TRUNC if act else 0)
        if not math.isfinite(rs.lse) or math.isnan(wt) or math.isnan(r):
            f |= FLAG_NONFINITE
        flags[i], logp[i], w[i], acted[i], rho[i] = f, rs.logp, wt, act, r
        logk[i] = lo_ - lq
        eps[i] = displacement(lo_, lq, one_minus_p_old)
        g_on = ppo_gate(r, A, prm.clip_low, prm.clip_high)
        gate[i] = g_on
        sw_ = prm.scale * wt
        term[i] = 0.0 if (sw_ == 0.0 or A == 0.0) else \
            sw_ * ppo_surrogate(r, A, prm.clip_low, prm.clip_high)
        coef = ppo_coef(sw_, A, r, g_on)
        if with_grad:
            if coef == 0.0:
                grad[i] = 0.0
            else:
                with np.errstate(invalid="ignore", over="ignore"):
                    g = -coef * np.exp(z - rs.lse)
                g[y] = coef * rs.one_minus_p
                grad[i] = g
    return _finish(n, V, sel, logp, w, acted, term, flags, logk, eps, gate, rho, grad)
