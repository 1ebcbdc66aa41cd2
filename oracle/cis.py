"""Plain float64 CPU oracle for the CIS token loss, forward and backward.

TEST INFRASTRUCTURE ONLY. This package checks the product and is not part of it: only the test
suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import it.
The HIP library never calls it, and it shares no code, tables or constants with it.

Source: Yu et al., "Rethinking Training-Inference Mismatch in LLM Reinforcement Learning:
Where It Arises and How to Correct It" (arXiv 2609.32444). Everything below restates the paper
in plain numpy, one token row at a time, in float64:

* Sec. 2.1, Eq. (1) (``eq:objective``): sampled token y_t, training-side probability
  p_t = softmax(z)_y, inference-side probability q_t, mismatch ratio k_t = p_t / q_t.
* Sec. 3.1, Lemma 1 (``lem:ratio_displacement``, Eq. ``eq:k_geometry``): the log-odds
  displacement eps_t = logit p_t - logit q_t and k_t = p_t + (1 - p_t) e^{eps_t}.
* Sec. 3.3, Eq. (4) (``eq:cis_operator``): the CIS operator
  f_lambda(k, p) = min{k, 1 + lambda (1 - p)}; the paper evaluates the right-hand form from the
  difference of the two log-probabilities.
* Sec. 3.3, Algorithm 1 (``alg:cis``) and the paragraph after it: the deployed weight
  f = min{k, 1 + lambda * max(1 - p, kappa)}, detached (stop-gradient), multiplying the
  per-token policy-gradient payload; the inference log-probability is the raw value recorded
  at sampling.
* App. C.1 "Operators": p_t is taken from the training-side log-probability; the weight
  multiplies the token loss and carries no gradient.

The per-token loss is the REINFORCE form at update ratio rho = 1 (the first minibatch, where
the training parameters equal the rollout snapshot), whose gradient with respect to the
training logits is the one the method applies:

    term_t = scale * w_t * A_t * log p_t,
    dterm_t / dz_t = scale * w_t * A_t * (onehot(y_t) - softmax(z_t)),

with w_t held constant (stop-gradient). ``scale`` is the caller's normalisation (for example
-1/N_valid for a token-mean loss to be minimised); per-response 1/|y_i| factors of Eq. (1) fold
into A_t.

Readings where the paper is silent:

* A row is valid when its mask is nonzero and 0 <= y < V; invalid rows produce zeros.
* 1 - p is evaluated as the complement mass sum_{j != y} e^{z_j - m} / sum_j e^{z_j - m}, a
  sum of its own, so that it keeps its relative accuracy as p -> 1 (the same resolution
  problem that motivates the floor kappa in Sec. 3.3).
* The truncation flag is strict: a token is truncated when k > 1 + lambda*phi (at equality
  both branches give the same weight).
* term_t is defined as 0 when the coefficient scale*w*A is 0 (so that p = 0 with w = 0 gives
  0 rather than 0 * -inf).
* A row is "non-finite" when its log-sum-exp is not finite or its weight is NaN; values in
  such rows are unspecified and only the flag is compared.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

__all__ = [
    "bf16_bits_to_float64",
    "round_float64_to_bf16_bits",
    "bf16_neighbors",
    "Bf16Matrix",
    "row_log_softmax",
    "cis_weight",
    "cis_weights",
    "log_odds_displacement",
    "cis_loss",
    "CisResult",
]


# --------------------------------------------------------------------------------------------
# bfloat16 <-> float64 (storage format of the training logits and of the gradient)
# --------------------------------------------------------------------------------------------

def bf16_bits_to_float64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bfloat16 bit patterns (uint16) as float64.

    A bfloat16 is the upper half of an IEEE binary32, so the value is exact in float64.
    """
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


_BF16_MAX = math.ldexp(2.0 - 2.0 ** -7, 127)      # largest finite bfloat16
_BF16_MIN_NORMAL = 2.0 ** -126
_BF16_SUB_ULP = 2.0 ** -133                         # spacing of bfloat16 subnormals


def _round_half_even(x: np.ndarray) -> np.ndarray:
    # numpy's rint rounds halfway cases to the even integer
    return np.rint(x)


def round_float64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bfloat16 (round to nearest, ties to even), returning uint16 bits.

    Rounds directly from float64 (no intermediate float32, so no double rounding). bfloat16 has
    an 8-bit significand (7 stored bits), binary32's exponent range, subnormals down to
    2^-133, and overflows to infinity at or beyond _BF16_MAX + half an ulp.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.float64)
    ax = np.abs(x)
    finite = np.isfinite(x)
    normal = finite & (ax >= _BF16_MIN_NORMAL)
    sub = finite & (ax < _BF16_MIN_NORMAL)
    # normal range: x = m * 2^e with m in [0.5, 1); keep 8 significant bits
    m, e = np.frexp(np.where(normal, x, 1.0))
    rn = np.ldexp(_round_half_even(m * 256.0), e - 8)
    out[normal] = rn[normal]
    # subnormal range: multiples of 2^-133
    out[sub] = _round_half_even(x[sub] / _BF16_SUB_ULP) * _BF16_SUB_ULP
    out[~finite] = x[~finite]
    # overflow: rounding may carry past the largest finite value
    with np.errstate(over="ignore"):
        big = finite & (np.abs(out) > _BF16_MAX)
    out[big] = np.copysign(np.inf, x[big])
    # float64 -> float32 is exact for every value produced above; take the upper 16 bits
    f32 = out.astype(np.float32)
    bits = (f32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    # NaN: canonical quiet NaN with the input's sign
    nan = np.isnan(x)
    bits[nan] = np.where(np.signbit(x[nan]), 0xFFC0, 0x7FC0).astype(np.uint16)
    return bits


class Bf16Matrix:
    """Read-only [T, V] matrix of bfloat16 bit patterns whose rows read as float64.

    Lets the oracle walk a large bfloat16 logits matrix one row at a time without holding a
    float64 copy of all of it.
    """

    def __init__(self, bits: np.ndarray):
        self.bits = np.asarray(bits, dtype=np.uint16)
        self.shape = self.bits.shape

    def __getitem__(self, t) -> np.ndarray:
        return bf16_bits_to_float64(self.bits[t])


def bf16_neighbors(x: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """The two bfloat16 values that bracket each float64 x (equal when x is representable).

    Returns float64 arrays (lo, hi) with lo <= x <= hi. A result that is lo or hi is a faithful
    rounding of x.
    """
    x = np.asarray(x, dtype=np.float64)
    r = bf16_bits_to_float64(round_float64_to_bf16_bits(x))
    # step to the adjacent bfloat16 in the direction of x
    rb = round_float64_to_bf16_bits(x).astype(np.int32)
    up = np.where(r < x, 1, np.where(r > x, -1, 0))
    # bfloat16 ordering on sign-magnitude bits: moving away from zero increments the
    # magnitude bits, for either sign
    sign = np.where(np.signbit(r), -1, 1)
    other_bits = (rb + up * sign).astype(np.uint16)
    other = bf16_bits_to_float64(other_bits)
    other = np.where(up == 0, r, other)
    lo = np.minimum(r, other)
    hi = np.maximum(r, other)
    return lo, hi


# --------------------------------------------------------------------------------------------
# Training-side log-softmax of one row (Sec. 3.1: p_t = softmax(z)_y)
# --------------------------------------------------------------------------------------------

@dataclass
class RowSoftmax:
    m: float          # max_j z_j
    s: float          # sum_j exp(z_j - m)
    s_rest: float     # sum_{j != y} exp(z_j - m), summed on its own
    lse: float        # log sum_j exp(z_j)
    logp: float       # log p_y = z_y - lse
    one_minus_p: float  # s_rest / s


def row_log_softmax(z: np.ndarray, y: int) -> RowSoftmax:
    """log softmax(z)_y and the complement mass 1 - p_y for one float64 row."""
    z = np.asarray(z, dtype=np.float64)
    with np.errstate(invalid="ignore", over="ignore"):
        m = float(np.max(z))
        e = np.exp(z - m)
        s = float(np.sum(e))
        e_rest = e.copy()
        e_rest[y] = 0.0
        s_rest = float(np.sum(e_rest))
        lse = m + math.log(s) if s > 0 and math.isfinite(s) else (
            -math.inf if s == 0 else math.nan)
        logp = float(z[y]) - lse
        one_minus_p = s_rest / s if s > 0 else math.nan
    return RowSoftmax(m, s, s_rest, lse, logp, one_minus_p)


# --------------------------------------------------------------------------------------------
# The CIS weight (Eq. (4) and Algorithm 1)
# --------------------------------------------------------------------------------------------

def cis_weight(logp_train: float, logp_infer: float, one_minus_p: float,
               lam: float, kappa: float) -> tuple[float, bool]:
    """Algorithm 1 for one token: (w, truncated).

    k = exp(l_train - l_infer); phi = max(1 - p, kappa); w = min{k, 1 + lambda*phi}.
    ``one_minus_p`` is 1 - p_t of the training side. ``truncated`` is True when the cap is
    strictly smaller than k.
    """
    delta = logp_train - logp_infer
    if math.isnan(delta):
        k = math.nan
    elif delta > 709.0:            # exp overflows float64: k = +inf
        k = math.inf
    else:
        k = math.exp(delta)
    phi = max(one_minus_p, kappa)
    cap = 1.0 + lam * phi
    if math.isnan(k):
        return math.nan, False
    truncated = k > cap
    w = cap if truncated else k
    return w, truncated


def cis_weights(logp_train: np.ndarray, logp_infer: np.ndarray, mask: np.ndarray | None,
                lam: float, kappa: float) -> tuple[np.ndarray, np.ndarray]:
    """Algorithm 1 over arrays of recorded log-probabilities: (w [n] float64, trunc [n] bool).

    Here p comes from the given training log-probability, and 1 - p is evaluated as
    -expm1(l_train), which equals 1 - exp(l_train) without its cancellation as p -> 1.
    Masked tokens (mask == 0) get w = 0, trunc = False.
    """
    lt = np.asarray(logp_train, dtype=np.float64)
    li = np.asarray(logp_infer, dtype=np.float64)
    n = lt.shape[0]
    w = np.zeros(n, dtype=np.float64)
    tr = np.zeros(n, dtype=bool)
    for i in range(n):
        if mask is not None and not mask[i]:
            continue
        one_minus_p = -math.expm1(lt[i])
        w[i], tr[i] = cis_weight(float(lt[i]), float(li[i]), one_minus_p, lam, kappa)
    return w, tr


def log_odds_displacement(logp_train: float, logp_infer: float) -> float:
    """eps_t = logit p_t - logit q_t (Lemma 1, log-odds form), from two log-probabilities.

    logit p = log p - log(1 - p) = l - log(-expm1(l)). Undefined (nan) when a probability is 1.
    """
    def logit_from_log(l: float) -> float:
        if l >= 0.0:
            return math.nan
        return l - math.log(-math.expm1(l))
    return logit_from_log(logp_train) - logit_from_log(logp_infer)


# --------------------------------------------------------------------------------------------
# The fused token loss and its gradient
# --------------------------------------------------------------------------------------------

FLAG_VALID = 1
FLAG_BAD_ID = 2
FLAG_NONFINITE = 4
FLAG_TRUNC = 8


@dataclass
class CisResult:
    logp_train: np.ndarray   # [T] float64, 0 on invalid rows
    w: np.ndarray            # [T] float64, 0 on invalid rows
    trunc: np.ndarray        # [T] bool
    term: np.ndarray         # [T] float64, scale*w*A*logp (0 when the coefficient is 0)
    flags: np.ndarray        # [T] uint8, FLAG_* bits
    loss: float              # math.fsum(term)
    grad: np.ndarray | None  # [T, V] float64 or None


def cis_loss(logits: np.ndarray, ids: np.ndarray, logp_infer: np.ndarray, adv: np.ndarray,
             mask: np.ndarray | None, lam: float, kappa: float, scale: float,
             with_grad: bool = True, rows: np.ndarray | None = None) -> CisResult:
    """CIS-weighted token loss over logits [T, V] (float64), and optionally dL/dlogits.

    ``logits`` is any [T, V] matrix whose rows convert to float64 (a numpy array, or a
    Bf16Matrix of bfloat16 bit patterns). ``rows`` restricts the work to a subset of row
    indices; the returned arrays are indexed like ``rows`` (all rows when it is None).
    """
    T, V = logits.shape
    sel = np.arange(T) if rows is None else np.asarray(rows, dtype=np.int64)
    n = sel.shape[0]
    logp = np.zeros(n)
    w = np.zeros(n)
    trunc = np.zeros(n, dtype=bool)
    term = np.zeros(n)
    flags = np.zeros(n, dtype=np.uint8)
    grad = np.zeros((n, V)) if with_grad else None
    for i, t in enumerate(sel):
        y = int(ids[t])
        masked_in = True if mask is None else bool(mask[t])
        if not masked_in:
            continue
        if not (0 <= y < V):
            flags[i] = FLAG_BAD_ID
            continue
        z = np.asarray(logits[t], dtype=np.float64)
        rs = row_log_softmax(z, y)
        wt, tr = cis_weight(rs.logp, float(logp_infer[t]), rs.one_minus_p, lam, kappa)
        f = FLAG_VALID | (FLAG_TRUNC if tr else 0)
        if not math.isfinite(rs.lse) or math.isnan(wt):
            f |= FLAG_NONFINITE
        flags[i] = f
        logp[i] = rs.logp
        w[i] = wt
        trunc[i] = tr
        coef = scale * wt * float(adv[t])
        term[i] = 0.0 if coef == 0.0 else coef * rs.logp
        if with_grad:
            with np.errstate(invalid="ignore", over="ignore"):
                g = -coef * np.exp(z - rs.lse)
            g[y] = coef * rs.one_minus_p
            grad[i] = g
    loss = math.fsum(term.tolist()) if np.all(np.isfinite(term)) else float(np.sum(term))
    return CisResult(logp, w, trunc, term, flags, loss, grad)
