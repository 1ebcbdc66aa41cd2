"""Plain float64 CPU oracle for the CIS token loss behind the language-model head:
logits = hidden @ W^T, then the loss of ``oracle.cis`` / ``oracle.ops``, and the gradients with
respect to the hidden states and the head's weight.

TEST INFRASTRUCTURE ONLY (like ``oracle.cis``): only the test suite, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py`` may import it; the HIP library shares nothing with it.

What it restates (arXiv 2609.32444): the training engine's logits of Sec. 3.1 are the output of
the model's final projection, z_t = W h_t with h_t the last hidden state of token t and W the
[V, H] head weight (the training engine of App. C.1 computes them in bf16). The loss is the one of
``oracle.cis.cis_loss`` (rate 1) or ``oracle.ops.cis_ppo_loss`` (decoupled path) on those logits.
With G = dL/dz ([T, V]), the chain rule gives

    dL/dh = G @ W        ([T, H]),
    dL/dW = G^T @ h      ([V, H]).

Readings:

* The logits are the exact products of the bf16 inputs (float64 here). A kernel that keeps them
  in float32 accumulators differs by the float32 dot-product rounding; one that rounds them to
  bf16 first (as a materialised bf16 logits tensor would) differs by bf16 rounding.
* Matrix products are numpy's (a library primitive), in float64, over bf16 inputs converted
  exactly. Large problems are processed in row chunks; the sum over chunks of G_c^T h_c is the
  same product regrouped.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

from . import cis as O
from . import ops as X

__all__ = ["LmHeadResult", "lmhead_logits", "lmhead_cis_loss"]


def lmhead_logits(hidden: np.ndarray, W: np.ndarray) -> np.ndarray:
    """z = hidden @ W^T in float64 (hidden [T, H], W [V, H], both float64 or exactly
    convertible)."""
    return np.asarray(hidden, dtype=np.float64) @ np.asarray(W, dtype=np.float64).T


@dataclass
class LmHeadResult:
    logp_train: np.ndarray    # [T]
    w: np.ndarray             # [T]
    acted: np.ndarray         # [T] bool
    term: np.ndarray          # [T]
    flags: np.ndarray         # [T] uint8
    logk: np.ndarray          # [T] log k of the operator's weight (oracle.ops)
    eps: np.ndarray           # [T] displacement
    gate: np.ndarray          # [T] bool, the PPO gradient flows (decoupled path)
    rho: np.ndarray           # [T] update ratio (1 on the rate-1 path)
    loss: float
    dhidden: np.ndarray | None  # [T, H] float64
    dW: np.ndarray | None       # [V, H] float64
    grad: np.ndarray | None = None  # [T, V] dL/dz (keep_grad only)


def lmhead_cis_loss(hidden, W, ids, logp_infer, adv, mask, prm: "X.OpParams",
                    logp_old=None, offsets=None, with_grad: bool = True,
                    chunk: int = 1024, keep_grad: bool = False) -> LmHeadResult:
    """The CIS loss (or any operator of oracle.ops; the decoupled path with logp_old) on the
    logits hidden @ W^T, and its gradients with respect to hidden and W, in float64.
    keep_grad also returns dL/dz itself (small problems)."""
    hidden = np.asarray(hidden, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    T, H = hidden.shape
    V = W.shape[0]
    out = {k: [] for k in ("logp_train", "w", "acted", "term", "flags", "logk", "eps", "gate",
                           "rho")}
    dhidden = np.zeros((T, H)) if with_grad else None
    dW = np.zeros((V, H)) if with_grad else None
    grads = [] if (with_grad and keep_grad) else None
    for t0 in range(0, T, chunk):
        t1 = min(T, t0 + chunk)
        z = lmhead_logits(hidden[t0:t1], W)
        sl = slice(t0, t1)
        m = None if mask is None else np.asarray(mask)[sl]
        if logp_old is None:
            r = X.cis_ops_loss(z, np.asarray(ids)[sl], np.asarray(logp_infer)[sl],
                               np.asarray(adv)[sl], m, prm, with_grad=with_grad)
        else:
            # sequence operators need the whole batch: pass every row, keep this chunk's
            r = X.cis_ppo_loss(_Rows(z, t0, T), ids, logp_infer, logp_old, adv, mask, prm,
                               offsets=offsets, with_grad=with_grad, rows=np.arange(t0, t1))
        for k in out:
            out[k].append(getattr(r, k))
        if with_grad:
            G = r.grad
            if grads is not None:
                grads.append(G)
            dhidden[t0:t1] = G @ W
            dW += G.T @ hidden[t0:t1]
    res = {k: np.concatenate(v) for k, v in out.items()}
    term = res["term"]
    loss = math.fsum(term.tolist()) if np.all(np.isfinite(term)) else float(np.sum(term))
    return LmHeadResult(res["logp_train"], res["w"], res["acted"], term, res["flags"],
                        res["logk"], res["eps"], res["gate"], res["rho"], loss, dhidden, dW,
                        np.concatenate(grads) if grads else None)


class _Rows:
    """Row access to one chunk of logits as if it were the whole [T, V] matrix (only the
    chunk's rows are ever read)."""

    def __init__(self, z, t0, T):
        self.z, self.t0 = z, t0
        self.shape = (T, z.shape[1])

    def __getitem__(self, t):
        return self.z[t - self.t0]
