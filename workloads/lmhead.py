"""Seeded synthetic inputs for the loss behind the language-model head: last hidden states h
[T, H] and a head weight W [V, H] (bf16), whose logits z = h W^T follow the MoE rollout's
distribution (Zipf-ranked bias plus N(0, 2^2) per logit), and the rollout quantities of
``workloads.synth`` drawn from those logits.

Like ``workloads.synth`` this module only draws inputs and holds none of the CIS arithmetic.

Exact logits. Every hidden entry is a multiple of 1/4 with at most 4 significant bits
(round(4 N(0, 1)) / 4, clipped to [-15/4, 15/4]) except column 0, which is 1 and carries the
bias; every head entry of columns 1.. is m 2^-p with |m| <= 127 (about N(0, 4 / (H - 1))), and
column 0 holds the bias -1.1 ln(v + 1) rounded to a multiple of 2^-(p+2) and to bf16. All
products are then integer multiples of 2^-(p+2), and for H up to 8192 every partial sum of a
row's dot product stays below 2^24 such units: float32 accumulation in any order gives the
exact logits, so a kernel's float32 logits equal the float64 ones and the loss comparisons see
only the loss's own rounding.

General inputs (exact=False). Hidden entries N(0, 1) and head entries N(0, 4 / (H - 1)) rounded
once to bf16 (column 0 as above: 1 and the bias rounded to bf16), with no further quantisation:
float32 dot products of these are not exact, which is what a test of the products' own rounding
needs.

The sampled ids come from softmax(z + delta) (Gumbel-max), delta ~ N(0, 0.03^2) per logit with
0.1% of the rows at N(0, 2^2), and the recorded inference log-probability is
log_softmax(z + delta)[y] in float32 (the model of ``workloads.synth``). Advantages are GRPO
group-normalised binary rewards over packed responses (groups of 16, lengths
U{min_len..max_len}); the optional mask is Bernoulli(mask_p).
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional

import torch

from .synth import KAPPA, _gen, _mixed_rewards, _sample_and_record, group_advantages, lambda_of

MAX_EXACT_H = 8192


@dataclass
class LmHeadBatch:
    hidden: torch.Tensor          # [T, H] bf16 (row stride ld_h)
    weight: torch.Tensor          # [V, H] bf16 (row stride ld_w)
    ids: torch.Tensor             # [T] int64
    logp_infer: torch.Tensor      # [T] float32
    adv: torch.Tensor             # [T] float32
    mask: torch.Tensor            # [T] uint8
    offsets: torch.Tensor         # [n_seq + 1] int64 response boundaries
    lam: float
    kappa: float
    scale: float
    logp_old: Optional[torch.Tensor] = None   # [T] float32 (decoupled path)
    meta: dict = field(default_factory=dict)

    @property
    def T(self) -> int:
        return self.hidden.shape[0]

    @property
    def H(self) -> int:
        return self.hidden.shape[1]

    @property
    def V(self) -> int:
        return self.weight.shape[0]


def _scale_exponent(H: int) -> int:
    """p with sigma_w 2^p in [16, 32), sigma_w = 2 / sqrt(max(H - 1, 1))."""
    sw = 2.0 / math.sqrt(max(H - 1, 1))
    return int(math.ceil(math.log2(16.0 / sw)))


def _padded(rows: int, cols: int, ld: int, device) -> torch.Tensor:
    store = torch.full((rows, ld), float("nan"), dtype=torch.bfloat16, device=device)
    return store[:, :cols]


def make_lmhead_batch(T: int, V: int, H: int, device="cuda", seed: int = 0, c: float = 1.0,
                      mask_p: float = 1.0, min_len: int = 256, max_len: int = 1536,
                      group: int = 16, zipf: bool = True, delta_sd: float = 0.03,
                      outlier_frac: float = 0.001, outlier_sd: float = 2.0,
                      old_sd: Optional[float] = None, ld_h: Optional[int] = None,
                      ld_w: Optional[int] = None, rows_per_step: int = 1024,
                      exact: bool = True) -> LmHeadBatch:
    """One batch; `old_sd` also draws logp_old = log_softmax(z + old_sd N(0, 1))[y] (the
    rollout snapshot of the decoupled objective). ld_h / ld_w >= H give padded row strides
    (padding holds NaN). exact=False draws general bf16 inputs (module docstring)."""
    if exact and H > MAX_EXACT_H:
        raise ValueError(f"exact logits need H <= {MAX_EXACT_H}")
    g = _gen(device, seed)
    p = _scale_exponent(H)
    unit = 2.0 ** -(p + 2)

    # ---- per-row quantities ---------------------------------------------------------------
    offs = [0]
    lens = []
    gl = torch.Generator(device="cpu")
    gl.manual_seed(int(seed) + 104729)
    while offs[-1] < T:
        n = int(torch.randint(min_len, max_len + 1, (1,), generator=gl).item())
        offs.append(min(T, offs[-1] + n))
        lens.append(offs[-1] - offs[-2])
    n_resp = len(lens)
    n_groups = (n_resp + group - 1) // group
    adv_resp = group_advantages(_mixed_rewards(g, n_groups, group, device)).reshape(-1)[:n_resp]
    lengths = torch.tensor(lens, dtype=torch.int64, device=device)
    adv = torch.repeat_interleave(adv_resp, lengths).to(torch.float32).contiguous()
    if mask_p >= 1.0:
        mask = torch.ones(T, dtype=torch.uint8, device=device)
    else:
        mask = (torch.rand(T, generator=g, device=device) < mask_p).to(torch.uint8)
    n_odd = round(outlier_frac * T)
    odd = torch.zeros(T, dtype=torch.bool, device=device)
    if n_odd > 0:
        odd[torch.randperm(T, generator=g, device=device)[:n_odd]] = True

    # ---- head weight and hidden states ------------------------------------------------------
    sw = 2.0 / math.sqrt(max(H - 1, 1))
    weight = _padded(V, H, ld_w or H, device)
    if exact:
        m = torch.round(sw * 2.0 ** p * torch.randn(V, H, generator=g, device=device))
        wt = m.clamp_(-127, 127) * 2.0 ** -p
    else:
        m = None
        wt = sw * torch.randn(V, H, generator=g, device=device)
    if zipf:
        bias = -1.1 * torch.log(torch.arange(1, V + 1, device=device, dtype=torch.float64))
        if exact:
            bias = torch.round(bias / unit) * unit
        bias = bias.to(torch.bfloat16).float()
    else:
        bias = torch.zeros(V, device=device)
    wt[:, 0] = bias
    weight.copy_(wt.to(torch.bfloat16))
    del wt, m
    hidden = _padded(T, H, ld_h or H, device)
    hv = torch.randn(T, H, generator=g, device=device)
    if exact:
        hv = torch.round(4.0 * hv).clamp_(-15, 15) / 4.0
    hv[:, 0] = 1.0
    hidden.copy_(hv.to(torch.bfloat16))
    del hv

    # ---- sampled ids and recorded log-probabilities, from the exact logits -----------------
    ids = torch.empty(T, dtype=torch.int64, device=device)
    lq = torch.empty(T, dtype=torch.float32, device=device)
    lold = torch.empty(T, dtype=torch.float32, device=device) if old_sd is not None else None
    go = _gen(device, 7919 + seed) if old_sd is not None else None
    wf = weight.float()
    for r0 in range(0, T, rows_per_step):
        n = min(rows_per_step, T - r0)
        z = hidden[r0:r0 + n].float() @ wf.T
        sd = torch.where(odd[r0:r0 + n], outlier_sd, delta_sd)[:, None]
        delta = sd * torch.randn(z.shape, generator=g, device=device)
        y, l = _sample_and_record((z + delta).to(torch.bfloat16), g)
        ids[r0:r0 + n] = y
        lq[r0:r0 + n] = l
        if lold is not None:
            zo = z + old_sd * torch.randn(z.shape, generator=go, device=device)
            lold[r0:r0 + n] = torch.log_softmax(zo, dim=1).gather(1, y[:, None])[:, 0]
        del z, delta
    del wf
    n_valid = int(mask.sum().item())
    meta = {"seed": seed, "c": c, "p": p, "n_resp": n_resp, "outlier_rows": int(n_odd),
            "exact": bool(exact)}
    return LmHeadBatch(hidden, weight, ids, lq, adv, mask,
                       torch.tensor(offs, dtype=torch.int64, device=device), lambda_of(c),
                       KAPPA, -1.0 / max(n_valid, 1), lold, meta)
