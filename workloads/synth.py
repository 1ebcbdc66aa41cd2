"""Seeded synthetic rollouts shaped like the paper's MoE RL workloads.

This module only draws inputs: training logits, the inference engine's perturbed logits, the
sampled ids and the log-probabilities the inference engine records at sampling, advantages and
masks. It holds none of the CIS arithmetic (no training-side log-softmax, weights or
gradients); both the HIP path and the CPU oracle consume what it produces.

Model of the two engines (Sec. 3.1): the training engine's logits are z, the inference
engine's are z + delta with a per-logit perturbation delta. The sampled id is drawn from
softmax(z + delta) at temperature 1 (Gumbel-max, exact), and the recorded inference
log-probability is log_softmax(z + delta)[y] (App. C.4: the raw value from the sampling step).
Advantages are GRPO group-normalised binary rewards (Sec. 2.1).

Configurations (the sizes of the five workloads the library is measured and checked on):

  0  tiny:    T = 256 (1 prompt x 4 responses x 64 tokens), V = 1024, float32 logits
              z ~ N(0, 3^2); delta ~ N(0, 0.02^2) per logit, and 1% of the rows (3) get
              delta ~ N(0, 1) instead; all rows valid; c = 1.
  1  small:   T = 32768 slots (16 prompts x 8 responses x 256), V = 32768, bf16 logits
              z ~ N(0, 3^2) plus one peaked entry per row at (row max + PEAK_1); response
              lengths U{64..256} with a padding mask; delta as in 0; c = 1.
  2  MoE:     T = 16384 packed tokens of 32 prompts x 16 responses with lengths U{256..1536},
              V = 151936, bf16 logits z_j = -1.1 ln(j+1) + N(0, 2^2) (token id = Zipf rank);
              delta ~ N(0, 0.03^2), and 0.1% of the rows (16) get delta ~ N(0, 2^2);
              c in {0.5, 1, 2}.
  3  long:    T = 524288 (8 prompts x 8 responses x 8192) in 8 chunks of 65536 (one prompt
              group per chunk), V = 151936, distributions of 2 plus a peak (row max + PEAK_3)
              on a fraction PEAK_3_FRACTION of the rows, so that about 80% of the tokens have
              sampled training probability > 0.95; c = 1.
  4  wide:    T = 32768, V = 262144, logits as in 2; delta = 0.05 * Student-t(3) per logit;
              mask ~ Bernoulli(0.75); A ~ N(0, 1); c = 1.

The threshold c bounds the log-odds displacement, so lambda = e^c - 1; kappa = 5e-3 (the
paper's floor); scale = -1/N_valid (token-mean loss, minimised).
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch

# Peak offsets, calibrated by workloads/calibrate.py (see that script for the targets).
PEAK_1 = 4.69            # small workload: mean sampled training probability ~ 0.80
PEAK_3 = 9.0             # long response: peaked rows have training probability of the peak > 0.99
PEAK_3_FRACTION = 0.81   # long response: ~80% of tokens with sampled training probability > 0.95

KAPPA = 5e-3

CONFIGS = {
    0: dict(name="tiny", T=256, V=1024, dtype="float32", c=(1.0,)),
    1: dict(name="small-bf16", T=32768, V=32768, dtype="bfloat16", c=(1.0,)),
    2: dict(name="moe-rollout", T=16384, V=151936, dtype="bfloat16", c=(0.5, 1.0, 2.0)),
    3: dict(name="long-response", T=524288, V=151936, dtype="bfloat16", c=(1.0,), chunk=65536),
    4: dict(name="wide-vocab", T=32768, V=262144, dtype="bfloat16", c=(1.0,)),
}


@dataclass
class Batch:
    """One batch of inputs for the CIS loss (tensors on one device)."""
    logits: torch.Tensor          # [T, V] bf16 or fp32 (training engine)
    ids: torch.Tensor             # [T] int64 sampled ids
    logp_infer: torch.Tensor      # [T] fp32 inference log-prob of the sampled id
    adv: torch.Tensor             # [T] fp32 advantages
    mask: torch.Tensor            # [T] uint8 (1 = token counts)
    lam: float                    # threshold lambda
    kappa: float                  # floor kappa
    scale: float                  # loss normalisation
    meta: dict = field(default_factory=dict)

    @property
    def T(self) -> int:
        return self.logits.shape[0]

    @property
    def V(self) -> int:
        return self.logits.shape[1]


def lambda_of(c: float) -> float:
    return math.expm1(c)


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def group_advantages(rewards: torch.Tensor, eps: float = 1e-6) -> torch.Tensor:
    """GRPO advantages (r - mean) / (std + eps) within each group (rows of `rewards`)."""
    r = rewards.to(torch.float64)
    mean = r.mean(dim=1, keepdim=True)
    std = r.std(dim=1, unbiased=False, keepdim=True)
    return ((r - mean) / (std + eps)).to(torch.float32)


def _mixed_rewards(g: torch.Generator, groups: int, size: int, device) -> torch.Tensor:
    """Bernoulli(0.5) rewards; each group is redrawn until it is not all-equal (a group with
    identical rewards has zero advantage everywhere and exercises nothing)."""
    out = torch.empty(groups, size, device=device)
    for i in range(groups):
        while True:
            r = torch.bernoulli(torch.full((size,), 0.5, device=device), generator=g)
            if 0 < int(r.sum().item()) < size:
                out[i] = r
                break
    return out


def _sample_and_record(z_inf: torch.Tensor, g: torch.Generator):
    """Inference engine: y ~ softmax(z_inf) (Gumbel-max) and log_softmax(z_inf)[y] in float32."""
    zf = z_inf.float()
    u = torch.rand(zf.shape, generator=g, device=zf.device, dtype=torch.float32)
    u = u.clamp_(min=1e-30, max=1.0 - 1e-7)
    y = torch.argmax(zf - torch.log(-torch.log(u)), dim=1)
    lq = torch.log_softmax(zf, dim=1).gather(1, y[:, None])[:, 0]
    return y, lq


def _zipf_logits(rows: int, V: int, g: torch.Generator, device) -> torch.Tensor:
    bias = -1.1 * torch.log(torch.arange(1, V + 1, device=device, dtype=torch.float32))
    return bias[None, :] + 2.0 * torch.randn(rows, V, generator=g, device=device)


def _fill_rows(batch_logits, ids, lq, r0, z, delta, g, store_dtype):
    zq = z.to(store_dtype)
    z_inf = (zq.float() + delta).to(store_dtype)
    y, l = _sample_and_record(z_inf, g)
    batch_logits[r0:r0 + z.shape[0]] = zq
    ids[r0:r0 + z.shape[0]] = y
    lq[r0:r0 + z.shape[0]] = l


def make_batch(cfg: int, device="cuda", seed: int | None = None, chunk: int = 0,
               c: float | None = None, rows: int | None = None,
               rows_per_step: int = 1024) -> Batch:
    """Builds the inputs of workload `cfg` (chunk `chunk` of the chunked long-response workload).

    Every per-row quantity of the full batch (advantages, masks, outlier and peak rows) is
    drawn first and the logits afterwards, `rows_per_step` rows at a time; `rows` keeps only
    the first rows of the batch, which coincide with the full batch's when `rows` is a
    multiple of `rows_per_step`.
    """
    spec = CONFIGS[cfg]
    V = spec["V"]
    T = spec.get("chunk", spec["T"])
    R = T if rows is None else int(rows)
    c = spec["c"][0] if c is None else float(c)
    if seed is None:
        seed = cfg if cfg != 3 else 3000 + chunk
    g = _gen(device, seed)
    dt = torch.float32 if spec["dtype"] == "float32" else torch.bfloat16
    meta = {"config": cfg, "name": spec["name"], "seed": seed, "chunk": chunk, "c": c,
            "rows": R, "T_full": T}

    # ---- per-row quantities of the full batch ---------------------------------------------
    mask = torch.ones(T, dtype=torch.uint8, device=device)
    peaked = None
    if cfg == 0:
        adv = group_advantages(_mixed_rewards(g, 1, 4, device)).repeat_interleave(64, dim=1)
    elif cfg == 1:
        adv = group_advantages(_mixed_rewards(g, 16, 8, device)).repeat_interleave(256, dim=1)
        lengths = torch.randint(64, 257, (128,), generator=g, device=device)
        pos = torch.arange(256, device=device)[None, :]
        mask = (pos < lengths[:, None]).reshape(T).to(torch.uint8)
    elif cfg == 2:
        lengths = torch.randint(256, 1537, (32, 16), generator=g, device=device)
        adv_resp = group_advantages(_mixed_rewards(g, 32, 16, device)).reshape(-1)
        adv = torch.repeat_interleave(adv_resp, lengths.reshape(-1))[:T]
        meta["responses_in_batch"] = int((torch.cumsum(lengths.reshape(-1), 0) < T).sum()) + 1
    elif cfg == 3:
        adv = group_advantages(_mixed_rewards(g, 1, 8, device)).repeat_interleave(8192, dim=1)
        peaked = torch.rand(T, generator=g, device=device) < PEAK_3_FRACTION
    elif cfg == 4:
        adv = torch.randn(T, generator=g, device=device)
        mask = (torch.rand(T, generator=g, device=device) < 0.75).to(torch.uint8)
    else:
        raise ValueError(f"unknown config {cfg}")
    adv = adv.reshape(T).to(torch.float32)
    frac = 0.01 if cfg in (0, 1) else (0.001 if cfg in (2, 3) else 0.0)
    odd_rows = torch.randperm(T, generator=g, device=device)[:round(frac * T)]
    odd = torch.zeros(T, dtype=torch.bool, device=device)
    odd[odd_rows] = True
    meta["outlier_rows"] = sorted(odd_rows.tolist())

    # ---- logits, sampled ids and recorded inference log-probs, row block by row block -------
    logits = torch.empty(R, V, dtype=dt, device=device)
    ids = torch.empty(R, dtype=torch.int64, device=device)
    lq = torch.empty(R, dtype=torch.float32, device=device)
    for r0 in range(0, R, rows_per_step):
        n = min(rows_per_step, R - r0)
        if cfg in (0, 1):
            z = 3.0 * torch.randn(n, V, generator=g, device=device)
        else:
            z = _zipf_logits(n, V, g, device)
        if cfg in (1, 3):
            peak = torch.randint(0, V, (n,), generator=g, device=device)
            top = z.max(dim=1).values
            sel = torch.ones(n, dtype=torch.bool, device=device) if cfg == 1 else peaked[r0:r0 + n]
            rr = torch.arange(n, device=device)[sel]
            z[rr, peak[sel]] = top[sel] + (PEAK_1 if cfg == 1 else PEAK_3)
        if cfg == 4:
            # Student-t(3) = N(0,1) / sqrt(chi2_3 / 3), drawn from the seeded generator
            nrm = torch.randn(n, V, generator=g, device=device)
            chi = torch.zeros(n, V, device=device)
            for _ in range(3):
                chi += torch.randn(n, V, generator=g, device=device) ** 2
            delta = 0.05 * nrm / torch.sqrt(chi / 3.0)
            del nrm, chi
        else:
            base, wide = (0.02, 1.0) if cfg in (0, 1) else (0.03, 2.0)
            sd = torch.where(odd[r0:r0 + n], wide, base)[:, None]
            delta = sd * torch.randn(n, V, generator=g, device=device)
        _fill_rows(logits, ids, lq, r0, z, delta, g, dt)
        del z, delta

    mask = mask[:R].contiguous()
    n_valid = int(mask.sum().item())
    scale = -1.0 / max(n_valid, 1)
    return Batch(logits, ids, lq, adv[:R].contiguous(), mask, lambda_of(c), KAPPA, scale, meta)


def make_random_batch(T: int, V: int, dtype=torch.bfloat16, device="cuda", seed: int = 0,
                      sd: float = 3.0, delta_sd: float = 0.5, c: float = 1.0,
                      kappa: float = KAPPA, mask_p: float = 1.0, ld: int | None = None) -> Batch:
    """A small generic batch (edge-case tests): z ~ N(0, sd^2), delta ~ N(0, delta_sd^2),
    A ~ N(0, 1), mask ~ Bernoulli(mask_p); optional row stride ld >= V (padding columns are
    filled with NaN so that reading them would show)."""
    g = _gen(device, seed)
    z = sd * torch.randn(T, V, generator=g, device=device)
    delta = delta_sd * torch.randn(T, V, generator=g, device=device)
    ld = V if ld is None else ld
    store = torch.full((T, ld), float("nan"), dtype=dtype, device=device)
    ids = torch.empty(T, dtype=torch.int64, device=device)
    lq = torch.empty(T, dtype=torch.float32, device=device)
    view = store[:, :V]
    zq = z.to(dtype)
    y, l = _sample_and_record((zq.float() + delta).to(dtype), g)
    view.copy_(zq)
    ids.copy_(y)
    lq.copy_(l)
    adv = torch.randn(T, generator=g, device=device)
    mask = (torch.rand(T, generator=g, device=device) < mask_p).to(torch.uint8)
    n_valid = max(int(mask.sum().item()), 1)
    return Batch(view, ids, lq, adv, mask, lambda_of(c), kappa, -1.0 / n_valid,
                 {"seed": seed, "ld": ld})


def old_logprobs(b: Batch, sd: float = 0.3, seed: int = 0) -> torch.Tensor:
    """Training-side log-probabilities of the sampled ids at a rollout snapshot theta_old, for
    the decoupled objective (App. C.1: both engines' log-probabilities are recorded per token):
    log_softmax(z + sd * N(0, 1))[y] in float32, with z the stored training logits. The update
    ratio exp(l_train - l_old) then spreads around 1 by about sd in log space."""
    g = _gen(b.logits.device, 7919 + seed)
    T = b.T
    out = torch.empty(T, dtype=torch.float32, device=b.logits.device)
    step = max(1, min(T, (1 << 27) // max(b.V, 1)))
    for r0 in range(0, T, step):
        z = b.logits[r0:r0 + step].float()
        z = z + sd * torch.randn(z.shape, generator=g, device=z.device)
        y = b.ids[r0:r0 + step].clamp(0, b.V - 1)
        out[r0:r0 + step] = torch.log_softmax(z, dim=1).gather(1, y[:, None])[:, 0]
    return out


def response_offsets(T: int, min_len: int, max_len: int, seed: int = 0,
                     device="cuda") -> torch.Tensor:
    """CSR offsets [n + 1] of responses packed back to back over T tokens, lengths uniform in
    [min_len, max_len] (the last one cut at T)."""
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    offs = [0]
    while offs[-1] < T:
        n = int(torch.randint(min_len, max_len + 1, (1,), generator=g).item())
        offs.append(min(T, offs[-1] + n))
    return torch.tensor(offs, dtype=torch.int64, device=device)
