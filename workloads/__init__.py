"""Seeded synthetic inputs for the CIS loss (no CIS arithmetic; see workloads.synth)."""
from .synth import (  # noqa: F401
    CONFIGS, KAPPA, Batch, group_advantages, lambda_of, make_batch, make_random_batch,
    old_logprobs, response_offsets,
)
from .lmhead import LmHeadBatch, make_lmhead_batch  # noqa: F401,E402
