"""The LM-head input generator's promise (workloads/lmhead.py): every float32 partial sum of
h W^T is exact, so float32 logits in any summation order equal the float64 ones; and the logits
follow the MoE rollout's distribution (Zipf bias plus spread about 2)."""

import numpy as np
import pytest
import torch

from workloads import make_lmhead_batch


@pytest.mark.parametrize("T,V,H", [(64, 3001, 136), (16, 1000, 2048), (8, 257, 8), (4, 64, 8192)])
def test_float32_sums_are_exact(T, V, H):
    b = make_lmhead_batch(T, V, H, device="cpu", seed=3, min_len=4, max_len=16)
    h = b.hidden.double().numpy()
    W = b.weight.double().numpy()
    z = h @ W.T
    # sequential float32 accumulation, forwards and backwards over H
    for order in (range(H), range(H - 1, -1, -1)):
        acc = np.zeros((T, V), np.float32)
        for j in order:
            acc += h[:, j:j + 1].astype(np.float32) * W[:, j].astype(np.float32)[None, :]
        assert np.array_equal(acc.astype(np.float64), z)
    # the values are bf16 numbers with the stated structure
    assert np.all(h[:, 0] == 1.0)
    assert np.all(np.abs(h[:, 1:] * 4) <= 15) and np.all((h[:, 1:] * 4) == np.round(h[:, 1:] * 4))


def test_logit_distribution_and_rollout_fields():
    b = make_lmhead_batch(256, 20000, 512, device="cpu", seed=5, min_len=16, max_len=64,
                          old_sd=0.3)
    z = b.hidden.double().numpy() @ b.weight.double().numpy().T
    bias = -1.1 * np.log(np.arange(1, 20001))
    spread = (z - bias[None, :]).std()
    assert 1.8 < spread < 2.3
    assert b.ids.min() >= 0 and b.ids.max() < 20000
    assert torch.all(b.logp_infer <= 0) and torch.all(b.logp_old <= 0)
    offs = b.offsets.numpy()
    assert offs[0] == 0 and offs[-1] == 256 and np.all(np.diff(offs) > 0)
    assert abs(b.scale + 1.0 / 256) < 1e-15
