"""Concurrent calls on two streams.

The library keeps no device state of its own between or during calls: everything a call writes
lives in the caller's outputs and workspace (the LM head's work queues included). Two calls on
two streams, each with its own workspace, may therefore run at the same time. Each test runs two
different batches concurrently and compares every output, bit for bit, with the same calls
made one after the other on the default stream.
"""

import pytest
import torch

import paper_2609_32444_amd as cis
from workloads import make_lmhead_batch, make_random_batch

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _same(a, b):
    return a.shape == b.shape and torch.equal(a.view(torch.uint8), b.view(torch.uint8))


def _concurrent(calls):
    """Runs each zero-argument call on a stream of its own (default priority) and waits."""
    cur = torch.cuda.current_stream()
    streams = [torch.cuda.Stream() for _ in calls]
    outs = []
    for s, call in zip(streams, calls):
        s.wait_stream(cur)
        with torch.cuda.stream(s):
            outs.append(call())
    for s in streams:
        cur.wait_stream(s)
    torch.cuda.synchronize()
    return outs


def test_fused_loss_on_two_streams():
    batches = [make_random_batch(2048, 32000, device=DEV, seed=s, mask_p=0.9, ld=32000)
               for s in (41, 42)]
    calls = [cis.LossCall(b.logits, b.ids, b.logp_infer, b.adv, b.mask, lam=b.lam,
                          kappa=b.kappa, scale=b.scale) for b in batches]
    seq = []
    for c in calls:
        seq.append({k: v.clone() for k, v in c.run().items() if k != "workspace"})
    torch.cuda.synchronize()
    for rep in range(3):
        outs = _concurrent([c.run for c in calls])
        for i, (o, ref) in enumerate(zip(outs, seq)):
            for k, v in ref.items():
                assert _same(o[k], v), f"repeat {rep}, call {i}: {k} differs"


def test_lmhead_on_two_streams():
    """Queued products (274 tiles) in both calls: each call's work queues are its own."""
    batches = [make_lmhead_batch(256, 70000, 256, device=DEV, seed=s, min_len=16, max_len=96)
               for s in (43, 44)]
    prms = [cis.params(cis.OP_CIS, lam=b.lam, kappa=b.kappa, scale=b.scale) for b in batches]

    def call(i):
        b = batches[i]
        return lambda: cis.lmhead_loss_bwd(b.hidden, b.weight, b.ids, b.logp_infer, b.adv,
                                           b.mask, params=prms[i], chunk=128)

    seq = [call(i)() for i in range(2)]
    torch.cuda.synchronize()
    keys = ("logp_train", "w", "acted", "terms", "eps", "loss", "dhidden", "dweight")
    for rep in range(2):
        outs = _concurrent([call(0), call(1)])
        for i, (o, ref) in enumerate(zip(outs, seq)):
            for k in keys:
                assert _same(o[k], ref[k]), f"repeat {rep}, call {i}: {k} differs"
