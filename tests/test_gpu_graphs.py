"""HIP graph capture of the library's calls.

A call launches on the caller's stream and allocates, clears and synchronizes nothing itself (the
product queues are cleared by a kernel, not a memset), so a captured call can be replayed. Each
test captures one call, then replays it five times with eager work and a synchronization
between replays. Twice the captured inputs are rewritten in place with a second batch, and then
restored. Every replay must equal, bit for bit, an eager call on the same data; the kernels are
deterministic.
"""

import pytest
import torch

import paper_2609_32444_amd as cis
from workloads import make_lmhead_batch, make_random_batch

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _same(a, b):
    """Bitwise equality (NaN-safe): both tensors viewed as bytes."""
    return a.shape == b.shape and torch.equal(a.view(torch.uint8), b.view(torch.uint8))


def _clone(t):
    """A copy with the same row stride (a padded [T, V] view stays padded; clone() would pack
    it)."""
    if t.dim() == 2 and t.stride(0) != t.shape[1]:
        base = torch.empty((t.shape[0], t.stride(0)), dtype=t.dtype, device=t.device)
        view = base[:, :t.shape[1]]
        view.copy_(t)
        return view
    return t.clone()


def _eager_work():
    x = torch.randn(512, 512, device=DEV)
    float((x @ x).sum().item())  # a library product, a reduction and a synchronization


def _capture(fn):
    """Warm-up on a side stream (torch's recipe), then capture fn(); returns (graph, outputs)."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out = fn()
    torch.cuda.synchronize()
    return g, out


def _replay_and_compare(g, out, inputs, datasets, eager, keys):
    """inputs: the captured input tensors; datasets: tuples of tensors of the same shapes copied
    into them in turn; eager(data) computes the reference on separate buffers."""
    originals = tuple(_clone(t) for t in inputs)
    refs = {}
    for rep, which in enumerate((0, 0, 1, 1, 0)):
        data = originals if which == 0 else datasets[which - 1]
        for dst, src in zip(inputs, data):
            dst.copy_(src)
        if which not in refs:
            refs[which] = eager(tuple(_clone(t) for t in data))
            torch.cuda.synchronize()
        _eager_work()
        g.replay()
        torch.cuda.synchronize()
        for k in keys:
            assert _same(out[k], refs[which][k]), f"replay {rep} (data set {which}): {k} differs"
    for dst, src in zip(inputs, originals):
        dst.copy_(src)


# (700 rows of 5003: every row is a workgroup's first or second; 3000 rows of 151936 on the
# 256-workgroup grid: 2488 rows come from the row queue, whose counter the captured call
# clears with a kernel node on every replay)
@pytest.mark.parametrize("dtype,T,V,ld", [(torch.bfloat16, 700, 5003, 5008),
                                          (torch.float32, 700, 5003, 5008),
                                          (torch.bfloat16, 3000, 151936, 151936)])
def test_fused_loss_graph_replays(dtype, T, V, ld):
    b = make_random_batch(T, V, dtype=dtype, device=DEV, seed=21, mask_p=0.9, ld=ld)
    b2 = make_random_batch(T, V, dtype=dtype, device=DEV, seed=22, mask_p=0.9, ld=ld)
    kw = dict(lam=b.lam, kappa=b.kappa, scale=b.scale)  # baked into the graph: kept for b2 too
    call = cis.LossCall(b.logits, b.ids, b.logp_infer, b.adv, b.mask, **kw)
    g, out = _capture(call.run)
    inputs = (b.logits, b.ids, b.logp_infer, b.adv, b.mask)

    def eager(d):
        logits, ids, linf, adv, mask = d
        return cis.LossCall(logits, ids, linf, adv, mask, **kw).run()

    _replay_and_compare(g, out, inputs, [(b2.logits, b2.ids, b2.logp_infer, b2.adv, b2.mask)],
                        eager, ("logp_train", "w", "trunc", "terms", "loss", "dlogits"))


def test_decoupled_loss_graph_replays():
    T, V, ld = 600, 7001, 7008
    b = make_random_batch(T, V, device=DEV, seed=31, mask_p=0.95, ld=ld)
    b2 = make_random_batch(T, V, device=DEV, seed=32, mask_p=0.95, ld=ld)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(33)
    old = (b.logp_infer + 0.3 * torch.randn(T, device=DEV, generator=gen)).clamp(max=0.0)
    old2 = (b2.logp_infer + 0.3 * torch.randn(T, device=DEV, generator=gen)).clamp(max=0.0)
    prm = cis.params(cis.OP_CIS, lam=b.lam, kappa=b.kappa, clip_low=0.2, clip_high=0.28,
                     scale=b.scale)
    call = cis.LossCall(b.logits, b.ids, b.logp_infer, b.adv, b.mask, params=prm, logp_old=old)
    g, out = _capture(call.run)
    inputs = (b.logits, b.ids, b.logp_infer, b.adv, b.mask, old)

    def eager(d):
        logits, ids, linf, adv, mask, lold = d
        return cis.LossCall(logits, ids, linf, adv, mask, params=prm, logp_old=lold).run()

    _replay_and_compare(g, out, inputs,
                        [(b2.logits, b2.ids, b2.logp_infer, b2.adv, b2.mask, old2)], eager,
                        ("logp_train", "w", "trunc", "terms", "loss", "dlogits"))


def test_lmhead_graph_replays():
    """Two chunks of 128 rows; the logits and dL/dW products have 274 tiles (more than the
    CUs: work queues cleared inside the graph) and dL/dh is split along V (partials and their
    reduction inside the graph)."""
    T, V, H, chunk = 256, 70000, 256, 128
    b = make_lmhead_batch(T, V, H, device=DEV, seed=23, min_len=16, max_len=96)
    b2 = make_lmhead_batch(T, V, H, device=DEV, seed=24, min_len=16, max_len=96)
    prm = cis.params(cis.OP_CIS, lam=b.lam, kappa=b.kappa, scale=b.scale)
    inputs = (b.hidden, b.weight, b.ids, b.logp_infer, b.adv, b.mask)

    def run(d=inputs):
        return cis.lmhead_loss_bwd(*d, params=prm, chunk=chunk)

    g, out = _capture(run)
    _replay_and_compare(g, out, inputs,
                        [(b2.hidden, b2.weight, b2.ids, b2.logp_infer, b2.adv, b2.mask)], run,
                        ("logp_train", "w", "acted", "terms", "eps", "loss", "dhidden",
                         "dweight"))
