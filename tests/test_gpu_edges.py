"""Edge cases of the HIP path against the CPU oracle: ragged and tiny vocabularies, every
row-kernel variant (register-resident and streamed rows), row strides, empty and fully masked
batches, invalid ids, extreme probabilities, kappa = 0, lambda = 0, in-place gradients, float32
logits, the elementwise weight kernel, and argument errors raised through the binding."""

import math

import numpy as np
import pytest
import torch

import paper_2609_32444_amd as cis
from oracle import cis as O
from tests import parity as P
from workloads import make_random_batch

pytestmark = pytest.mark.gpu
DEV = "cuda"


def run_and_check(b, bwd=True, report=None, **kw):
    fn = cis.loss_bwd if bwd else cis.loss_fwd
    out = fn(b.logits, b.ids, b.logp_infer, b.adv, b.mask, lam=b.lam, kappa=b.kappa,
             scale=b.scale, V=b.V, **kw)
    torch.cuda.synchronize()
    report = {} if report is None else report
    ref = P.oracle_for_batch(b, with_grad=False, grad=out["dlogits"] if bwd else None)
    P.compare_scalars(out, ref, b, report)
    P.compare_loss(out, ref, report)
    if bwd:
        P.check_grad_stats(ref["grad_stats"], report)
    st = cis.read_stats(out["workspace"])
    assert st["n_valid"] == int(((ref["flags"] & O.FLAG_VALID) > 0).sum())
    assert st["n_bad_id"] == int(((ref["flags"] & O.FLAG_BAD_ID) > 0).sum())
    return out, ref, report


# V values chosen to hit every row-kernel variant of both element types, ragged last vectors
# (V % 8 != 0), single partial vectors, and rows longer than the register-resident capacity.
# Fused-pass row capacities in 16-byte vectors: 128, 256, 512, 1024, 2048, 4096, 8192, 12288,
# 16384, 19456 in registers, then 27648 with LDS (bf16: 8 logits per vector, fp32: 4); longer
# rows stream the rest. The lists put rows in every variant, at and just past capacities.
BF16_VS = [1, 2, 7, 8, 9, 1000, 1001, 2048, 2049, 4097, 8192, 12000, 16384, 30000, 32768,
           40961, 65536, 90001, 100000, 130001, 151936, 155648, 155649, 160000, 200000, 200003,
           221184, 221185, 250001]
F32_VS = [1, 3, 4, 5, 1024, 2000, 3000, 4097, 20000, 30001, 45001, 60001, 70000, 77825, 90001,
          110592, 130001]


@pytest.mark.parametrize("V", BF16_VS)
def test_bf16_vocab_sizes(V):
    ld = ((V + 7) // 8) * 8 + (8 if V % 3 == 0 else 0)
    T = 24 if V <= 70000 else 8
    b = make_random_batch(T, V, torch.bfloat16, DEV, seed=V, ld=ld, mask_p=0.85)
    run_and_check(b)


@pytest.mark.parametrize("V", F32_VS)
def test_f32_vocab_sizes(V):
    ld = ((V + 3) // 4) * 4
    b = make_random_batch(16, V, torch.float32, DEV, seed=V + 1, ld=ld, mask_p=0.85)
    run_and_check(b)


@pytest.mark.parametrize("V,dtype", [(200003, torch.bfloat16), (90001, torch.float32)])
def test_long_rows_many_per_workgroup(V, dtype):
    # more rows than resident workgroups: each workgroup refills its LDS slots row after row
    epv = 8 if dtype == torch.bfloat16 else 4
    ld = ((V + epv - 1) // epv) * epv
    b = make_random_batch(600, V, dtype, DEV, seed=V + 7, ld=ld, mask_p=0.9)
    run_and_check(b)


# Fused-pass rows come from a queue once every workgroup has had two rows. The row counts put
# thousands of rows in the queue for the one-wave, 512-thread, 1024-thread and LDS variants
# (resident grids of up to 7168, 768, 256 and 256 workgroups). The queue is eight counters, each
# handing out every eighth row; 515 and 517 rows of 151936 leave 3 and 5 queued rows on a grid
# of 256, so most counters are empty from the start and the workgroups on them must move on.
@pytest.mark.parametrize("V,T", [(1000, 20000), (32768, 4096), (151936, 1500), (250001, 700),
                                 (151936, 515), (151936, 517)])
def test_row_queue_and_stale_workspace(V, T):
    """The workspace starts as all 0xFF bytes: as the row queue's counter that would hand out
    no queued row at all, so the call must clear it itself. Every row (15% masked) against the
    oracle, then a second call on the same workspace gives identical bits."""
    b = make_random_batch(T, V, torch.bfloat16, DEV, seed=V + 11, ld=((V + 7) // 8) * 8,
                          mask_p=0.85)
    ws = torch.full((cis.workspace_bytes(T),), 255, dtype=torch.uint8, device=DEV)
    out, _, _ = run_and_check(b, workspace=ws)
    g1 = out["dlogits"].clone()
    t1 = out["terms"].clone()
    out2 = cis.loss_bwd(b.logits, b.ids, b.logp_infer, b.adv, b.mask, lam=b.lam, kappa=b.kappa,
                        scale=b.scale, V=b.V, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(out2["dlogits"].view(torch.int16), g1.view(torch.int16))
    assert torch.equal(out2["terms"], t1)


# Forward pass: rows of fewer than 2048 16-byte vectors go through the row kernel (capacities
# 128, 256, 512, 1024, 2048 vectors); rows of 2048 up to 131072 vectors through the split
# kernels (segments of 1024, 2048 or 4096 vectors, at most 32 per row); longer rows through the
# streamed row kernel. The list puts rows at and just past each boundary, with ragged ends.
@pytest.mark.parametrize("V,dtype", [(V, torch.bfloat16) for V in
                                     (1000, 2048, 4000, 8000, 16000, 16384, 16392, 30001, 60000,
                                      90001, 131080, 151936, 155649, 262144, 262152, 524296,
                                      1048576, 1048584)] +
                                    [(V, torch.float32) for V in (1000, 8192, 16000, 60001, 65537,
                                                                  131072, 131076)])
def test_forward_only_matches(V, dtype):
    epv = 8 if dtype == torch.bfloat16 else 4
    ld = ((V + epv - 1) // epv) * epv
    b = make_random_batch(12, V, dtype, DEV, seed=5, mask_p=0.8, ld=ld)
    run_and_check(b, bwd=False)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_largest_vocabulary(dtype):
    """V = 2^28, the largest the ABI accepts (a row's byte offsets stay within 32 bits; 2^28 + 1
    is refused, tests/test_abi_cpu.py): two rows of 512 MB (bf16) or 1 GB (float32) through the
    streamed row path, fused and forward only, every element against the oracle."""
    b = make_random_batch(2, 1 << 28, dtype=dtype, device=DEV, seed=71)
    run_and_check(b)
    run_and_check(b, bwd=False)


def test_empty_batch():
    b = make_random_batch(1, 16, torch.bfloat16, DEV, seed=1)
    z = b.logits[:0]
    e64 = torch.empty(0, dtype=torch.int64, device=DEV)
    e32 = torch.empty(0, dtype=torch.float32, device=DEV)
    out = cis.loss_bwd(z, e64, e32, e32, None, lam=1.0, kappa=5e-3, scale=1.0, V=16)
    torch.cuda.synchronize()
    assert out["loss"].item() == 0.0 and out["dlogits"].shape == (0, 16)
    assert cis.read_stats(out["workspace"])["n_valid"] == 0


@pytest.mark.parametrize("V,bwd", [(3000, True), (3000, False), (40000, False)])
def test_all_masked_and_invalid_ids(V, bwd):
    """(V = 40000 runs the forward pass through the split-row kernels.)"""
    b = make_random_batch(32, V, torch.bfloat16, DEV, seed=2)
    b.mask.zero_()
    out, ref, _ = run_and_check(b, bwd=bwd)
    assert out["loss"].item() == 0.0
    if bwd:
        assert torch.count_nonzero(out["dlogits"]) == 0
    b = make_random_batch(32, V, torch.bfloat16, DEV, seed=3)
    b.ids[::3] = -1
    b.ids[1::5] = V
    b.ids[2::7] = 1 << 40
    out, ref, _ = run_and_check(b, bwd=bwd)
    st = cis.read_stats(out["workspace"])
    assert st["n_bad_id"] > 0
    bad = ((b.ids < 0) | (b.ids >= V)) & (b.mask > 0)
    if bwd:
        assert torch.count_nonzero(out["dlogits"][bad]) == 0


@pytest.mark.parametrize("V,bwd", [(5000, True), (5000, False), (151936, True), (151936, False)])
def test_confident_rows_and_extremes(V, bwd):
    """p -> 1 (1 - p down to ~1e-30), l_infer = -inf, z_y = -inf, -inf and huge-negative logits;
    fused and forward only, on short rows and on rows of the split forward pass."""
    T = 16
    b = make_random_batch(T, V, torch.bfloat16, DEV, seed=4, mask_p=1.0)
    z = b.logits
    y = b.ids
    for t, gap in enumerate([5, 10, 15, 20, 30, 40, 60, 80]):
        z[t, y[t]] = float(z[t].float().max()) + gap
    b.logp_infer[8] = -math.inf
    z[9, y[9]] = -math.inf
    z[10, ::2] = -math.inf
    z[10, y[10]] = 1.0
    z[11, :] = -3.0e38
    z[11, y[11]] = 0.5
    z[12, 7] = -math.inf
    b.logp_infer[13] = 0.0
    out, ref, rep = run_and_check(b, bwd=bwd)
    assert out["w"][9].item() == 0.0 and out["trunc"][8].item() == 1
    for t in range(8):
        lt = out["logp_train"][t].item()
        assert lt <= 0


@pytest.mark.parametrize("kappa,c", [(0.0, 1.0), (0.0, 0.25), (5e-3, 0.0), (1.0, 1.0),
                                     (0.1, 3.0), (5e-3, 30.0)])
def test_threshold_and_floor_settings(kappa, c):
    b = make_random_batch(64, 4096, torch.bfloat16, DEV, seed=int(100 * kappa + 10 * c),
                          delta_sd=1.5, c=c, kappa=kappa)
    # make a third of the rows confident so that the floor matters
    rows = torch.arange(0, 64, 3, device=DEV)
    b.logits[rows, b.ids[rows]] = b.logits[rows].float().max(dim=1).values.to(torch.bfloat16) + 9
    out, ref, rep = run_and_check(b)
    if c == 0.0:
        w = out["w"].cpu().numpy()
        k = np.exp(out["logp_train"].cpu().double().numpy() - b.logp_infer.cpu().double().numpy())
        assert np.allclose(w, np.minimum(k, 1.0), rtol=1e-5)


@pytest.mark.parametrize("V,ld", [(9001, 9008), (151936, 151936), (200003, 200016)])
def test_in_place_gradient(V, ld):
    # The gradient overwrites the logits row by row (each element is read before the same
    # thread writes it). Checked against the oracle on the original logits, and bit for bit
    # against a separate output buffer.
    b = make_random_batch(40, V, torch.bfloat16, DEV, seed=9, ld=ld)
    store = torch.empty(2, 40, ld, dtype=torch.bfloat16, device=DEV)
    store[0, :, :V] = b.logits
    buf = store[0, :, :V]
    sep = store[1, :, :V]
    ref_out = cis.loss_bwd(buf, b.ids, b.logp_infer, b.adv, b.mask, lam=b.lam, kappa=b.kappa,
                           scale=b.scale, V=V, dlogits=sep)
    torch.cuda.synchronize()
    ref = P.oracle_for_batch(b, with_grad=False, grad=ref_out["dlogits"])
    out = cis.loss_bwd(buf, b.ids, b.logp_infer, b.adv, b.mask, lam=b.lam, kappa=b.kappa,
                       scale=b.scale, V=V, dlogits=buf)
    torch.cuda.synchronize()
    rep = {}
    P.check_grad_stats(ref["grad_stats"], rep)
    ref_ip = P.oracle_for_batch(b, with_grad=False, grad=buf)
    P.check_grad_stats(ref_ip["grad_stats"], rep)
    P.compare_scalars(out, ref_ip, b, rep)
    assert torch.equal(buf.view(torch.int16), sep.view(torch.int16))
    assert torch.equal(out["w"], ref_out["w"])


def test_padding_columns_untouched():
    V, ld = 1001, 1016
    b = make_random_batch(8, V, torch.bfloat16, DEV, seed=11, ld=ld)
    g = torch.full((8, ld), 7.0, dtype=torch.bfloat16, device=DEV)
    cis.loss_bwd(b.logits, b.ids, b.logp_infer, b.adv, b.mask, lam=b.lam, kappa=b.kappa,
                 scale=b.scale, V=V, dlogits=g)
    torch.cuda.synchronize()
    assert torch.all(g[:, V:] == 7.0)


def test_weights_kernel_matches_oracle():
    rng = np.random.default_rng(0)
    n = 100003
    lt = -np.abs(rng.normal(0, 2, n)) * rng.choice([1e-9, 1e-4, 1e-2, 1, 3], n)
    li = lt - rng.normal(0, 1.0, n)
    li[::1000] = -np.inf
    mask = (rng.random(n) > 0.1).astype(np.uint8)
    lt32, li32 = lt.astype(np.float32), li.astype(np.float32)
    for lam, kappa in [(2.3, 5e-3), (math.e - 1, 0.0), (0.0, 5e-3), (6.0, 1.0)]:
        w, tr = cis.weights(torch.from_numpy(lt32).to(DEV), torch.from_numpy(li32).to(DEV),
                            torch.from_numpy(mask).to(DEV), lam=lam, kappa=kappa)
        w64, tr64 = O.cis_weights(lt32.astype(np.float64), li32.astype(np.float64), mask,
                                  float(np.float32(lam)), float(np.float32(kappa)))
        w = w.cpu().double().numpy()
        tr = tr.cpu().numpy().astype(bool)
        assert np.all(np.abs(w - w64) <= 1e-5 * np.abs(w64) + 1e-38)
        phi = np.maximum(-np.expm1(lt32.astype(np.float64)), np.float32(kappa))
        margin = np.abs((lt32.astype(np.float64) - li32) - np.log1p(np.float32(lam) * phi))
        assert np.all((tr == tr64) | (margin < 1e-5))


def test_weights_beyond_2_31_tokens():
    """T = 2^31 + 2^24 tokens (about 30 GB of device arrays): the elementwise weights kernel
    indexes in 64 bits. Outputs are compared with the oracle on the first and last 2^20 tokens
    and on 2^20 random ones."""
    T = (1 << 31) + (1 << 24)
    g = torch.Generator(device=DEV)
    g.manual_seed(5)
    lt = torch.rand(T, generator=g, device=DEV).mul_(-6.0)          # log p in (-6, 0]
    li = torch.randn(T, generator=g, device=DEV).neg_().add_(lt)    # log q = log p - N(0, 1)
    mask = (torch.rand(T, generator=g, device=DEV) > 0.1).to(torch.uint8)
    lam, kappa = 2.3, 5e-3
    w, tr = cis.weights(lt, li, mask, lam=lam, kappa=kappa)
    idx = torch.cat([torch.arange(0, 1 << 20, device=DEV),
                     torch.arange(T - (1 << 20), T, device=DEV),
                     torch.randint(0, T, (1 << 20,), generator=g, device=DEV)])
    lt64, li64 = lt[idx].double().cpu().numpy(), li[idx].double().cpu().numpy()
    m = mask[idx].cpu().numpy()
    w64, tr64 = O.cis_weights(lt64, li64, m, float(np.float32(lam)), float(np.float32(kappa)))
    wg = w[idx].double().cpu().numpy()
    tg = tr[idx].cpu().numpy().astype(bool)
    assert np.all(np.abs(wg - w64) <= 1e-5 * np.abs(w64) + 1e-38)
    phi = np.maximum(-np.expm1(lt64), np.float32(kappa))
    margin = np.abs((lt64 - li64) - np.log1p(np.float32(lam) * phi))
    assert np.all((tg == tr64) | (margin < 1e-5))


def test_binding_errors():
    b = make_random_batch(4, 64, torch.bfloat16, DEV, seed=1)
    with pytest.raises(cis.CisError) as e:
        cis.loss_fwd(b.logits, b.ids, b.logp_infer, b.adv, b.mask, lam=-1.0)
    assert e.value.status == -4
    with pytest.raises(cis.CisError) as e:
        cis.loss_bwd(b.logits, b.ids, b.logp_infer, b.adv, b.mask, lam=1.0, kappa=2.0)
    assert e.value.status == -4
    odd = torch.zeros(4, 63, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(cis.CisError) as e:
        cis.loss_fwd(odd, b.ids, b.logp_infer, b.adv, None, lam=1.0)
    assert e.value.status == -5
    with pytest.raises(ValueError):
        cis.loss_fwd(b.logits, b.ids.int(), b.logp_infer, b.adv, b.mask, lam=1.0)
