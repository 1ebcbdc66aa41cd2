"""The C-ABI library on the host: it loads, exports every entry point include/cis.h declares,
and rejects bad arguments before touching a device. No kernel is launched here."""

import ctypes
import os
import re

import pytest
import torch

import paper_2609_32444_amd as cis
from paper_2609_32444_amd import _binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cis.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(cis_\w+)\s*\(", text, flags=re.M)))


def test_probe_library_exports():
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2609_32444_amd", "libcis_probe.so"))
    assert hasattr(lib, "cis_probe_bandwidth")


def test_library_exports_every_declared_symbol():
    lib = cis.load_library()
    names = declared_functions()
    assert set(names) == {"cis_workspace_bytes", "cis_workspace_bytes_ex", "cis_status_string",
                          "cis_weights", "cis_weights_ex", "cis_loss_fwd", "cis_loss_bwd",
                          "cis_loss_fwd_ex", "cis_loss_bwd_ex", "cis_lmhead_workspace_bytes",
                          "cis_lmhead_loss_fwd", "cis_lmhead_loss_bwd", "cis_loss_bwd_noalloc"}
    for n in names:
        assert hasattr(lib, n), n


def test_workspace_bytes_layout():
    assert cis.workspace_bytes(-1) == 0
    assert cis.workspace_bytes(0) == 1280  # statistics and the row-queue counters
    for T in (1, 255, 256, 16384, 65536, 524288):
        n = cis.workspace_bytes(T)
        # stats, four float arrays and two byte arrays per row, and the forward pass's
        # per-segment partials (32 float pairs) and sampled logit per row
        assert n % 256 == 0 and n >= 1280 + (18 + 32 * 8 + 4) * T
        assert cis.workspace_bytes_ex(T, 0) == n
        assert cis.workspace_bytes_ex(T, 1000) >= n + 8 * 1000
    assert cis.workspace_bytes_ex(-1, 0) == 0 and cis.workspace_bytes_ex(4, -1) == 0


def test_status_strings():
    for code in range(0, -10, -1):
        s = cis.status_string(code)
        assert s and s != "unknown status"
    assert cis.status_string(-99) == "unknown status"


NULL = None
FAKE = 0x10000   # a 16-byte aligned non-null address; never dereferenced on these paths


def _fwd(**kw):
    a = dict(logits=FAKE, dtype=0, T=4, V=8, ld=8, ids=FAKE, linf=FAKE, adv=FAKE, mask=NULL,
             lam=1.0, kappa=5e-3, scale=-0.25, lt=NULL, w=NULL, tr=NULL, terms=NULL, loss=NULL,
             ws=FAKE, wsb=1 << 20, stream=NULL)
    a.update(kw)
    return cis.load_library().cis_loss_fwd(
        a["logits"], a["dtype"], a["T"], a["V"], a["ld"], a["ids"], a["linf"], a["adv"],
        a["mask"], a["lam"], a["kappa"], a["scale"], a["lt"], a["w"], a["tr"], a["terms"],
        a["loss"], a["ws"], a["wsb"], a["stream"])


def _bwd(**kw):
    a = dict(logits=FAKE, dtype=0, T=4, V=8, ld=8, ids=FAKE, linf=FAKE, adv=FAKE, mask=NULL,
             lam=1.0, kappa=5e-3, scale=-0.25, dl=FAKE * 16, ldg=8, ws=FAKE, wsb=1 << 20)
    a.update(kw)
    return cis.load_library().cis_loss_bwd(
        a["logits"], a["dtype"], a["T"], a["V"], a["ld"], a["ids"], a["linf"], a["adv"],
        a["mask"], a["lam"], a["kappa"], a["scale"], a["dl"], a["ldg"], NULL, NULL, NULL, NULL,
        NULL, a["ws"], a["wsb"], NULL)


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=7), -3),
    (dict(T=-1), -2), (dict(V=0), -2), (dict(ld=7), -2),
    (dict(V=(1 << 28) + 1, ld=(1 << 28) + 8), -2),
    (dict(lam=-1.0), -4), (dict(lam=float("inf")), -4), (dict(lam=float("nan")), -4),
    (dict(kappa=-0.1), -4), (dict(kappa=1.5), -4), (dict(scale=float("nan")), -4),
    (dict(ws=NULL), -1), (dict(logits=NULL), -1), (dict(ids=NULL), -1), (dict(adv=NULL), -1),
    (dict(linf=NULL), -1),
    (dict(ws=FAKE + 16), -5), (dict(logits=FAKE + 2), -5), (dict(V=7, ld=7), -5),
    (dict(wsb=100), -7),
])
def test_fwd_argument_errors(kw, code):
    assert _fwd(**kw) == code


@pytest.mark.parametrize("kw,code", [
    (dict(dl=NULL), -1), (dict(ldg=4), -2), (dict(dl=FAKE * 16 + 8), -5),
    (dict(ldg=12), -5),                              # 24-byte row stride
    (dict(dl=FAKE, ldg=16), -8),                     # same base, different stride
    (dict(dl=FAKE + 32), -8),                        # partial overlap
])
def test_bwd_argument_errors(kw, code):
    assert _bwd(**kw) == code


def test_weights_argument_errors():
    lib = cis.load_library()
    assert lib.cis_weights(FAKE, FAKE, NULL, -1, 1.0, 0.0, FAKE, NULL, NULL) == -2
    assert lib.cis_weights(FAKE, FAKE, NULL, 4, -1.0, 0.0, FAKE, NULL, NULL) == -4
    assert lib.cis_weights(FAKE, FAKE, NULL, 4, 1.0, 2.0, FAKE, NULL, NULL) == -4
    assert lib.cis_weights(NULL, FAKE, NULL, 4, 1.0, 0.0, FAKE, NULL, NULL) == -1
    assert lib.cis_weights(FAKE, FAKE, NULL, 4, 1.0, 0.0, NULL, NULL, NULL) == -1
    assert lib.cis_weights(NULL, NULL, NULL, 0, 1.0, 0.0, NULL, NULL, NULL) == 0


def test_binding_raises_cis_error_type():
    e = _binding.CisError("cis_loss_fwd", -4)
    assert e.status == -4 and "lambda" in str(e)


def test_lambda_from_logodds():
    import math
    assert cis.lambda_from_logodds(0.0) == 0.0
    assert abs(cis.lambda_from_logodds(1.0) - (math.e - 1)) < 1e-15
    assert abs(cis.lambda_from_logodds(math.log(3.3)) - 2.3) < 1e-12


def _prm(**kw):
    p = cis.params(cis.OP_CIS, scale=-0.25)
    for k, v in kw.items():
        setattr(p, k, v)
    return p


def _fwd_ex(prm, **kw):
    a = dict(logits=FAKE, dtype=0, T=4, V=8, ld=8, ids=FAKE, linf=FAKE, lold=NULL, adv=FAKE,
             mask=NULL, offs=NULL, nseq=0, ws=FAKE, wsb=1 << 20)
    a.update(kw)
    pp = ctypes.byref(prm) if prm is not None else None
    return cis.load_library().cis_loss_fwd_ex(
        a["logits"], a["dtype"], a["T"], a["V"], a["ld"], a["ids"], a["linf"], a["lold"],
        a["adv"], a["mask"], a["offs"], a["nseq"], pp, NULL, NULL, NULL, NULL, NULL, NULL,
        a["ws"], a["wsb"], NULL)


@pytest.mark.parametrize("prm,kw,code", [
    (None, {}, -1),
    (dict(op=10), {}, -4), (dict(op=-1), {}, -4), (dict(scale=float("inf")), {}, -4),
    (dict(lam=-1.0), {}, -4), (dict(kappa=2.0), {}, -4),
    (dict(op=2, lo=2.0, hi=1.0), {}, -4), (dict(op=2, lo=-1.0, hi=1.0), {}, -4),
    (dict(op=4, lo=float("nan"), hi=1.0), {}, -4), (dict(op=3, hi=-1.0), {}, -4),
    (dict(op=5, hi=float("nan")), {}, -4), (dict(op=7, lam=float("inf")), {}, -4),
    # sequence operators need logp_old, and responses
    (dict(op=8, hi=2.0), {}, -4),
    (dict(op=9, lo=0.5, hi=2.0), dict(lold=FAKE, nseq=0), -2),
    (dict(op=8, hi=2.0), dict(lold=FAKE, nseq=2), -1),
    (dict(op=8, hi=2.0), dict(lold=FAKE, nseq=-1), -2),
    # the decoupled path checks the PPO clip
    (dict(clip_low=1.5), dict(lold=FAKE), -4), (dict(clip_high=-0.1), dict(lold=FAKE), -4),
    (dict(clip_high=float("inf")), dict(lold=FAKE), -4),
    ({}, dict(wsb=100), -7), ({}, dict(ws=FAKE + 16), -5), ({}, dict(dtype=9), -3),
])
def test_fwd_ex_argument_errors(prm, kw, code):
    p = None if prm is None else _prm(**prm)
    assert _fwd_ex(p, **kw) == code


def test_fwd_ex_accepts_valid_arguments_up_to_the_device_check():
    # on a host without a gfx950 device, valid arguments get as far as CIS_ERR_DEVICE
    for op, extra in ((0, {}), (2, dict(lo=1e-6, hi=1e6)), (3, dict(hi=2.0)),
                      (4, dict(lo=0.5, hi=5.0)), (5, dict(hi=2.0)), (6, {}), (7, {}), (1, {})):
        assert _fwd_ex(_prm(op=op, **extra)) == -9
        assert _fwd_ex(_prm(op=op, **extra), lold=FAKE) == -9
    assert _fwd_ex(_prm(op=8, hi=2.0), lold=FAKE, offs=FAKE, nseq=2) == -9


def test_weights_ex_argument_errors():
    lib = cis.load_library()

    def call(prm, T=4, lp=FAKE, offs=NULL, nseq=0, w=FAKE, ws=FAKE, wsb=1 << 20):
        pp = ctypes.byref(prm) if prm is not None else None
        return lib.cis_weights_ex(lp, FAKE, NULL, T, offs, nseq, pp, w, NULL, NULL, ws, wsb, NULL)
    assert call(None) == -1
    assert call(_prm(), T=-1) == -2
    assert call(_prm(op=12)) == -4
    assert call(_prm(op=8, hi=2.0)) == -2           # sequence operator without responses
    assert call(_prm(op=8, hi=2.0), nseq=1) == -1   # ... or without offsets
    assert call(_prm(), lp=NULL) == -1
    assert call(_prm(), w=NULL) == -1
    assert call(_prm(), ws=NULL) == -1
    assert call(_prm(), ws=FAKE + 8) == -5
    assert call(_prm(), wsb=16) == -7
    assert call(_prm()) == -9


def test_lmhead_workspace_bytes():
    f = cis.lmhead_workspace_bytes
    T, V, H = 16384, 151936, 2048
    fwd, bwd = f(T, V, H, 4096, 0, False), f(T, V, H, 4096, 0, True)
    loss = 256 + 18 * T
    # the loss rows' scratch plus, per chunk row, one (max, exp-sum) pair per 64 columns, the
    # sampled logit and the gradient parameters: the logits themselves are never stored
    ntv = (V + 255) // 256 * 4
    assert fwd >= loss + 4096 * (8 * ntv + 4 + 16) and fwd % 256 == 0
    assert fwd < 4096 * V                       # far less than one float32 chunk of logits
    # the backward adds the chunk's float32 logits, W^T, the chunk's bf16 gradient and the two
    # transposed operands
    assert bwd >= fwd + 4 * 4096 * V + 2 * V * H + 2 * 4096 * V + 2 * (V + H) * 4096
    # a chunk larger than the batch only needs the batch's rows
    assert f(100, 1000, 64, 4096, 0, True) == f(100, 1000, 64, 100, 0, True)
    assert f(T, V, H, 4096, 10, True) >= bwd
    for bad in ((-1, V, H, 1), (T, 0, H, 1), (T, V, 0, 1), (T, V, H, 0), (T, (1 << 22) + 1, H, 1),
                (T, V, 1 << 17, 1), (T, V, H, 1 << 17)):
        assert f(*bad, 0, True) == 0, bad
    assert f(T, V, H, 64, -1, True) == 0
    # the backward that never stores the logits needs exactly one float32 chunk less
    rec = cis.lmhead_workspace_bytes(T, V, H, 4096, 0, True, recompute=True)
    assert 4 * 4096 * V <= bwd - rec <= 4 * 4096 * (V + 8) + 256
    assert rec >= fwd + 2 * V * H + 2 * 4096 * V
    assert cis.load_library().cis_lmhead_workspace_bytes(T, V, H, 4096, 0, 3) == 0


# distinct fake buffers for the LM-head calls, 4 GiB apart (never dereferenced)
LM_H, LM_W, LM_DH, LM_DW, LM_WS = (k << 32 for k in range(1, 6))


def _lm(bwd=True, **kw):
    a = dict(hidden=LM_H, T=4, H=64, ld_h=64, weight=LM_W, V=1000, ld_w=64, ids=FAKE, linf=FAKE,
             lold=NULL, adv=FAKE, mask=NULL, offs=NULL, nseq=0, prm=_prm(), chunk=4096,
             dh=LM_DH, ld_dh=64, dw=LM_DW, ld_dw=64, ws=LM_WS, wsb=1 << 30, recompute=0)
    a.update(kw)
    pp = ctypes.byref(a["prm"]) if a["prm"] is not None else None
    lib = cis.load_library()
    head = (a["hidden"], a["T"], a["H"], a["ld_h"], a["weight"], a["V"], a["ld_w"], a["ids"],
            a["linf"], a["lold"], a["adv"], a["mask"], a["offs"], a["nseq"], pp, a["chunk"])
    tail = (NULL, NULL, NULL, NULL, NULL, NULL, a["ws"], a["wsb"], NULL)
    if bwd:
        return lib.cis_lmhead_loss_bwd(*head, a["dh"], a["ld_dh"], a["dw"], a["ld_dw"], 0,
                                       a["recompute"], *tail)
    return lib.cis_lmhead_loss_fwd(*head, *tail)


@pytest.mark.parametrize("kw,code", [
    (dict(prm=None), -1), (dict(hidden=NULL), -1), (dict(weight=NULL), -1), (dict(ids=NULL), -1),
    (dict(dh=NULL), -1), (dict(dw=NULL), -1), (dict(ws=NULL), -1),
    (dict(T=-1), -2), (dict(V=0), -2), (dict(H=0), -2), (dict(ld_h=32), -2),
    (dict(ld_w=32), -2), (dict(ld_dh=32), -2), (dict(ld_dw=32), -2), (dict(chunk=0), -2),
    (dict(chunk=1 << 17), -2), (dict(H=1 << 17, ld_h=1 << 17, ld_w=1 << 17), -2),
    (dict(V=(1 << 22) + 1), -2), (dict(ld_h=(1 << 22) + 8), -2), (dict(ld_w=(1 << 22) + 8), -2),
    (dict(ld_h=68, H=60), -5), (dict(ld_w=68, H=60), -5), (dict(hidden=LM_H + 8), -5),
    (dict(weight=LM_W + 8), -5), (dict(ws=LM_WS + 16), -5), (dict(wsb=1000), -7),
    (dict(recompute=2), -4), (dict(recompute=-1), -4),
    (dict(prm=None), -1), (dict(lold=FAKE, prm=None), -1),
])
def test_lmhead_argument_errors(kw, code):
    assert _lm(True, **kw) == code


def test_lmhead_fwd_needs_no_gradient_buffers():
    # the forward ignores dhidden / dweight; valid arguments reach the device check
    assert _lm(False, dh=NULL, dw=NULL) == -9
    assert _lm(True) == -9
    # no rows: hidden and the per-row arrays may be NULL, dweight is still written
    assert _lm(True, T=0, hidden=NULL, ids=NULL, linf=NULL, adv=NULL, dh=NULL) == -9
    assert _lm(True, T=0, dw=NULL) == -1
    # H not a multiple of 8 with a padded row stride is fine
    assert _lm(True, H=60, ld_h=64, ld_w=64) == -9
    # a sequence operator needs logp_old and responses
    assert _lm(True, prm=_prm(op=8, hi=2.0)) == -4
    assert _lm(True, prm=_prm(op=8, hi=2.0), lold=FAKE, nseq=2, offs=FAKE) == -9


def test_lmhead_gradient_overlaps():
    V, ld = 1000, 64
    w_end = LM_W + V * ld * 2                       # one past weight's last byte
    assert _lm(True, dh=LM_H) == -8                 # dL/dh over hidden
    assert _lm(True, dw=LM_W) == -8                 # dL/dW over weight
    assert _lm(True, dw=w_end - 16) == -8           # dL/dW starting in weight's last row
    assert _lm(True, dw=LM_WS + 4096) == -8         # inside the workspace
    assert _lm(True, dh=LM_DW + 1024) == -8         # the two gradients overlap
    assert _lm(True, dh=LM_DW - 16) == -8           # dL/dh runs into dL/dW
    assert _lm(True, dw=w_end) == -9                # adjacent is fine
    assert _lm(True, dw=LM_H - V * ld * 4) == -9    # ends right where hidden starts
    # no rows: dL/dh is not written, so it may sit anywhere; the forward writes neither
    assert _lm(True, T=0, hidden=NULL, ids=NULL, linf=NULL, adv=NULL, dh=LM_W) == -9
    assert _lm(False, dh=LM_H, dw=LM_W) == -9


def test_lmhead_binding_rejects_accumulating_into_nothing():
    import torch
    h = torch.zeros(4, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        cis.lmhead_loss_bwd(h, torch.zeros(10, 64, dtype=torch.bfloat16),
                            torch.zeros(4, dtype=torch.int64), torch.zeros(4), torch.zeros(4),
                            params=cis.params(), accumulate=True)


def test_binding_rejects_a_vocabulary_wider_than_the_logits():
    """V may not exceed the logits' columns (the kernel would read past each row, and for a
    single row past the tensor); it is checked before anything touches a device."""
    z = torch.zeros(1, 8, dtype=torch.bfloat16)
    for V in (9, 1 << 20, 0, -1):
        with pytest.raises(ValueError, match="V must be in"):
            _binding._logits_args(z, V)
    z4 = torch.zeros(4, 16, dtype=torch.float32)[:, :12]
    with pytest.raises(ValueError, match="V must be in"):
        _binding._logits_args(z4, 13)
    # in range, the host tensor is refused only as not being a device tensor
    with pytest.raises(ValueError, match="device tensor"):
        _binding._logits_args(z4, 12)


def test_noalloc_rejects_more_rows_than_its_scratch_holds():
    """cis_loss_bwd_noalloc refuses T > CIS_NOALLOC_MAX_T before anything else (no device is
    needed to see it), and says why."""
    lib = cis.load_library()
    T = cis.NOALLOC_MAX_T + 1
    rc = lib.cis_loss_bwd_noalloc(FAKE, 0, T, 8, 8, FAKE, FAKE, FAKE, NULL, 1.0, 0.0, 1.0,
                                  FAKE, 8, NULL, NULL, NULL, NULL, NULL, NULL, NULL)
    assert rc == -10
    assert "262144" in cis.status_string(rc)
    hdr = open(HEADER).read()
    assert re.search(r"#define CIS_NOALLOC_MAX_T 262144\b", hdr)
