"""GPU parity of the gate variants against the oracle: the highway scaling
correction alpha of Sec. 3.2 and the reset gate reading c_t (the order of
Algorithm 1), through the scans alone and through whole layers (fp32 and
bf16 products, both directions, k = 3 and 4, masks)."""

import numpy as np
import pytest
import torch

from helpers import TOL_BF16, TOL_FP32, check, dev, host
from oracle import sru_oracle as O
from paper_1709_02755_amd import sru
from paper_1709_02755_amd.workloads import random_layer_case

pytestmark = pytest.mark.gpu

VARIANTS = [(np.sqrt(3.0), False), (1.0, True), (O.scaling_alpha(-3.0), True)]

SCAN_CASES = [
    # (L, B, d_in, d, direction, masked)
    (1, 2, 4, 4, O.DIR_FWD, False),
    (13, 3, 65, 65, O.DIR_REV, True),
    (33, 4, 96, 64, O.DIR_BI, False),
    (40, 5, 128, 128, O.DIR_BI, True),
    (11, 64, 1024, 1024, O.DIR_REV, True),  # a wave on every SIMD: shorter backward ring
    (10, 32, 512, 1024, O.DIR_BI, True),  # k = 4, both directions, 256-unit workgroups
    (45, 8, 1024, 1024, O.DIR_FWD, True),  # 8,192 lanes: the time-parallel backward
]


def _case(seed, L, B, d_in, d, direction, **kw):
    return random_layer_case(np.random.default_rng(seed), L, B, d_in, d, direction, **kw)


@pytest.mark.parametrize("alpha,reset_new", VARIANTS)
@pytest.mark.parametrize("case", SCAN_CASES)
def test_scans_with_variants(case, alpha, reset_new):
    L, B, d_in, d, direction, masked = case
    print(f"variant scans L={L} B={B} d_in={d_in} d={d} dir={direction} mask={masked} "
          f"alpha={alpha:.3f} reset_new={reset_new}", flush=True)
    c = _case(L * 7 + d + int(10 * alpha), L, B, d_in, d, direction, masked=masked, c0=True,
              dc_last=True, bias_scale=0.5, v_scale=1.0)
    v = dict(alpha=alpha, reset_new=reset_new)
    args = (c["X"], c["W"], c["v_f"], c["v_r"], c["b_f"], c["b_r"])
    fw = O.forward(*args, c["c0"], direction, c["mask"], **v)
    bw = O.backward(*args, c["dH"], c["c0"], direction, c["mask"], O.GEMM_FP32, c["dc_last"],
                    fw=fw, **v)
    gv = dict(highway_scale=alpha, reset_new=reset_new)
    U = dev(fw["U"].astype(np.float32))
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    out = sru.scan_forward(U, dev(c["X"]), *p, dev(c["c0"]), direction, dev(c["mask"]), **gv)
    bo = sru.scan_backward(U, dev(c["X"]), dev(fw["C"].astype(np.float32)), dev(c["dH"]), *p,
                           dev(c["c0"]), dev(c["dc_last"]), direction, dev(c["mask"]),
                           d_in=d_in, **gv)
    torch.cuda.synchronize()
    for k in ("H", "C", "c_last"):
        check(k, out[k], fw[k], TOL_FP32)
    check("dU", bo["dU"], bw["dU"], TOL_FP32)
    if d_in == d:
        check("dxh", bo["dxh"], bw["dxh"], TOL_FP32)
    for k in ("dv_f", "dv_r", "db_f", "db_r", "dc0"):
        check(k, bo[k], bw[k], TOL_FP32)


LAYER_CASES = [
    # (L, B, d_in, d, direction, masked, gemm)
    (20, 3, 63, 63, O.DIR_BI, True, O.GEMM_FP32),
    (31, 4, 96, 64, O.DIR_FWD, False, O.GEMM_FP32),
    (33, 9, 256, 256, O.DIR_REV, True, O.GEMM_BF16),
    (24, 6, 256, 128, O.DIR_BI, False, O.GEMM_BF16),
]


@pytest.mark.parametrize("alpha,reset_new", VARIANTS)
@pytest.mark.parametrize("case", LAYER_CASES)
def test_layer_with_variants(case, alpha, reset_new):
    L, B, d_in, d, direction, masked, gemm = case
    print(f"variant layer L={L} B={B} d_in={d_in} d={d} dir={direction} mask={masked} "
          f"gemm={gemm} alpha={alpha:.3f} reset_new={reset_new}", flush=True)
    c = _case(L + 100 * d + int(10 * alpha), L, B, d_in, d, direction, masked=masked, c0=True,
              dc_last=True, bias_scale=0.5)
    gv = dict(highway_scale=alpha, reset_new=reset_new)
    X, W = dev(c["X"]), dev(c["W"])
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    c0, mask = dev(c["c0"]), dev(c["mask"])
    fw = sru.forward(X, W, *p, c0=c0, direction=direction, mask=mask, gemm_dtype=gemm, **gv)
    bw = sru.backward(X, W, *p, fw["U"], fw["C"], dev(c["dH"]), c0=c0, dc_last=dev(c["dc_last"]),
                      direction=direction, mask=mask, gemm_dtype=gemm, **gv)
    torch.cuda.synchronize()
    v = dict(alpha=alpha, reset_new=reset_new)
    args = (c["X"], c["W"], c["v_f"], c["v_r"], c["b_f"], c["b_r"])
    rf = O.forward(*args, c["c0"], direction, c["mask"], gemm, **v)
    rb = O.backward(*args, c["dH"], c["c0"], direction, c["mask"], gemm, c["dc_last"], fw=rf, **v)
    tol = TOL_FP32 if gemm == O.GEMM_FP32 else TOL_BF16
    for k in ("H", "C", "c_last"):
        check(k, fw[k], rf[k], tol)
    for k in ("dX", "dW", "dv_f", "dv_r", "db_f", "db_r", "dc0"):
        check(k, bw[k], rb[k], tol)


def test_default_options_equal_no_options():
    """highway_scale = 1 with the Eq. 3 order passed as an explicit struct
    gives bit-identical results to NULL options."""
    import ctypes
    L, B, d = 17, 3, 64
    c = _case(5, L, B, d, d, O.DIR_BI, masked=True, c0=True, bias_scale=0.5)
    U = O.forward(c["X"], c["W"], c["v_f"], c["v_r"], c["b_f"], c["b_r"], c["c0"], O.DIR_BI,
                  c["mask"])["U"].astype(np.float32)
    Ud, Xd = dev(U), dev(c["X"])
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    outs = []
    for opts in (None, ctypes.byref(sru.Options(1.0, sru.RESET_PREV))):
        H = torch.empty((L, B, 2 * d), device="cuda")
        st = sru.lib().sru_scan_forward(sru._ptr(Ud), sru._ptr(Xd), *[sru._ptr(t) for t in p],
                                        sru._ptr(dev(c["c0"])), L, B, d, d, O.DIR_BI,
                                        sru._ptr(dev(c["mask"])), opts, sru._ptr(H), None, None,
                                        None, None, 0, sru._stream())
        assert st == 0
        outs.append(H)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])


@pytest.mark.parametrize("gemm", [O.GEMM_FP32, O.GEMM_BF16])
def test_layer_with_the_papers_reset_bias(gemm):
    """The setting of the character-level language model experiments (Sec.
    4): the reset gate's bias at -3, so the gate starts mostly closed and the
    highway carries most of x, with the correction Sec. 3.2 gives for a
    non-zero bias, alpha = sqrt(1 + 2 e^-3); a whole layer, forward and
    backward, against the oracle."""
    L, B, d, direction = 29, 5, 128, O.DIR_BI
    c = _case(77 + gemm, L, B, d, d, direction, masked=True, c0=True, dc_last=True,
              bias_scale=0.5)
    c["b_r"] = np.full_like(c["b_r"], -3.0)
    alpha = O.scaling_alpha(-3.0)
    X, W = dev(c["X"]), dev(c["W"])
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    c0, mask = dev(c["c0"]), dev(c["mask"])
    fw = sru.forward(X, W, *p, c0=c0, direction=direction, mask=mask, gemm_dtype=gemm,
                     highway_scale=alpha)
    bw = sru.backward(X, W, *p, fw["U"], fw["C"], dev(c["dH"]), c0=c0, dc_last=dev(c["dc_last"]),
                      direction=direction, mask=mask, gemm_dtype=gemm, highway_scale=alpha)
    torch.cuda.synchronize()
    args = (c["X"], c["W"], c["v_f"], c["v_r"], c["b_f"], c["b_r"])
    rf = O.forward(*args, c["c0"], direction, c["mask"], gemm, alpha=alpha)
    rb = O.backward(*args, c["dH"], c["c0"], direction, c["mask"], gemm, c["dc_last"], fw=rf,
                    alpha=alpha)
    tol = TOL_FP32 if gemm == O.GEMM_FP32 else TOL_BF16
    for k in ("H", "C", "c_last"):
        check(k, fw[k], rf[k], tol)
    for k in ("dX", "dW", "dv_f", "dv_r", "db_f", "db_r", "dc0"):
        check(k, bw[k], rb[k], tol)
