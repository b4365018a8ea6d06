"""GPU parity under padding that is not a suffix: holes inside a sequence, a
fully padded sequence, left padding and a single valid step (the layer's mask
is any [L, B] pattern).  Whole layers through the C ABI against the oracle,
for the gated recurrence, the gate variants, the projection trick and the
linear recurrence (whose chunked scan composes padded steps as identity
maps), fp32 and bf16 products, every direction, k = 3 and 4, the backward's
shorter ring at 65,536+ lanes, and the fused inference kernel."""

import numpy as np
import pytest
import torch

from helpers import TOL_BF16, TOL_FP32, check, dev, host
from oracle import sru_oracle as O
from paper_1709_02755_amd import sru
from paper_1709_02755_amd.workloads import irregular_mask, random_layer_case

pytestmark = pytest.mark.gpu

VARIANTS = dict(gated={}, alpha_reset_new=dict(alpha=1.6, reset_new=True),
                linear=dict(linear=True))

CASES = [
    # (L, B, d_in, d, direction, gemm, variant)
    (23, 10, 96, 96, O.DIR_BI, O.GEMM_FP32, "gated"),
    (23, 10, 130, 65, O.DIR_FWD, O.GEMM_BF16, "gated"),
    (40, 10, 256, 256, O.DIR_REV, O.GEMM_BF16, "alpha_reset_new"),
    (30, 10, 64, 64, O.DIR_BI, O.GEMM_FP32, "linear"),
    (600, 5, 64, 64, O.DIR_FWD, O.GEMM_FP32, "linear"),  # few lanes: time segments
    (20, 70, 1024, 1024, O.DIR_FWD, O.GEMM_BF16, "gated"),  # 71,680 lanes
]


def _case(seed, L, B, d_in, d, direction):
    rng = np.random.default_rng(seed)
    c = random_layer_case(rng, L, B, d_in, d, direction, c0=True, dc_last=True,
                          bias_scale=0.5, v_scale=1.2)
    c["mask"] = irregular_mask(rng, L, B)
    return c


@pytest.mark.parametrize("case", CASES)
def test_layer_with_irregular_mask(case):
    L, B, d_in, d, direction, gemm, variant = case
    print(f"irregular mask L={L} B={B} d_in={d_in} d={d} dir={direction} gemm={gemm} "
          f"{variant}", flush=True)
    c = _case(L + d + B, L, B, d_in, d, direction)
    v = VARIANTS[variant]
    linear = v.get("linear", False)
    gv = dict(highway_scale=v.get("alpha", 1.0), reset_new=v.get("reset_new", False),
              linear=linear)
    X, W = dev(c["X"]), dev(c["W"])
    p = [None, None] if linear else [dev(c["v_f"]), dev(c["v_r"])]
    p += [dev(c["b_f"]), dev(c["b_r"])]
    c0, mask = dev(c["c0"]), dev(c["mask"])
    fw = sru.forward(X, W, *p, c0=c0, direction=direction, mask=mask, gemm_dtype=gemm, **gv)
    bw = sru.backward(X, W, *p, fw["U"], fw["C"], dev(c["dH"]), c0=c0,
                      dc_last=dev(c["dc_last"]), direction=direction, mask=mask,
                      gemm_dtype=gemm, **gv)
    torch.cuda.synchronize()

    vr = (None, None) if linear else (c["v_f"], c["v_r"])
    args = (c["X"], c["W"], *vr, c["b_f"], c["b_r"])
    rf = O.forward(*args, c["c0"], direction, c["mask"], gemm, **v)
    rb = O.backward(*args, c["dH"], c["c0"], direction, c["mask"], gemm, c["dc_last"], fw=rf,
                    **v)
    tol = TOL_FP32 if gemm == O.GEMM_FP32 else TOL_BF16
    for k in ("H", "C", "c_last"):
        check(k, fw[k], rf[k], tol)
    grads = ("dX", "dW", "db_f", "db_r", "dc0") + (() if linear else ("dv_f", "dv_r"))
    for k in grads:
        check(k, bw[k], rb[k], tol)

    m = c["mask"].astype(bool)
    assert np.all(host(fw["H"])[m] == 0.0)
    assert np.all(host(bw["dX"])[m] == 0.0)
    # a fully padded sequence passes its state and its state gradient through
    # unchanged: c_last = c0 and dc0 = dc_last, bit for bit
    empty = np.flatnonzero(m.all(axis=0))
    assert empty.size > 0
    for b in empty:
        assert torch.equal(fw["c_last"][b], c0[b])
        assert torch.equal(bw["dc0"][b], dev(c["dc_last"])[b])


@pytest.mark.parametrize("linear", [False, True])
def test_fused_inference_with_irregular_mask(linear):
    """The fused projection + scan (U and C not stored; k = 4, at most 64
    steps) under the same masks, against the oracle."""
    L, B, d_in, d, direction = 64, 10, 256, 128, O.DIR_BI
    assert sru.fused_available(L, B, d_in, d, direction, O.GEMM_BF16)
    c = _case(17 + linear, L, B, d_in, d, direction)
    p = [None, None] if linear else [dev(c["v_f"]), dev(c["v_r"])]
    p += [dev(c["b_f"]), dev(c["b_r"])]
    ndir = 2
    out = dict(U=None, H=torch.empty((L, B, ndir * d), device="cuda"), C=None,
               c_last=torch.empty((B, ndir * d), device="cuda"),
               H_bf16=torch.empty((L, B, ndir * d), dtype=torch.bfloat16, device="cuda"))
    sru.forward(dev(c["X"]), dev(c["W"]), *p, c0=dev(c["c0"]), direction=direction,
                mask=dev(c["mask"]), gemm_dtype=O.GEMM_BF16, store_c=False, out=out,
                linear=linear)
    torch.cuda.synchronize()
    vr = (None, None) if linear else (c["v_f"], c["v_r"])
    rf = O.forward(c["X"], c["W"], *vr, c["b_f"], c["b_r"], c["c0"], direction, c["mask"],
                   O.GEMM_BF16, linear=linear)
    for k in ("H", "c_last"):
        check(k, out[k], rf[k], TOL_BF16)
    m = c["mask"].astype(bool)
    assert np.all(host(out["H"])[m] == 0.0)


@pytest.mark.parametrize("gemm", [O.GEMM_FP32, O.GEMM_BF16])
def test_lowrank_layer_with_irregular_mask(gemm):
    """The projection trick (Wcat = P Q^T, Sec. 4.4) under the same masks:
    T = X Q runs over padded steps too, but no gradient of a padded step
    reaches dX, dQ or dP."""
    L, B, d_in, d, dp, direction = 29, 10, 128, 64, 32, O.DIR_BI
    print(f"lowrank irregular mask gemm={gemm}", flush=True)
    c = _case(41 + gemm, L, B, d_in, d, direction)
    rng = np.random.default_rng(43 + gemm)
    ndir, k = c["W"].shape[:2]
    Q = (rng.uniform(-1, 1, (d_in, dp)) * np.sqrt(3.0 / d_in)).astype(np.float32)
    P = (rng.uniform(-1, 1, (ndir, k, d, dp)) * np.sqrt(3.0 / dp)).astype(np.float32)
    p = [dev(c[key]) for key in ("v_f", "v_r", "b_f", "b_r")]
    X, Qd, Pd, c0, mask = dev(c["X"]), dev(Q), dev(P), dev(c["c0"]), dev(c["mask"])
    fw = sru.forward_lowrank(X, Qd, Pd, *p, c0=c0, direction=direction, mask=mask,
                             gemm_dtype=gemm)
    bw = sru.backward_lowrank(X, Qd, Pd, *p, fw["T"], fw["U"], fw["C"], dev(c["dH"]), c0=c0,
                              dc_last=dev(c["dc_last"]), direction=direction, mask=mask,
                              gemm_dtype=gemm)
    torch.cuda.synchronize()
    args = (c["X"], Q, P, c["v_f"], c["v_r"], c["b_f"], c["b_r"])
    rf = O.forward_lowrank(*args, c["c0"], direction, c["mask"], gemm)
    rb = O.backward_lowrank(*args, c["dH"], c["c0"], direction, c["mask"], gemm, c["dc_last"],
                            fw=rf)
    tol = TOL_FP32 if gemm == O.GEMM_FP32 else TOL_BF16
    for key in ("H", "C", "c_last"):
        check(key, fw[key], rf[key], tol)
    for key in ("dX", "dQ", "dP", "dv_f", "dv_r", "db_f", "db_r", "dc0"):
        check(key, bw[key], rb[key], tol)
    m = c["mask"].astype(bool)
    assert np.all(host(fw["H"])[m] == 0.0)
    assert np.all(host(bw["dX"])[m] == 0.0)
