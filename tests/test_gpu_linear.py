"""GPU parity of the linear recurrence (ablation (1) of Sec. 4.5: v * c_{t-1}
removed from both gates) against the oracle.  The GPU scans this variant in
parallel over chunks of time, and with few lanes also over segments of time
run by separate workgroups; the cases below span one chunk per lane up to
16 chunks per workgroup, several time blocks with a ragged last block, one
to 32 segments with a short last one, lanes past the end of the last
workgroup, masks, both directions, k = 3 and 4, and the layer calls in fp32
and bf16."""

import numpy as np
import pytest
import torch

from helpers import TOL_BF16, TOL_FP32, check, dev
from oracle import sru_oracle as O
from paper_1709_02755_amd import sru
from paper_1709_02755_amd.workloads import random_layer_case

pytestmark = pytest.mark.gpu

SCAN_CASES = [
    # (L, B, d_in, d, direction, masked)
    (1, 1, 4, 4, O.DIR_FWD, False),      # one step, lanes past the end
    (5, 2, 3, 3, O.DIR_REV, True),       # shorter than one chunk
    (100, 2, 64, 64, O.DIR_BI, False),   # one block, empty trailing chunks
    (400, 32, 128, 128, O.DIR_BI, True),  # workload-2 shape: 16 chunks, ragged blocks
    (1000, 1, 130, 65, O.DIR_REV, True),  # many blocks, a partial workgroup, k = 4
    (37, 64, 1024, 1024, O.DIR_FWD, True),  # many lanes: few chunks per workgroup
    (4000, 2, 64, 64, O.DIR_FWD, True),   # two lane groups: 21 / 32 segments
    (777, 3, 96, 96, O.DIR_BI, False),    # 9 lane groups: 5 / 7 segments, short last one
]


def _case(seed, L, B, d_in, d, direction, **kw):
    return random_layer_case(np.random.default_rng(seed), L, B, d_in, d, direction, **kw)


@pytest.mark.parametrize("case", SCAN_CASES)
def test_linear_scans(case):
    L, B, d_in, d, direction, masked = case
    print(f"linear scans L={L} B={B} d_in={d_in} d={d} dir={direction} mask={masked}",
          flush=True)
    c = _case(L * 3 + d, L, B, d_in, d, direction, masked=masked, c0=True, dc_last=True,
              bias_scale=1.0)
    alpha = 1.25
    args = (c["X"], c["W"], None, None, c["b_f"], c["b_r"])
    fw = O.forward(*args, c["c0"], direction, c["mask"], alpha=alpha, linear=True)
    bw = O.backward(*args, c["dH"], c["c0"], direction, c["mask"], O.GEMM_FP32, c["dc_last"],
                    fw=fw, alpha=alpha, linear=True)
    U = dev(fw["U"].astype(np.float32))
    p = (None, None, dev(c["b_f"]), dev(c["b_r"]))
    gv = dict(highway_scale=alpha, linear=True)
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
    for k in ("db_f", "db_r", "dc0"):
        check(k, bo[k], bw[k], TOL_FP32)
    assert bo["dv_f"] is None and bo["dv_r"] is None


def test_linear_scan_padded_state_and_last_state():
    """C holds the carried state at padded steps and c_last is the state
    after each sequence's last valid step.  c_last is bit-equal to C at the
    last position (the same wave's state); across a chunk boundary the
    incoming state is the composition of the earlier chunks' maps, which
    rounds differently from the previous chunk's rescan, so C at later padded
    steps equals the last valid state to fp32 rounding, not bit for bit."""
    L, B, d = 300, 3, 64
    c = _case(3, L, B, d, d, O.DIR_FWD, masked=True, c0=True, bias_scale=1.0)
    fw = O.forward(c["X"], c["W"], None, None, c["b_f"], c["b_r"], c["c0"], O.DIR_FWD,
                   c["mask"], linear=True)
    U = dev(fw["U"].astype(np.float32))
    out = sru.scan_forward(U, dev(c["X"]), None, None, dev(c["b_f"]), dev(c["b_r"]),
                           dev(c["c0"]), O.DIR_FWD, dev(c["mask"]), linear=True)
    torch.cuda.synchronize()
    C = out["C"].cpu().numpy()
    cl = out["c_last"].cpu().numpy()
    assert np.array_equal(C[-1], cl)          # padded tail carries the state unchanged
    lengths = c["lengths"]
    for b in range(B):
        n = lengths[b]
        assert n < L or b == 0
        np.testing.assert_allclose(C[n - 1:, b], np.broadcast_to(C[n - 1, b], C[n - 1:, b].shape),
                                   rtol=1e-6, atol=1e-7)


def test_linear_scans_deterministic():
    L, B, d = 400, 32, 128
    c = _case(11, L, B, d, d, O.DIR_BI, masked=True, c0=True, dc_last=True, bias_scale=1.0)
    fw = O.forward(c["X"], c["W"], None, None, c["b_f"], c["b_r"], c["c0"], O.DIR_BI, c["mask"],
                   linear=True)
    U, X = dev(fw["U"].astype(np.float32)), dev(c["X"])
    Cd = dev(fw["C"].astype(np.float32))
    p = (None, None, dev(c["b_f"]), dev(c["b_r"]))
    runs = []
    for _ in range(2):
        o = sru.scan_forward(U, X, *p, dev(c["c0"]), O.DIR_BI, dev(c["mask"]), linear=True)
        b = sru.scan_backward(U, X, Cd, dev(c["dH"]), *p, dev(c["c0"]), dev(c["dc_last"]),
                              O.DIR_BI, dev(c["mask"]), linear=True)
        runs.append((o, b))
    torch.cuda.synchronize()
    for k in ("H", "C", "c_last"):
        assert torch.equal(runs[0][0][k], runs[1][0][k]), k
    for k in ("dU", "dxh", "db_f", "db_r", "dc0"):
        assert torch.equal(runs[0][1][k], runs[1][1][k]), k


LAYER_CASES = [
    # (L, B, d_in, d, direction, masked, gemm)
    (64, 4, 63, 63, O.DIR_BI, True, O.GEMM_FP32),
    (200, 2, 96, 64, O.DIR_FWD, False, O.GEMM_FP32),
    (130, 8, 256, 256, O.DIR_REV, True, O.GEMM_BF16),
    (96, 4, 256, 128, O.DIR_BI, False, O.GEMM_BF16),
]


@pytest.mark.parametrize("case", LAYER_CASES)
def test_linear_layer(case):
    L, B, d_in, d, direction, masked, gemm = case
    print(f"linear layer L={L} B={B} d_in={d_in} d={d} dir={direction} mask={masked} "
          f"gemm={gemm}", flush=True)
    c = _case(L + 7 * d, L, B, d_in, d, direction, masked=masked, c0=True, dc_last=True,
              bias_scale=0.5)
    X, W = dev(c["X"]), dev(c["W"])
    p = (None, None, dev(c["b_f"]), dev(c["b_r"]))
    c0, mask = dev(c["c0"]), dev(c["mask"])
    fw = sru.forward(X, W, *p, c0=c0, direction=direction, mask=mask, gemm_dtype=gemm,
                     linear=True)
    bw = sru.backward(X, W, *p, fw["U"], fw["C"], dev(c["dH"]), c0=c0, dc_last=dev(c["dc_last"]),
                      direction=direction, mask=mask, gemm_dtype=gemm, linear=True)
    torch.cuda.synchronize()
    args = (c["X"], c["W"], None, None, c["b_f"], c["b_r"])
    rf = O.forward(*args, c["c0"], direction, c["mask"], gemm, linear=True)
    rb = O.backward(*args, c["dH"], c["c0"], direction, c["mask"], gemm, c["dc_last"], fw=rf,
                    linear=True)
    tol = TOL_FP32 if gemm == O.GEMM_FP32 else TOL_BF16
    for k in ("H", "C", "c_last"):
        check(k, fw[k], rf[k], tol)
    for k in ("dX", "dW", "db_f", "db_r", "dc0"):
        check(k, bw[k], rb[k], tol)


def test_linear_layer_ignores_v():
    """Passing v (any values) or NULL gives bit-identical results."""
    L, B, d = 150, 4, 64
    c = _case(21, L, B, d, d, O.DIR_BI, masked=True, c0=True, bias_scale=0.5, v_scale=3.0)
    X, W = dev(c["X"]), dev(c["W"])
    outs = []
    for vf, vr in ((None, None), (dev(c["v_f"]), dev(c["v_r"]))):
        fw = sru.forward(X, W, vf, vr, dev(c["b_f"]), dev(c["b_r"]), c0=dev(c["c0"]),
                         direction=O.DIR_BI, mask=dev(c["mask"]), linear=True)
        bw = sru.backward(X, W, vf, vr, dev(c["b_f"]), dev(c["b_r"]), fw["U"], fw["C"],
                          dev(c["dH"]), c0=dev(c["c0"]), direction=O.DIR_BI, mask=dev(c["mask"]),
                          linear=True)
        outs.append((fw, bw))
    torch.cuda.synchronize()
    for k in ("H", "C", "c_last"):
        assert torch.equal(outs[0][0][k], outs[1][0][k]), k
    for k in ("dX", "dW", "db_f", "db_r", "dc0"):
        assert torch.equal(outs[0][1][k], outs[1][1][k]), k


def test_linear_lowrank_layer():
    """The projection trick with the linear recurrence (bf16 products)."""
    L, B, d_in, d, dp, direction = 120, 6, 128, 128, 64, O.DIR_BI
    rng = np.random.default_rng(5)
    c = random_layer_case(rng, L, B, d_in, d, direction, masked=True, c0=True, dc_last=True,
                          bias_scale=0.5)
    ndir = 2
    Q = (rng.standard_normal((d_in, dp)) / np.sqrt(d_in)).astype(np.float32)
    P = (rng.standard_normal((ndir, 3, d, dp)) / np.sqrt(dp)).astype(np.float32)
    gemm = O.GEMM_BF16
    p = (None, None, dev(c["b_f"]), dev(c["b_r"]))
    fw = sru.forward_lowrank(dev(c["X"]), dev(Q), dev(P), *p, c0=dev(c["c0"]), direction=direction,
                             mask=dev(c["mask"]), gemm_dtype=gemm, linear=True)
    bw = sru.backward_lowrank(dev(c["X"]), dev(Q), dev(P), *p, fw["T"], fw["U"], fw["C"],
                              dev(c["dH"]), c0=dev(c["c0"]), dc_last=dev(c["dc_last"]),
                              direction=direction, mask=dev(c["mask"]), gemm_dtype=gemm,
                              linear=True)
    torch.cuda.synchronize()
    args = (c["X"], Q, P, None, None, c["b_f"], c["b_r"])
    rf = O.forward_lowrank(*args, c["c0"], direction, c["mask"], gemm, linear=True)
    rb = O.backward_lowrank(*args, c["dH"], c["c0"], direction, c["mask"], gemm, c["dc_last"],
                            fw=rf, linear=True)
    for k in ("H", "C", "c_last"):
        check(k, fw[k], rf[k], TOL_BF16)
    for k in ("dX", "dQ", "dP", "db_f", "db_r", "dc0"):
        check(k, bw[k], rb[k], TOL_BF16)
