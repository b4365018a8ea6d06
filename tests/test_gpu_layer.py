"""GPU parity of one full layer (sru_forward + sru_backward through the C ABI)
against the oracle, over shapes that span several tiles and ragged tails,
both directions, k = 3 and 4, masks, c0 / dc_last, fp32 and bf16 GEMMs."""

import numpy as np
import pytest
import torch

from helpers import TOL_BF16, TOL_FP32, check, dev, host
from oracle import sru_oracle as O
from paper_1709_02755_amd import sru
from paper_1709_02755_amd.workloads import random_layer_case

pytestmark = pytest.mark.gpu

LAYER_CASES = [
    # (L, B, d_in, d, direction, masked, gemm)
    (1, 1, 1, 1, O.DIR_FWD, False, O.GEMM_FP32),
    (3, 2, 5, 5, O.DIR_REV, True, O.GEMM_FP32),
    (20, 3, 63, 63, O.DIR_BI, True, O.GEMM_FP32),
    (37, 5, 130, 65, O.DIR_FWD, False, O.GEMM_FP32),
    (64, 8, 128, 128, O.DIR_BI, True, O.GEMM_FP32),
    (50, 6, 256, 128, O.DIR_BI, True, O.GEMM_FP32),
    (31, 4, 300, 300, O.DIR_FWD, True, O.GEMM_FP32),
    (20, 3, 63, 63, O.DIR_BI, True, O.GEMM_BF16),
    (33, 9, 260, 260, O.DIR_FWD, False, O.GEMM_BF16),
    (48, 7, 512, 256, O.DIR_REV, True, O.GEMM_BF16),
    (64, 16, 512, 512, O.DIR_FWD, True, O.GEMM_BF16),
    # bidirectional, k = 3: dX adds both directions' highway gradients; whole
    # 256 x 256 tiles (epilogue through LDS) and a ragged row of tiles
    (40, 13, 256, 256, O.DIR_BI, True, O.GEMM_BF16),
    # one GPU's share of the headline batch (B = 8): 32 tiles of dX, split over K
    (256, 8, 1024, 1024, O.DIR_FWD, False, O.GEMM_BF16),
]


def run_layer(c, direction, gemm):
    X, W = dev(c["X"]), dev(c["W"])
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    c0, mask, dcl, dH = dev(c["c0"]), dev(c["mask"]), dev(c["dc_last"]), dev(c["dH"])
    fw = sru.forward(X, W, *p, c0=c0, direction=direction, mask=mask, gemm_dtype=gemm)
    bw = sru.backward(X, W, *p, fw["U"], fw["C"], dH, c0=c0, dc_last=dcl, direction=direction,
                      mask=mask, gemm_dtype=gemm)
    torch.cuda.synchronize()
    return fw, bw


@pytest.mark.parametrize("case", LAYER_CASES)
def test_layer_forward_backward(case):
    L, B, d_in, d, direction, masked, gemm = case
    print(f"layer L={L} B={B} d_in={d_in} d={d} dir={direction} mask={masked} gemm={gemm}",
          flush=True)
    c = random_layer_case(np.random.default_rng(L + 100 * d), L, B, d_in, d, direction,
                          masked=masked, c0=True, dc_last=True, bias_scale=0.5)
    fw, bw = run_layer(c, direction, gemm)
    args = (c["X"], c["W"], c["v_f"], c["v_r"], c["b_f"], c["b_r"])
    rf = O.forward(*args, c["c0"], direction, c["mask"], gemm)
    rb = O.backward(*args, c["dH"], c["c0"], direction, c["mask"], gemm, c["dc_last"])
    tol = TOL_FP32 if gemm == O.GEMM_FP32 else TOL_BF16
    check("U", fw["U"], rf["U"], TOL_FP32)  # bf16 products are exact: accumulation only
    for k in ("H", "C", "c_last"):
        check(k, fw[k], rf[k], tol)
    for k in ("dX", "dW", "dv_f", "dv_r", "db_f", "db_r", "dc0"):
        check(k, bw[k], rb[k], tol)
    if masked:
        m = c["mask"].astype(bool)
        assert np.all(host(fw["H"])[m] == 0.0)
        assert np.all(host(bw["dX"])[m] == 0.0)


def test_layer_deterministic_and_fully_written():
    """Two runs give bit-identical outputs, and outputs pre-filled with NaN
    are completely overwritten."""
    L, B, d = 29, 6, 96
    c = random_layer_case(np.random.default_rng(9), L, B, d, d, O.DIR_BI, masked=True, c0=True,
                          dc_last=True, bias_scale=0.5)
    outs = []
    for _ in range(2):
        X, W = dev(c["X"]), dev(c["W"])
        p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
        nan = lambda shape: torch.full(shape, float("nan"), device="cuda")
        fo = dict(U=nan((L, B, 2, 3, d)), H=nan((L, B, 2 * d)), C=nan((L, B, 2 * d)),
                  c_last=nan((B, 2 * d)))
        fw = sru.forward(X, W, *p, c0=dev(c["c0"]), direction=O.DIR_BI, mask=dev(c["mask"]),
                         gemm_dtype=O.GEMM_BF16, out=fo)
        bo = dict(dX=nan((L, B, d)), dW=nan((2, 3, d, d)), dv_f=nan((2, d)), dv_r=nan((2, d)),
                  db_f=nan((2, d)), db_r=nan((2, d)), dc0=nan((B, 2 * d)))
        ws = torch.full((sru.backward_workspace_bytes(L, B, d, d, O.DIR_BI, O.GEMM_BF16),),
                        255, dtype=torch.uint8, device="cuda")
        bw = sru.backward(X, W, *p, fw["U"], fw["C"], dev(c["dH"]), c0=dev(c["c0"]),
                          dc_last=dev(c["dc_last"]), direction=O.DIR_BI, mask=dev(c["mask"]),
                          gemm_dtype=O.GEMM_BF16, out=bo, ws=ws)
        torch.cuda.synchronize()
        outs.append({k: host(v) for k, v in {**fw, **bw}.items()})
    for k, v in outs[0].items():
        assert np.all(np.isfinite(v)), k
        assert np.array_equal(v, outs[1][k]), k


def test_forward_without_state_output():
    """C = NULL (inference) gives the same H and c_last."""
    L, B, d = 19, 4, 64
    c = random_layer_case(np.random.default_rng(4), L, B, d, d, O.DIR_FWD, masked=True, c0=True)
    X, W = dev(c["X"]), dev(c["W"])
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    a = sru.forward(X, W, *p, c0=dev(c["c0"]), mask=dev(c["mask"]))
    b = sru.forward(X, W, *p, c0=dev(c["c0"]), mask=dev(c["mask"]), store_c=False)
    torch.cuda.synchronize()
    assert b["C"] is None
    assert torch.equal(a["H"], b["H"]) and torch.equal(a["c_last"], b["c_last"])


def test_chunked_state_carry_on_gpu():
    """[0, L) in one call equals [0, L/2) then [L/2, L) with c_last -> c0."""
    L, B, d = 24, 5, 80
    c = random_layer_case(np.random.default_rng(8), L, B, d, d, O.DIR_FWD, c0=True, bias_scale=0.5)
    X, W = dev(c["X"]), dev(c["W"])
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    full = sru.forward(X, W, *p, c0=dev(c["c0"]))
    a = sru.forward(X[: L // 2].contiguous(), W, *p, c0=dev(c["c0"]))
    b = sru.forward(X[L // 2:].contiguous(), W, *p, c0=a["c_last"])
    torch.cuda.synchronize()
    assert torch.equal(torch.cat([a["H"], b["H"]]), full["H"])
    assert torch.equal(b["c_last"], full["c_last"])


@pytest.mark.parametrize("direction,gemm", [(O.DIR_FWD, O.GEMM_FP32), (O.DIR_FWD, O.GEMM_BF16),
                                            (O.DIR_REV, O.GEMM_BF16)])
def test_chunked_backward_carry_on_gpu(direction, gemm):
    """Truncation-free back-propagation in chunks: forward over the chunks
    with c_last -> c0, backward over them in reverse processing order with
    dc0 -> dc_last.  H, dX and dc0 equal the one-call layer bit for bit (the
    same operations per step and per output row); parameter gradients are
    the chunks' sum, equal to the one-call ones within the tolerance (a
    different summation order)."""
    L, B, d, h = 40, 6, 128, 24
    print(f"chunked backward dir={direction} gemm={gemm}", flush=True)
    c = random_layer_case(np.random.default_rng(21 + direction), L, B, d, d, direction,
                          c0=True, dc_last=True, bias_scale=0.5)
    X, W = dev(c["X"]), dev(c["W"])
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    c0, dcl, dH = dev(c["c0"]), dev(c["dc_last"]), dev(c["dH"])
    kw = dict(direction=direction, gemm_dtype=gemm)
    full = sru.forward(X, W, *p, c0=c0, **kw)
    fb = sru.backward(X, W, *p, full["U"], full["C"], dH, c0=c0, dc_last=dcl, **kw)
    first, second = (slice(0, h), slice(h, L)) if direction == O.DIR_FWD else (slice(h, L),
                                                                               slice(0, h))
    part = lambda t, s: t[s].contiguous()
    fa = sru.forward(part(X, first), W, *p, c0=c0, **kw)
    fs = sru.forward(part(X, second), W, *p, c0=fa["c_last"], **kw)
    gs = sru.backward(part(X, second), W, *p, fs["U"], fs["C"], part(dH, second), c0=fa["c_last"],
                      dc_last=dcl, **kw)
    ga = sru.backward(part(X, first), W, *p, fa["U"], fa["C"], part(dH, first), c0=c0,
                      dc_last=gs["dc0"], **kw)
    torch.cuda.synchronize()
    H = torch.empty_like(full["H"])
    H[first], H[second] = fa["H"], fs["H"]
    dX = torch.empty_like(fb["dX"])
    dX[first], dX[second] = ga["dX"], gs["dX"]
    assert torch.equal(H, full["H"])
    assert torch.equal(dX, fb["dX"])
    assert torch.equal(ga["dc0"], fb["dc0"])
    tol = TOL_FP32 if gemm == O.GEMM_FP32 else 1e-5
    for k in ("dW", "dv_f", "dv_r", "db_f", "db_r"):
        check(k, ga[k] + gs[k], host(fb[k]), tol)


@pytest.mark.parametrize("direction", [O.DIR_FWD, O.DIR_REV])
def test_chunked_backward_carry_time_parallel(direction):
    """The same chunked back-propagation at 8,192 lanes, where the backward
    scan runs time-parallel: a chunk's incoming gradient is composed from
    maps, so the calls agree with the one-call layer to fp32 rounding rather
    than bit for bit.  H is still bit for bit (the forward is sequential)."""
    L, B, d, h = 50, 8, 1024, 21
    print(f"chunked backward, time-parallel scan, dir={direction}", flush=True)
    c = random_layer_case(np.random.default_rng(31 + direction), L, B, d, d, direction,
                          masked=True, c0=True, dc_last=True, bias_scale=0.5)
    X, W, mask = dev(c["X"]), dev(c["W"]), dev(c["mask"])
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    c0, dcl, dH = dev(c["c0"]), dev(c["dc_last"]), dev(c["dH"])
    kw = dict(direction=direction, gemm_dtype=O.GEMM_FP32)
    full = sru.forward(X, W, *p, c0=c0, mask=mask, **kw)
    fb = sru.backward(X, W, *p, full["U"], full["C"], dH, c0=c0, dc_last=dcl, mask=mask, **kw)
    first, second = (slice(0, h), slice(h, L)) if direction == O.DIR_FWD else (slice(h, L),
                                                                               slice(0, h))
    part = lambda t, s: t[s].contiguous()
    fa = sru.forward(part(X, first), W, *p, c0=c0, mask=part(mask, first), **kw)
    fs = sru.forward(part(X, second), W, *p, c0=fa["c_last"], mask=part(mask, second), **kw)
    gs = sru.backward(part(X, second), W, *p, fs["U"], fs["C"], part(dH, second), c0=fa["c_last"],
                      dc_last=dcl, mask=part(mask, second), **kw)
    ga = sru.backward(part(X, first), W, *p, fa["U"], fa["C"], part(dH, first), c0=c0,
                      dc_last=gs["dc0"], mask=part(mask, first), **kw)
    torch.cuda.synchronize()
    H = torch.empty_like(full["H"])
    H[first], H[second] = fa["H"], fs["H"]
    dX = torch.empty_like(fb["dX"])
    dX[first], dX[second] = ga["dX"], gs["dX"]
    assert torch.equal(H, full["H"])
    check("dX", dX, host(fb["dX"]), TOL_FP32)
    check("dc0", ga["dc0"], host(fb["dc0"]), TOL_FP32)
    for k in ("dW", "dv_f", "dv_r", "db_f", "db_r"):
        check(k, ga[k] + gs[k], host(fb[k]), TOL_FP32)


def test_layers_on_two_streams_equal_serial():
    """Two layers enqueued at once on two streams (default priority) give the
    same bits as the same calls one after the other: the library keeps no
    state between calls, and each call's work stays on its own stream."""
    print("two streams: bf16 forward L=33 B=8 d=256 | fp32 bidirectional L=20 B=5 d=96", flush=True)
    cases = [(random_layer_case(np.random.default_rng(11), 33, 8, 256, 256, O.DIR_FWD, masked=True,
                                c0=True, dc_last=True, bias_scale=0.5), O.DIR_FWD, O.GEMM_BF16),
             (random_layer_case(np.random.default_rng(12), 20, 5, 96, 96, O.DIR_BI, masked=True,
                                c0=True, dc_last=True, bias_scale=0.5), O.DIR_BI, O.GEMM_FP32)]

    def enqueue(c, direction, gemm):
        X, W = dev(c["X"]), dev(c["W"])
        p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
        c0, mask, dcl, dH = dev(c["c0"]), dev(c["mask"]), dev(c["dc_last"]), dev(c["dH"])
        fw = sru.forward(X, W, *p, c0=c0, direction=direction, mask=mask, gemm_dtype=gemm)
        bw = sru.backward(X, W, *p, fw["U"], fw["C"], dH, c0=c0, dc_last=dcl,
                          direction=direction, mask=mask, gemm_dtype=gemm)
        return {**fw, **bw}

    serial = [enqueue(*a) for a in cases]
    torch.cuda.synchronize()
    serial = [{k: host(v) for k, v in r.items() if v is not None} for r in serial]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = []
    for st, a in zip(streams, cases):
        with torch.cuda.stream(st):
            outs.append(enqueue(*a))
    torch.cuda.synchronize()
    for ref, got in zip(serial, outs):
        for k, v in ref.items():
            assert np.array_equal(host(got[k]), v), k


@pytest.mark.parametrize("case", [
    (256, 8, 1024, 1024, O.DIR_FWD, False, O.GEMM_BF16, False),  # dW split: in its split-K sum
    (64, 16, 512, 512, O.DIR_FWD, True, O.GEMM_BF16, False),
    (50, 6, 256, 128, O.DIR_BI, True, O.GEMM_FP32, False),
    (3, 2, 5, 5, O.DIR_REV, True, O.GEMM_FP32, False),           # dW not split: own launch
    # the linear recurrence: b sums only, over (time segment, sequence) rows
    (2000, 4, 64, 64, O.DIR_FWD, True, O.GEMM_BF16, True),
    (400, 2, 64, 64, O.DIR_BI, True, O.GEMM_FP32, True),
])
def test_vb_sums_same_bits_as_standalone_scan(case):
    """The layer backward sums the v/b gradients over the batch inside the
    dW product's launches; the standalone backward scan sums them in its own
    launch.  Both run the same fixed-order sum: identical bits."""
    L, B, d_in, d, direction, masked, gemm, linear = case
    print(f"vb sums L={L} B={B} d_in={d_in} d={d} dir={direction} gemm={gemm} "
          f"linear={linear}", flush=True)
    c = random_layer_case(np.random.default_rng(5 * L + d), L, B, d_in, d, direction,
                          masked=masked, c0=True, dc_last=True, bias_scale=0.5)
    X, W = dev(c["X"]), dev(c["W"])
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    kw = dict(c0=dev(c["c0"]), direction=direction, mask=dev(c["mask"]), linear=linear)
    fw = sru.forward(X, W, *p, gemm_dtype=gemm, **kw)
    bw = sru.backward(X, W, *p, fw["U"], fw["C"], dev(c["dH"]), dc_last=dev(c["dc_last"]),
                      gemm_dtype=gemm, **kw)
    sb = sru.scan_backward(fw["U"], X, fw["C"], dev(c["dH"]), *p, dc_last=dev(c["dc_last"]),
                           **kw)
    torch.cuda.synchronize()
    for k in ("dv_f", "dv_r", "db_f", "db_r", "dc0"):
        if linear and k in ("dv_f", "dv_r"):
            assert bw[k] is None and sb[k] is None
            continue
        assert torch.equal(bw[k], sb[k]), k
