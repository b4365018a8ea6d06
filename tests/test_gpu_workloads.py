"""GPU parity on the five target workloads (stacked layers, forward and
backward) against the oracle.

* Workloads 0-2 run at their full sizes; the oracle finishes them in seconds.
* Workloads 3-4 run in full at reduced sizes with the same structure
  (layers, direction, mask recipe, bf16 GEMMs), and at their full sizes in the
  launch configuration the benchmark times: one full-size layer against the
  full oracle, and the full stack against the oracle on a slice of the batch
  (sequences never interact, so the oracle on a batch slice is exact for
  those sequences' H and dX).
* One GPU's shard of workload 3 (B = 8) runs in full at its full size, and
  so does the inference workload (on a batch slice), as the benchmark runs
  them.
"""

import numpy as np
import pytest
import torch

from helpers import TOL_BF16, TOL_BF16_LOWRANK_STACK, TOL_FP32, check, dev, host, layer_to_dev
from oracle import sru_oracle as O
from paper_1709_02755_amd import sru
from paper_1709_02755_amd.workloads import WORKLOADS, make_inputs, scaled

pytestmark = pytest.mark.gpu


def _tol(w):
    if w.gemm_dtype == O.GEMM_FP32:
        return TOL_FP32
    return TOL_BF16 if w.dp is None else TOL_BF16_LOWRANK_STACK


def run_stack(w, inp):
    layers = [layer_to_dev(p) for p in inp["layers"]]
    st = sru.Stack(layers, w.L, w.B, w.d_in, w.d, w.direction, w.gemm_dtype, "cuda",
                   backward=w.backward, linear=w.linear)
    X, mask = dev(inp["X"]), dev(inp["mask"])
    st.forward(X, mask)
    if w.backward:
        st.backward(X, dev(inp["dH"]), mask)
    torch.cuda.synchronize()
    return st


def compare_stack(w, inp, st, bsel=None):
    """Oracle on the whole batch (bsel None) or on the sequences in bsel."""
    sl = slice(None) if bsel is None else bsel
    X = inp["X"][:, sl]
    mask = None if inp["mask"] is None else inp["mask"][:, sl]
    dH = None if inp["dH"] is None else inp["dH"][:, sl]
    ref = O.stack_forward_backward(X, inp["layers"], w.direction, mask, w.gemm_dtype, dH,
                                   need_backward=w.backward, linear=w.linear)
    tol = _tol(w)
    for li in range(w.layers):
        check(f"H[{li}]", host(st.fw[li]["H"])[:, sl], ref["Hs"][li], tol)
        check(f"C[{li}]", host(st.fw[li]["C"])[:, sl], ref["Cs"][li], tol)
    if w.backward:
        for li in range(w.layers):
            check(f"dX[{li}]", host(st.bw[li]["dX"])[:, sl], ref["grads"][li]["dX"], tol)
            if bsel is None:
                for k in ("dW", "dQ", "dP", "dv_f", "dv_r", "db_f", "db_r"):
                    if ref["grads"][li].get(k) is not None:
                        check(f"{k}[{li}]", st.bw[li][k], ref["grads"][li][k], tol)


@pytest.mark.parametrize("wi", [0, 1, 2, 7])
def test_workload_full_size(wi):
    w = WORKLOADS[wi]
    print(f"workload {w.name}", flush=True)
    inp = make_inputs(w)
    st = run_stack(w, inp)
    compare_stack(w, inp, st)


@pytest.mark.parametrize("wi", [3, 4, 6])
def test_workload_reduced_size(wi):
    w = scaled(WORKLOADS[wi], L=48, B=12, d=256)
    print(f"workload {w.name}", flush=True)
    inp = make_inputs(w)
    st = run_stack(w, inp)
    compare_stack(w, inp, st)


@pytest.mark.slow
def test_shard_workload_full_size():
    """One GPU's share of the headline stack (B = 8 of its 64 sequences) at
    its full size, the whole batch against the oracle: every layer's H, C,
    dX, dW and v/b sums."""
    w = WORKLOADS[8]
    print(f"workload {w.name}", flush=True)
    inp = make_inputs(w)
    st = run_stack(w, inp)
    compare_stack(w, inp, st)


@pytest.mark.slow
@pytest.mark.parametrize("wi", [3, 4])
def test_workload_full_size_single_layer(wi):
    """Layer 1 of the workload at full size against the full oracle: every
    output and gradient, including dW and the v/b sums over all tokens."""
    w = WORKLOADS[wi]
    print(f"workload {w.name} single full layer", flush=True)
    inp = make_inputs(w)
    p = inp["layers"][0]
    X, mask = inp["X"], inp["mask"]
    rng = np.random.default_rng(100 + wi)
    dH = rng.standard_normal((w.L, w.B, w.ndir * w.d)).astype(np.float32)
    pd = layer_to_dev(p)
    args = (pd["v_f"], pd["v_r"], pd["b_f"], pd["b_r"])
    fw = sru.forward(dev(X), pd["W"], *args, direction=w.direction, mask=dev(mask),
                     gemm_dtype=w.gemm_dtype)
    bw = sru.backward(dev(X), pd["W"], *args, fw["U"], fw["C"], dev(dH), direction=w.direction,
                      mask=dev(mask), gemm_dtype=w.gemm_dtype)
    torch.cuda.synchronize()
    oargs = (X, p["W"], p["v_f"], p["v_r"], p["b_f"], p["b_r"])
    rf = O.forward(*oargs, None, w.direction, mask, w.gemm_dtype)
    rb = O.backward(*oargs, dH, None, w.direction, mask, w.gemm_dtype, fw=rf)
    tol = _tol(w)
    check("U", fw["U"], rf["U"], TOL_FP32)
    for k in ("H", "C", "c_last"):
        check(k, fw[k], rf[k], tol)
    for k in ("dX", "dW", "dv_f", "dv_r", "db_f", "db_r", "dc0"):
        check(k, bw[k], rb[k], tol)


@pytest.mark.slow
@pytest.mark.parametrize("wi", [3, 4])
def test_workload_full_size_stack_on_batch_slice(wi):
    """The full stack at full size; the oracle checks every layer's H and C
    and every layer's dX on two sequences (the full-length first one and the
    last one)."""
    w = WORKLOADS[wi]
    print(f"workload {w.name} full stack, batch slice", flush=True)
    inp = make_inputs(w)
    st = run_stack(w, inp)
    compare_stack(w, inp, st, bsel=[0, w.B - 1])


def test_inference_workload_full_size():
    """The Transformer-FFN inference shape (d_in 512 -> d 2048, k = 4,
    forward only, no C) at its full size in the benchmark's launch
    configuration (weights held in bf16); the oracle on a slice of the batch
    (sequences never interact)."""
    w = WORKLOADS[5]
    print(f"workload {w.name}", flush=True)
    assert not w.backward and not w.store_c and w.d_in != w.d
    inp = make_inputs(w)
    layers = [layer_to_dev(p) for p in inp["layers"]]
    for p in layers:  # the benchmark holds inference weights in bf16
        p["W"] = sru.round_bf16(p["W"])
    st = sru.Stack(layers, w.L, w.B, w.d_in, w.d, w.direction, w.gemm_dtype, "cuda",
                   backward=False, store_c=False)
    H = st.forward(dev(inp["X"]), None)
    torch.cuda.synchronize()
    assert st.fw[0]["C"] is None and "H_bf16" not in st.fw[0]
    bsel = slice(0, 8)
    ref = O.stack_forward_backward(inp["X"][:, bsel], inp["layers"], w.direction, None,
                                   w.gemm_dtype, None, need_backward=False)
    check("H", host(H)[:, bsel], ref["Hs"][0], _tol(w))
    check("c_last", host(st.fw[0]["c_last"])[bsel], ref["Cs"][0][-1], _tol(w))
