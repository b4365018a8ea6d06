"""The bf16 companions of the bf16-GEMM mode.  sru_forward can write bf16
copies of Wcat and H, and sru_forward / sru_backward can take bf16 copies of
X and Wcat instead of rounding them again.  A copy that equals the library's
own rounding must give bit-identical results; the copies it writes must be
exactly the round-to-nearest-even bf16 of Wcat and H; and the Stack, which
wires H_bf16 of one layer into the next, must equal per-layer calls without
companions.  Weights held in bf16 (a bfloat16 W, passed as the W_bf16 input
with W = NULL) give the same bits as fp32 weights rounded by the library."""

import numpy as np
import pytest
import torch

from helpers import dev
from oracle import sru_oracle as O
from paper_1709_02755_amd import sru
from paper_1709_02755_amd.workloads import random_layer_case

pytestmark = pytest.mark.gpu

CASES = [
    # (L, B, d_in, d, direction, masked): direct kernels, and (d_in = 60)
    # the paths for operands whose rows are not whole 16-byte chunks
    (33, 9, 256, 256, O.DIR_FWD, False),
    (20, 6, 128, 64, O.DIR_BI, True),
    (17, 5, 64, 64, O.DIR_REV, True),
    (12, 3, 60, 60, O.DIR_FWD, True),
]


def bits(t):
    return t.contiguous().view(torch.int16)


def same(a, b):
    return all(torch.equal(a[k], b[k]) for k in a if a[k] is not None and k in b)


@pytest.mark.parametrize("case", CASES)
def test_companions_bit_identical(case):
    L, B, d_in, d, direction, masked = case
    print(f"bf16 companions L={L} B={B} d_in={d_in} d={d} dir={direction}", flush=True)
    c = random_layer_case(np.random.default_rng(L * 7 + d), L, B, d_in, d, direction,
                          masked=masked, c0=True, dc_last=True, bias_scale=0.5)
    X, W = dev(c["X"]), dev(c["W"])
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    kw = dict(c0=dev(c["c0"]), direction=direction, mask=dev(c["mask"]), gemm_dtype=O.GEMM_BF16)
    ndir = 2 if direction == O.DIR_BI else 1

    fw0 = sru.forward(X, W, *p, **kw)
    k = W.shape[1]
    out = dict(U=torch.empty((L, B, ndir, k, d), device="cuda"),
               H=torch.empty((L, B, ndir * d), device="cuda"),
               C=torch.empty((L, B, ndir * d), device="cuda"),
               c_last=torch.empty((B, ndir * d), device="cuda"),
               W_bf16=torch.empty(tuple(W.shape), dtype=torch.bfloat16, device="cuda"),
               H_bf16=torch.empty((L, B, ndir * d), dtype=torch.bfloat16, device="cuda"))
    fw1 = sru.forward(X, W, *p, out=out, **kw)
    fw2 = sru.forward(X, W, *p, X_bf16=X.to(torch.bfloat16), **kw)
    torch.cuda.synchronize()
    for key in ("U", "H", "C", "c_last"):
        assert torch.equal(fw0[key], fw1[key]), key
        assert torch.equal(fw0[key], fw2[key]), key
    assert torch.equal(bits(fw1["W_bf16"]), bits(W.to(torch.bfloat16)))
    assert torch.equal(bits(fw1["H_bf16"]), bits(fw1["H"].to(torch.bfloat16)))

    args = (fw0["U"], fw0["C"], dev(c["dH"]))
    bkw = dict(kw, dc_last=dev(c["dc_last"]))
    bw0 = sru.backward(X, W, *p, *args, **bkw)
    bw1 = sru.backward(X, W, *p, *args, X_bf16=X.to(torch.bfloat16), W_bf16=fw1["W_bf16"], **bkw)
    bw2 = sru.backward(X, W, *p, *args, W_bf16=fw1["W_bf16"], **bkw)
    torch.cuda.synchronize()
    # the weights held in bf16 (W = NULL, W_bf16 read as the input)
    Wb = sru.round_bf16(W)
    fw3 = sru.forward(X, Wb, *p, **kw)
    bw3 = sru.backward(X, Wb, *p, *args, **bkw)
    torch.cuda.synchronize()
    for key in ("U", "H", "C", "c_last"):
        assert torch.equal(fw0[key], fw3[key]), key
    for key in bw0:
        if bw0[key] is None:
            continue
        assert torch.equal(bw0[key], bw1[key]), key
        assert torch.equal(bw0[key], bw2[key]), key
        assert torch.equal(bw0[key], bw3[key]), key


def test_stack_wiring_equals_plain_calls():
    L, B, d, layers = 16, 8, 128, 3
    rng = np.random.default_rng(5)
    cs = [random_layer_case(rng, L, B, d, d, O.DIR_FWD, masked=True, dc_last=False,
                            bias_scale=0.5) for _ in range(layers)]
    X, mask, dH = dev(cs[0]["X"]), dev(cs[0]["mask"]), dev(cs[-1]["dH"])
    ps = [{k: dev(c[k]) for k in ("W", "v_f", "v_r", "b_f", "b_r")} for c in cs]
    st = sru.Stack(ps, L, B, d, d, O.DIR_FWD, O.GEMM_BF16, torch.device("cuda"))
    H = st.forward(X, mask).clone()
    dX = st.backward(X, dH, mask).clone()
    grads = [{k: v.clone() for k, v in b.items() if v is not None} for b in st.bw]

    xs, fws = [X], []
    for p in ps:
        fws.append(sru.forward(xs[-1], p["W"], p["v_f"], p["v_r"], p["b_f"], p["b_r"], mask=mask,
                               gemm_dtype=O.GEMM_BF16))
        xs.append(fws[-1]["H"])
    g = dH
    ref = [None] * layers
    for li in range(layers - 1, -1, -1):
        p = ps[li]
        ref[li] = sru.backward(xs[li], p["W"], p["v_f"], p["v_r"], p["b_f"], p["b_r"],
                               fws[li]["U"], fws[li]["C"], g, mask=mask, gemm_dtype=O.GEMM_BF16)
        g = ref[li]["dX"]
    torch.cuda.synchronize()
    assert torch.equal(H, xs[-1])
    assert torch.equal(dX, g)
    for li in range(layers):
        for key, v in grads[li].items():
            assert torch.equal(v, ref[li][key]), (li, key)


def test_inference_stack_with_bf16_weights():
    """Inference at the fused kernel's shape (k = 4, L <= 128) with the
    weights held in bf16 (rounded once) equals the stack that rounds them on
    every call, bit for bit; so does the allocation-free forward."""
    L, B, d_in, d = 24, 10, 64, 128
    rng = np.random.default_rng(17)
    c = random_layer_case(rng, L, B, d_in, d, O.DIR_BI, masked=True, bias_scale=0.5)
    X, mask = dev(c["X"]), dev(c["mask"])
    p = {k: dev(c[k]) for k in ("W", "v_f", "v_r", "b_f", "b_r")}
    assert sru.fused_available(L, B, d_in, d, O.DIR_BI, O.GEMM_BF16)
    a = sru.Stack([p], L, B, d_in, d, O.DIR_BI, O.GEMM_BF16, torch.device("cuda"),
                  backward=False, store_c=False)
    b = sru.Stack([dict(p, W=sru.round_bf16(p["W"]))], L, B, d_in, d, O.DIR_BI, O.GEMM_BF16,
                  torch.device("cuda"), backward=False, store_c=False)
    Ha = a.forward(X, mask).clone()
    Hb = b.forward(X, mask).clone()
    out = dict(H=torch.empty_like(Ha), c_last=torch.empty((B, 2 * d), device="cuda"))
    sru.forward_noalloc(X, b.layers[0]["W"], p["v_f"], p["v_r"], p["b_f"], p["b_r"],
                        direction=O.DIR_BI, mask=mask, gemm_dtype=O.GEMM_BF16, out=out)
    torch.cuda.synchronize()
    assert a.fw[0]["U"] is None and b.fw[0]["U"] is None  # the fused kernel ran
    assert torch.equal(Ha, Hb)
    assert torch.equal(Ha, out["H"])
    assert torch.equal(a.fw[0]["c_last"], out["c_last"])


@pytest.mark.parametrize("n", [1, 7, 8, 4099, 1 << 20])
def test_round_bf16_equals_rne_cast(n):
    """sru_round_bf16 gives torch's round-to-nearest-even bf16 bit for bit,
    including ties, infinities and a ragged tail."""
    x = torch.randn(n, device="cuda") * 10.0
    if n >= 8:
        x[:4] = torch.tensor([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, float("inf"), -0.0])
    got = sru.round_bf16(x)
    torch.cuda.synchronize()
    assert torch.equal(bits(got), bits(x.to(torch.bfloat16)))
