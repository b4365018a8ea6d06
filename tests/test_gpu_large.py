"""Maximum sizes: one bf16 layer whose tensors pass 2 GiB.  dU in bf16 is
2.4 GB, beyond the byte range of a buffer resource over the whole operand,
so the direct products address it from each workgroup's own panel (a
tile's rows for dX, a split's k-rows for dW); U is 4.8 GB and every scan
offset runs past 2^31 elements of H and C.  Sequences never interact, so the
oracle on the first and the last sequence (the highest offsets of every
tensor) is exact for their outputs.  dH is zero on every other sequence,
whose gradients are then exactly zero: the parameter gradients (dW, summed
over all 393,216 tokens, and the v/b sums) equal the sum of the two
sequences' oracle gradients."""

import numpy as np
import pytest
import torch

from helpers import TOL_BF16, check, dev
from oracle import sru_oracle as O
from paper_1709_02755_amd import sru

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def test_layer_with_tensors_beyond_2gib():
    L, B, d = 1024, 384, 1024
    print(f"large layer L={L} B={B} d={d} bf16", flush=True)
    rng = np.random.default_rng(77)
    X = rng.standard_normal((L, B, d), dtype=np.float32)
    bound = np.sqrt(3.0 / d)
    W = rng.uniform(-bound, bound, (1, 3, d, d)).astype(np.float32)
    v_f, v_r = (rng.uniform(-0.5, 0.5, (1, d)).astype(np.float32) for _ in range(2))
    b_f = rng.uniform(-1, 1, (1, d)).astype(np.float32)
    b_r = np.zeros((1, d), np.float32)
    dH = np.zeros((L, B, d), np.float32)
    for b in (0, B - 1):
        dH[:, b] = rng.standard_normal((L, d), dtype=np.float32)
    M, N = L * B, 3 * d
    assert 2 * M * N > 2 ** 31 and 4 * M * N > 2 ** 32

    p = [dev(a) for a in (v_f, v_r, b_f, b_r)]
    Xd, Wd = dev(X), dev(W)
    fw = sru.forward(Xd, Wd, *p, gemm_dtype=O.GEMM_BF16)
    bw = sru.backward(Xd, Wd, *p, fw["U"], fw["C"], dev(dH), gemm_dtype=O.GEMM_BF16)
    torch.cuda.synchronize()
    grads = {k: 0.0 for k in ("dW", "dv_f", "dv_r", "db_f", "db_r")}
    for b in (0, B - 1):
        sl = slice(b, b + 1)
        args = (X[:, sl], W, v_f, v_r, b_f, b_r)
        rf = O.forward(*args, None, O.DIR_FWD, None, O.GEMM_BF16)
        rb = O.backward(*args, dH[:, sl], None, O.DIR_FWD, None, O.GEMM_BF16, fw=rf)
        for k in grads:
            grads[k] = grads[k] + np.asarray(rb[k], np.float64)
        for k in ("H", "C"):
            check(f"{k}[b={b}]", fw[k][:, sl], rf[k], TOL_BF16)
        check(f"c_last[b={b}]", fw["c_last"][sl], rf["c_last"], TOL_BF16)
        check(f"dX[b={b}]", bw["dX"][:, sl], rb["dX"], TOL_BF16)
        check(f"dc0[b={b}]", bw["dc0"][sl], rb["dc0"], TOL_BF16)
    for k, ref in grads.items():
        check(k, bw[k], ref, TOL_BF16)
