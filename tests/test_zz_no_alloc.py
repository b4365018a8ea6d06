"""sru_forward_noalloc (the forward whose workspace is a static device array)
against sru_forward with a caller workspace, through the C ABI.

Both run the same kernels, so the results must be identical bit for bit.
Each case makes two calls in a row, the second on a smaller input, so the
second call runs on an array that still holds the first call's contents."""

import numpy as np
import pytest
import torch

from helpers import dev
from oracle import sru_oracle as O
from paper_1709_02755_amd import sru
from paper_1709_02755_amd.workloads import random_layer_case

pytestmark = pytest.mark.gpu

# (L, B, d_in, d, direction, masked, gemm, linear, fused)
CASES = [
    [(64, 16, 512, 512, O.DIR_FWD, False, O.GEMM_BF16, False, False),
     (24, 5, 128, 128, O.DIR_FWD, True, O.GEMM_BF16, False, False)],
    [(48, 6, 256, 128, O.DIR_BI, True, O.GEMM_BF16, False, False),
     (17, 3, 64, 32, O.DIR_REV, True, O.GEMM_BF16, False, False)],
    # the linear recurrence with few lanes: time segments keep maps in the array
    [(400, 2, 64, 64, O.DIR_FWD, True, O.GEMM_FP32, True, False),
     (150, 1, 64, 64, O.DIR_BI, False, O.GEMM_FP32, True, False)],
    # inference with the fused projection + scan (U and C not kept)
    [(32, 8, 128, 256, O.DIR_FWD, True, O.GEMM_BF16, False, True),
     (16, 4, 64, 128, O.DIR_FWD, False, O.GEMM_BF16, False, True)],
]


def _outputs(L, B, d_in, d, ndir, k, bf16, fused):
    o = dict(U=None if fused else torch.empty((L, B, ndir, k, d), device="cuda"),
             H=torch.empty((L, B, ndir * d), device="cuda"),
             C=None if fused else torch.empty((L, B, ndir * d), device="cuda"),
             c_last=torch.empty((B, ndir * d), device="cuda"))
    if bf16:
        o["W_bf16"] = torch.empty((ndir, k, d, d_in), dtype=torch.bfloat16, device="cuda")
        o["H_bf16"] = torch.empty((L, B, ndir * d), dtype=torch.bfloat16, device="cuda")
    for t in o.values():
        if t is not None:
            t.fill_(float("nan")) if t.dtype == torch.float32 else t.fill_(0)
    return o


@pytest.mark.parametrize("pair", CASES)
def test_noalloc_forward_equals_forward_with_workspace(pair):
    for call, (L, B, d_in, d, direction, masked, gemm, linear, fused) in enumerate(pair):
        print(f"noalloc call {call}: L={L} B={B} d_in={d_in} d={d} dir={direction} "
              f"mask={masked} gemm={gemm} linear={linear} fused={fused}", flush=True)
        rng = np.random.default_rng(100 * L + B)
        c = random_layer_case(rng, L, B, d_in, d, direction, masked=masked, c0=True,
                              bias_scale=0.5)
        ndir, k = c["W"].shape[:2]
        bf16 = gemm == O.GEMM_BF16
        need = sru.forward_workspace_bytes(L, B, d_in, d, direction, gemm)
        assert need <= sru.NOALLOC_SCRATCH_BYTES
        if fused:
            assert sru.fused_available(L, B, d_in, d, direction, gemm)
        p = [dev(c[key]) for key in ("v_f", "v_r", "b_f", "b_r")]
        X, W, c0, mask = dev(c["X"]), dev(c["W"]), dev(c["c0"]), dev(c["mask"])
        kw = dict(c0=c0, direction=direction, mask=mask, gemm_dtype=gemm, linear=linear)
        ref = _outputs(L, B, d_in, d, ndir, k, bf16, fused)
        sru.forward(X, W, *p, out=ref, store_c=not fused, **kw)
        got = _outputs(L, B, d_in, d, ndir, k, bf16, fused)
        sru.forward_noalloc(X, W, *p, out=got, **kw)
        torch.cuda.synchronize()
        for key, t in ref.items():
            if t is None:
                assert got[key] is None
                continue
            a, b = t.cpu(), got[key].cpu()
            if a.dtype == torch.bfloat16:
                a, b = a.view(torch.int16), b.view(torch.int16)
            assert torch.equal(a, b), (call, key)
        # and the shared result is the oracle's (the layer's parity bar)
        rf = O.forward(c["X"], c["W"], c["v_f"], c["v_r"], c["b_f"], c["b_r"], c["c0"],
                       direction, c["mask"], gemm, linear=linear)
        h = got["H"].cpu().numpy().astype(np.float64)
        rms = np.sqrt(np.mean(rf["H"] ** 2))
        err = float(np.max(np.abs(h - rf["H"]) / np.maximum(np.abs(rf["H"]), rms)))
        assert err <= (2e-2 if bf16 else 1e-5), (call, err)


def test_noalloc_forward_refuses_an_oversized_shape():
    """A forward workspace beyond the array is SRU_E_WORKSPACE; nothing runs."""
    L, B, d = 1024, 128, 1024
    assert sru.forward_workspace_bytes(L, B, d, d, O.DIR_FWD, O.GEMM_BF16) > \
        sru.NOALLOC_SCRATCH_BYTES
    X = torch.zeros((L, B, d), device="cuda")
    W = torch.zeros((1, 3, d, d), device="cuda")
    z = torch.zeros((1, d), device="cuda")
    H = torch.full((L, B, d), 7.0, device="cuda")
    with pytest.raises(sru.SruError, match="WORKSPACE"):
        sru.forward_noalloc(X, W, z, z, z, z, gemm_dtype=O.GEMM_BF16, out=dict(
            U=torch.empty((L, B, 1, 3, d), device="cuda"), H=H))
    torch.cuda.synchronize()
    assert bool((H == 7.0).all())
