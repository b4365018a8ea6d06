"""The fused projection + scan of inference (sru_forward with U and C
omitted): H, c_last and the bf16 copy of H equal the unfused call's bit for
bit (the scan reads the same fp32 projections, in the same order), across
k = 3 and 4, tile plans of 2, 4 and 8 sequences, several time blocks per
tile, ragged step and sequence counts, every direction, padding, c0 and the
gate variants; and against the oracle, the linear recurrence included."""

import numpy as np
import pytest
import torch
from hypothesis import HealthCheck, Phase, given, settings
from hypothesis import strategies as st

from helpers import TOL_BF16, check, dev
from oracle import sru_oracle as O
from paper_1709_02755_amd import sru
from paper_1709_02755_amd.workloads import irregular_mask, random_layer_case

pytestmark = pytest.mark.gpu

CASES = [
    # (L, B, d_in, d, direction, masked, alpha, reset_new); d_in != d: k = 4
    (64, 9, 512, 192, O.DIR_FWD, True, 1.0, False),     # 4 per tile (the FFN plan), ragged B
    (50, 6, 128, 64, O.DIR_REV, True, 1.0, False),      # 4 per tile, ragged L
    (40, 5, 256, 128, O.DIR_BI, True, 1.7, True),       # both directions, variants
    (17, 11, 128, 64, O.DIR_BI, False, float(np.sqrt(3.0)), False),  # 8 per tile
    (1, 4, 256, 128, O.DIR_REV, False, 1.0, True),      # a single step
    (64, 80, 512, 2048, O.DIR_FWD, False, 1.0, False),  # the Transformer-FFN shape
    (100, 5, 256, 128, O.DIR_REV, True, 1.0, False),    # 2 per tile, 4 chunks, ragged L and B
    (128, 3, 128, 64, O.DIR_BI, True, 1.3, True),       # 2 per tile, both directions, variants
    # k = 3 (d_in = d): the highway input x_t read from X
    (64, 9, 192, 192, O.DIR_FWD, True, 1.0, False),
    (50, 6, 128, 128, O.DIR_REV, True, 1.7, True),
    (100, 5, 128, 128, O.DIR_BI, True, 1.0, False),
    (17, 11, 64, 64, O.DIR_BI, False, float(np.sqrt(3.0)), False),
    # longer than 128 steps where tiles of two sequences fill the chip: time
    # blocks of 128 steps, c carried from block to block
    (300, 32, 1024, 1024, O.DIR_FWD, True, 1.0, False),  # 3 blocks, the last of 44 steps
    (200, 16, 256, 2048, O.DIR_REV, True, 1.7, True),    # k = 4, reverse
    (150, 16, 1024, 1024, O.DIR_BI, True, 1.0, False),   # both directions, 22-step block
]


def _case(L, B, d_in, d, direction, masked, seed):
    return random_layer_case(np.random.default_rng(seed), L, B, d_in, d, direction,
                             masked=masked, c0=True, bias_scale=0.5, v_scale=0.8)


def _run(c, direction, gv, fused, linear=False):
    L, B, d_in = c["X"].shape
    ndir, k, d = c["W"].shape[:3]
    X, W = dev(c["X"]), dev(c["W"])
    p = [None, None] if linear else [dev(c["v_f"]), dev(c["v_r"])]
    p += [dev(c["b_f"]), dev(c["b_r"])]
    out = dict(U=None if fused else torch.empty((L, B, ndir, k, d), device="cuda"),
               H=torch.empty((L, B, ndir * d), device="cuda"), C=None,
               c_last=torch.empty((B, ndir * d), device="cuda"),
               H_bf16=torch.empty((L, B, ndir * d), dtype=torch.bfloat16, device="cuda"))
    sru.forward(X, W, *p, c0=dev(c["c0"]), direction=direction, mask=dev(c["mask"]),
                gemm_dtype=O.GEMM_BF16, store_c=False, out=out, linear=linear, **gv)
    return out


@pytest.mark.parametrize("case", CASES)
def test_fused_equals_unfused_bitwise(case):
    L, B, d_in, d, direction, masked, alpha, reset_new = case
    print(f"fused L={L} B={B} d_in={d_in} d={d} dir={direction} mask={masked}", flush=True)
    assert sru.fused_available(L, B, d_in, d, direction, O.GEMM_BF16)
    c = _case(L, B, d_in, d, direction, masked, L + d)
    gv = dict(highway_scale=alpha, reset_new=reset_new)
    ref = _run(c, direction, gv, fused=False)
    got = _run(c, direction, gv, fused=True)
    torch.cuda.synchronize()
    for k in ("H", "c_last"):
        assert torch.equal(got[k], ref[k]), k
    assert torch.equal(got["H_bf16"].view(torch.int16), ref["H_bf16"].view(torch.int16))


@pytest.mark.parametrize("linear,L,d_in", [(False, 60, 192), (True, 60, 192), (False, 96, 192),
                                           (False, 70, 128), (True, 40, 128)])
def test_fused_matches_oracle(linear, L, d_in):
    B, d, direction = 6, 128, O.DIR_BI
    c = _case(L, B, d_in, d, direction, True, 5 + linear)
    got = _run(c, direction, {}, fused=True, linear=linear)
    torch.cuda.synchronize()
    v = (None, None) if linear else (c["v_f"], c["v_r"])
    rf = O.forward(c["X"], c["W"], *v, c["b_f"], c["b_r"], c["c0"], direction, c["mask"],
                   O.GEMM_BF16, linear=linear)
    for k in ("H", "c_last"):
        check(k, got[k], rf[k], TOL_BF16)
    m = c["mask"].astype(bool)
    assert np.all(got["H"].cpu().numpy()[m] == 0.0)


def test_fused_not_available_keeps_u_required():
    """Where the fused kernel does not apply (fp32 products, sequences over
    128 steps with too few tiles to fill the chip, d not a multiple of 64) U
    stays required."""
    assert sru.fused_available(128, 2, 128, 64, O.DIR_FWD, O.GEMM_BF16)
    assert sru.fused_available(1024, 32, 1024, 1024, O.DIR_FWD, O.GEMM_BF16)  # 256 tiles
    assert not sru.fused_available(1024, 30, 1024, 1024, O.DIR_FWD, O.GEMM_BF16)  # 240
    assert sru.fused_available(8, 2, 64, 64, O.DIR_FWD, O.GEMM_BF16)   # k = 3
    assert not sru.fused_available(8, 2, 128, 64, O.DIR_FWD, O.GEMM_FP32)
    assert not sru.fused_available(129, 2, 128, 64, O.DIR_FWD, O.GEMM_BF16)
    assert not sru.fused_available(8, 2, 96, 32, O.DIR_FWD, O.GEMM_BF16)


SETTINGS = dict(deadline=None, derandomize=True, database=None, phases=[Phase.generate],
                suppress_health_check=list(HealthCheck))


@st.composite
def fused_cases(draw):
    L = draw(st.integers(1, 128))
    B = draw(st.integers(1, 12))
    d = draw(st.sampled_from([64, 128]))
    d_in = draw(st.sampled_from([d, 8, 72, 192]))  # d: k = 3, else k = 4
    direction = draw(st.sampled_from([O.DIR_FWD, O.DIR_REV, O.DIR_BI]))
    mask = draw(st.sampled_from(["none", "suffix", "irregular"]))
    alpha = draw(st.sampled_from([1.0, 1.7]))
    reset_new = draw(st.booleans())
    seed = draw(st.integers(0, 2 ** 16))
    return L, B, d_in, d, direction, mask, alpha, reset_new, seed


@settings(max_examples=40, **SETTINGS)
@given(case=fused_cases())
def test_fused_equals_unfused_on_random_cases(case):
    """Random small shapes up to 128 steps, k = 3 and 4, every direction,
    padding pattern and gate variant: the fused kernel's H, c_last and bf16
    H equal the separate product and scan's, bit for bit.  (The linear
    recurrence's separate scan evaluates its gates another way; its fused
    results are held to the oracle above.)"""
    L, B, d_in, d, direction, mask, alpha, reset_new, seed = case
    print(f"fused case {case}", flush=True)
    rng = np.random.default_rng(seed)
    c = random_layer_case(rng, L, B, d_in, d, direction, masked=mask == "suffix", c0=True,
                          bias_scale=0.5, v_scale=0.8)
    if mask == "irregular":
        c["mask"] = irregular_mask(rng, L, B)
    assert sru.fused_available(L, B, d_in, d, direction, O.GEMM_BF16)
    gv = dict(highway_scale=alpha, reset_new=reset_new)
    ref = _run(c, direction, gv, fused=False)
    got = _run(c, direction, gv, fused=True)
    torch.cuda.synchronize()
    for k in ("H", "c_last"):
        assert torch.equal(got[k], ref[k]), (k, case)
    assert torch.equal(got["H_bf16"].view(torch.int16), ref["H_bf16"].view(torch.int16)), case
