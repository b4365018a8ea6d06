"""Property tests: the GPU layer equals the oracle on randomly drawn small
cases (shapes, seeds, directions, padding patterns, gate variants, product
precision, c0 / dc_last), forward and backward through the C ABI.

Bounded and reproducible: a fixed number of derandomized examples, and no
shrinking phase, so a failure stops the test at the first failing case
(whose parameters the assertion prints).  Every call runs on a workspace
of the queried size followed by a guard region that must come back
untouched.

The cases include one-element tensors and sums whose terms cancel, where a
relative bar has no RMS to fall back on: beside the parity bars (1e-5 fp32,
2e-2 bf16, relative to max(|ref|, rms(ref))), an element may differ by
SLACK times how far the oracle itself moves when its inputs carry
rounding-sized noise.  A logic error (wrong index, term, sign or state)
moves results by orders of magnitude more."""

import numpy as np
import pytest
import torch
from hypothesis import HealthCheck, Phase, given, settings
from hypothesis import strategies as st

from helpers import TOL_BF16, TOL_FP32, dev, host
from oracle import sru_oracle as O
from paper_1709_02755_amd import sru
from paper_1709_02755_amd.workloads import irregular_mask, lengths_to_mask, random_layer_case

pytestmark = pytest.mark.gpu

PERTURB = 2.0 ** -18  # relative input noise: 64 fp32 rounding units
SLACK = 4.0


def sensitivity(run, inputs, keys, draws=2, seed=0):
    """How far each output of the oracle moves when its inputs move by
    PERTURB relative noise (max over `draws` draws): the scale of what fp32
    rounding of inputs and intermediates can do to that element, which
    matters where terms cancel (in a one-element tensor there is no RMS
    floor to absorb it)."""
    rng = np.random.default_rng(seed)
    ref = run(inputs)
    sens = {k: np.zeros_like(np.asarray(ref[k], np.float64)) for k in keys}
    for _ in range(draws):
        pert = {k: (None if v is None or not np.issubdtype(np.asarray(v).dtype, np.floating)
                    else np.asarray(v, np.float64) * (1.0 + PERTURB * rng.standard_normal(np.shape(v))))
                for k, v in inputs.items()}
        pert = {k: (inputs[k] if pert[k] is None else pert[k]) for k in inputs}
        out = run(pert)
        for k in keys:
            sens[k] = np.maximum(sens[k], np.abs(np.asarray(out[k]) - np.asarray(ref[k])))
    return ref, sens


def check_sens(name, got, ref, tol, sens):
    """Each element within tol of max(|ref|, rms(ref)), or within SLACK times
    the oracle's own sensitivity to rounding-sized input noise there."""
    g, r = host(got), np.asarray(ref, np.float64)
    rms = float(np.sqrt(np.mean(r * r))) if r.size else 0.0
    allowed = np.maximum(tol * np.maximum(np.abs(r), rms), SLACK * sens)
    bad = np.abs(g - r) > allowed
    assert np.all(np.isfinite(g)) and not bad.any(), \
        f"{name}: {int(bad.sum())} elements beyond the bound, worst excess " \
        f"{float(np.max(np.abs(g - r) - allowed)):.3e}"


SETTINGS = dict(deadline=None, derandomize=True, database=None, phases=[Phase.generate],
                suppress_health_check=list(HealthCheck))

GUARD, FILL = 1 << 20, 0xA5


def guarded(need):
    """A workspace of `need` bytes followed by a guard region: (buffer, ws)."""
    buf = torch.full((max(need, 1) + GUARD,), FILL, dtype=torch.uint8, device="cuda")
    return buf, buf[:max(need, 1)]


def guard_intact(buf, need, what):
    assert bool(torch.all(buf[max(need, 1):] == FILL)), f"{what} wrote past its workspace"


@st.composite
def layer_cases(draw):
    d = draw(st.integers(1, 96))
    k4 = draw(st.booleans())
    d_in = draw(st.integers(1, 96).filter(lambda x: x != d)) if k4 else d
    linear = draw(st.booleans())
    return dict(
        L=draw(st.integers(1, 40)), B=draw(st.integers(1, 6)), d=d, d_in=d_in,
        direction=draw(st.sampled_from([O.DIR_FWD, O.DIR_REV, O.DIR_BI])),
        mask=draw(st.sampled_from(["none", "lengths", "irregular"])),
        gemm=draw(st.sampled_from([O.GEMM_FP32, O.GEMM_BF16])),
        alpha=draw(st.sampled_from([1.0, float(np.sqrt(3.0)), 0.6])),
        reset_new=(not linear) and draw(st.booleans()), linear=linear,
        c0=draw(st.booleans()), dc_last=draw(st.booleans()),
        seed=draw(st.integers(0, 2 ** 31 - 1)))


def _inputs(case):
    rng = np.random.default_rng(case["seed"])
    L, B = case["L"], case["B"]
    c = random_layer_case(rng, L, B, case["d_in"], case["d"], case["direction"],
                          c0=case["c0"], dc_last=case["dc_last"], bias_scale=0.7, v_scale=0.8)
    if case["mask"] == "lengths":
        c["mask"] = lengths_to_mask(rng.integers(1, L + 1, size=B), L)
    elif case["mask"] == "irregular":
        c["mask"] = irregular_mask(rng, L, B)
    return c


@st.composite
def time_parallel_cases(draw):
    """Gated layers with 8,192 to 32,767 lanes (B * ndir * d), where the
    backward scan runs in time-parallel chunks; short sequences keep the
    oracle fast."""
    direction = draw(st.sampled_from([O.DIR_FWD, O.DIR_REV, O.DIR_BI]))
    ndir = 2 if direction == O.DIR_BI else 1
    d = draw(st.sampled_from([128, 256, 512]))
    lo = -(-8192 // (ndir * d))
    B = draw(st.integers(lo, min(32767 // (ndir * d), lo + 24)))
    k4 = draw(st.booleans())
    return dict(
        L=draw(st.integers(1, 24)), B=B, d=d,
        d_in=draw(st.sampled_from([64, 96, 200])) if k4 else d, direction=direction,
        mask=draw(st.sampled_from(["none", "lengths", "irregular"])),
        gemm=draw(st.sampled_from([O.GEMM_FP32, O.GEMM_BF16])),
        alpha=draw(st.sampled_from([1.0, float(np.sqrt(3.0)), 0.6])),
        reset_new=draw(st.booleans()), linear=False,
        c0=draw(st.booleans()), dc_last=draw(st.booleans()),
        seed=draw(st.integers(0, 2 ** 31 - 1)))


@settings(max_examples=150, **SETTINGS)
@given(case=layer_cases())
def test_layer_equals_oracle_on_random_cases(case):
    check_layer_case(case)


@settings(max_examples=25, **SETTINGS)
@given(case=time_parallel_cases())
def test_time_parallel_layer_equals_oracle_on_random_cases(case):
    check_layer_case(case)


def check_layer_case(case):
    print(f"property case {case}", flush=True)
    c = _inputs(case)
    direction, gemm, linear = case["direction"], case["gemm"], case["linear"]
    var = dict(highway_scale=case["alpha"], reset_new=case["reset_new"], linear=linear)
    p = [None if linear else dev(c["v_f"]), None if linear else dev(c["v_r"]),
         dev(c["b_f"]), dev(c["b_r"])]
    X, W, c0, mask = dev(c["X"]), dev(c["W"]), dev(c["c0"]), dev(c["mask"])
    L, B, d_in, d = case["L"], case["B"], case["d_in"], case["d"]
    nf = sru.forward_workspace_bytes(L, B, d_in, d, direction, gemm)
    nb = sru.backward_workspace_bytes(L, B, d_in, d, direction, gemm)
    (fbuf, fws), (bbuf, bws) = guarded(nf), guarded(nb)
    fw = sru.forward(X, W, *p, c0=c0, direction=direction, mask=mask, gemm_dtype=gemm, ws=fws,
                     **var)
    bw = sru.backward(X, W, *p, fw["U"], fw["C"], dev(c["dH"]), c0=c0,
                      dc_last=dev(c["dc_last"]), direction=direction, mask=mask,
                      gemm_dtype=gemm, ws=bws, **var)
    torch.cuda.synchronize()
    guard_intact(fbuf, nf, "the forward")
    guard_intact(bbuf, nb, "the backward")
    ov = dict(alpha=case["alpha"], reset_new=case["reset_new"], linear=linear)

    def run(x):
        args = (x["X"], x["W"], x["v_f"], x["v_r"], x["b_f"], x["b_r"])
        f = O.forward(*args, x["c0"], direction, c["mask"], gemm, **ov)
        b = O.backward(*args, x["dH"], x["c0"], direction, c["mask"], gemm, x["dc_last"], fw=f,
                       **ov)
        return {**{k: f[k] for k in ("U", "H", "C", "c_last")},
                **{k: b[k] for k in ("dX", "dW", "dv_f", "dv_r", "db_f", "db_r", "dc0")}}
    keys = ["U", "H", "C", "c_last", "dX", "dW", "db_f", "db_r", "dc0"] + \
        ([] if linear else ["dv_f", "dv_r"])
    ref, sens = sensitivity(run, {k: c[k] for k in ("X", "W", "v_f", "v_r", "b_f", "b_r", "c0",
                                                     "dH", "dc_last")}, keys)
    tol = TOL_FP32 if gemm == O.GEMM_FP32 else TOL_BF16
    out = {**fw, **bw}
    for key in keys:
        check_sens(key, out[key], ref[key], TOL_FP32 if key == "U" else tol, sens[key])
    if c["mask"] is not None:
        m = c["mask"].astype(bool)
        assert np.all(host(fw["H"])[m] == 0.0) and np.all(host(bw["dX"])[m] == 0.0)


@st.composite
def lowrank_cases(draw):
    d = draw(st.integers(2, 64))
    k4 = draw(st.booleans())
    gemm = draw(st.sampled_from([O.GEMM_FP32, O.GEMM_BF16]))
    if gemm == O.GEMM_BF16:  # bf16 low-rank products need whole 16-byte chunks
        d = 8 * max(1, d // 8)
        d_in = 8 * draw(st.integers(1, 12).filter(lambda x: 8 * x != d)) if k4 else d
        dp = 8 * draw(st.integers(1, 6))
    else:
        d_in = draw(st.integers(1, 80).filter(lambda x: x != d)) if k4 else d
        dp = draw(st.integers(1, 40))
    return dict(L=draw(st.integers(1, 32)), B=draw(st.integers(1, 5)), d=d, d_in=d_in, dp=dp,
                direction=draw(st.sampled_from([O.DIR_FWD, O.DIR_REV, O.DIR_BI])),
                mask=draw(st.sampled_from(["none", "lengths", "irregular"])), gemm=gemm,
                c0=True, dc_last=draw(st.booleans()), seed=draw(st.integers(0, 2 ** 31 - 1)))


@settings(max_examples=60, **SETTINGS)
@given(case=lowrank_cases())
def test_lowrank_layer_equals_oracle_on_random_cases(case):
    print(f"property case {case}", flush=True)
    c = _inputs(case)
    rng = np.random.default_rng(case["seed"] + 1)
    ndir, k = c["W"].shape[:2]
    d_in, d, dp = case["d_in"], case["d"], case["dp"]
    Q = rng.uniform(-1, 1, (d_in, dp)).astype(np.float32) * np.float32(np.sqrt(3.0 / d_in))
    P = rng.uniform(-1, 1, (ndir, k, d, dp)).astype(np.float32) * np.float32(np.sqrt(3.0 / dp))
    direction, gemm = case["direction"], case["gemm"]
    p = [dev(c[key]) for key in ("v_f", "v_r", "b_f", "b_r")]
    X, c0, mask = dev(c["X"]), dev(c["c0"]), dev(c["mask"])
    lib = sru.lib()
    L, B = case["L"], case["B"]
    nf = lib.sru_forward_lowrank_workspace_bytes(L, B, d_in, d, dp, direction, gemm)
    nb = lib.sru_backward_lowrank_workspace_bytes(L, B, d_in, d, dp, direction, gemm)
    (fbuf, fws), (bbuf, bws) = guarded(nf), guarded(nb)
    fw = sru.forward_lowrank(X, dev(Q), dev(P), *p, c0=c0, direction=direction, mask=mask,
                             gemm_dtype=gemm, ws=fws)
    bw = sru.backward_lowrank(X, dev(Q), dev(P), *p, fw["T"], fw["U"], fw["C"], dev(c["dH"]),
                              c0=c0, dc_last=dev(c["dc_last"]), direction=direction, mask=mask,
                              gemm_dtype=gemm, ws=bws)
    torch.cuda.synchronize()
    guard_intact(fbuf, nf, "the low-rank forward")
    guard_intact(bbuf, nb, "the low-rank backward")

    def run(x):
        args = (x["X"], x["Q"], x["P"], x["v_f"], x["v_r"], x["b_f"], x["b_r"])
        f = O.forward_lowrank(*args, x["c0"], direction, c["mask"], gemm)
        b = O.backward_lowrank(*args, x["dH"], x["c0"], direction, c["mask"], gemm,
                               x["dc_last"], fw=f)
        return {**{k: f[k] for k in ("T", "U", "H", "C", "c_last")},
                **{k: b[k] for k in ("dX", "dQ", "dP", "dv_f", "dv_r", "db_f", "db_r", "dc0")}}
    keys = ["T", "U", "H", "C", "c_last", "dX", "dQ", "dP", "dv_f", "dv_r", "db_f", "db_r", "dc0"]
    inputs = dict(X=c["X"], Q=Q, P=P, v_f=c["v_f"], v_r=c["v_r"], b_f=c["b_f"], b_r=c["b_r"],
                  c0=c["c0"], dH=c["dH"], dc_last=c["dc_last"])
    ref, sens = sensitivity(run, inputs, keys)
    tol = TOL_FP32 if gemm == O.GEMM_FP32 else TOL_BF16
    out = {**fw, **bw}
    for key in keys:
        check_sens(key, out[key], ref[key], tol, sens[key])
