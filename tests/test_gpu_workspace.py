"""The library's writes stay inside the workspace it asks for.  The dX
product may be split over K; the split partials sit at the end of the
backward workspace, sized from the same product descriptor the launch
uses (with the highway addend, which decides the tile shape and with it
the split count).  Each case runs the backward on a workspace followed by a
guard region and checks that the guard is untouched and that the results
equal those of a run on a workspace of exactly the queried size."""

import numpy as np
import pytest
import torch

from helpers import dev
from oracle import sru_oracle as O
from paper_1709_02755_amd import sru
from paper_1709_02755_amd.workloads import random_layer_case

pytestmark = pytest.mark.gpu

GUARD = 16 << 20
FILL = 0xA5


@pytest.mark.parametrize("L,B,d,direction", [
    (256, 16, 1024, O.DIR_FWD),   # dX split 4 ways on 256 x 256 tiles, dW 5 ways
    (96, 8, 1024, O.DIR_BI),      # two addends (both directions' highway gradients)
    (128, 8, 2048, O.DIR_FWD),
    (256, 8, 1024, O.DIR_FWD),    # one GPU's shard of the headline batch
])
def test_backward_stays_inside_its_workspace(L, B, d, direction):
    print(f"workspace guard L={L} B={B} d={d} dir={direction}", flush=True)
    c = random_layer_case(np.random.default_rng(L + B + d), L, B, d, d, direction,
                          masked=False, bias_scale=0.5)
    X, W = dev(c["X"]), dev(c["W"])
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    kw = dict(direction=direction, gemm_dtype=O.GEMM_BF16)
    fw = sru.forward(X, W, *p, **kw)
    need = sru.backward_workspace_bytes(L, B, d, d, direction, O.GEMM_BF16)
    buf = torch.full((need + GUARD,), FILL, dtype=torch.uint8, device="cuda")
    bw = sru.backward(X, W, *p, fw["U"], fw["C"], dev(c["dH"]), ws=buf[:need], **kw)
    ref = sru.backward(X, W, *p, fw["U"], fw["C"], dev(c["dH"]),
                       ws=torch.empty(need, dtype=torch.uint8, device="cuda"), **kw)
    torch.cuda.synchronize()
    assert bool(torch.all(buf[need:] == FILL)), "a kernel wrote past the workspace"
    for k in ("dX", "dW", "dv_f", "dv_r", "db_f", "db_r", "dc0"):
        assert torch.equal(bw[k], ref[k]), k


@pytest.mark.parametrize("linear", [False, True])
def test_forward_and_lowrank_backward_stay_inside(linear):
    """The same guard for the forward (bf16 operand copies, the linear
    recurrence's segment maps) and the low-rank backward (dP and dQ split)."""
    L, B, d_in, d, dp = 128, 12, 512, 512, 128
    print(f"workspace guard fwd + lowrank L={L} B={B} d={d} dp={dp} linear={linear}", flush=True)
    rng = np.random.default_rng(31)
    c = random_layer_case(rng, L, B, d_in, d, O.DIR_FWD, masked=True, bias_scale=0.5)
    X = dev(c["X"])
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    Q = dev((rng.uniform(-1, 1, (d_in, dp)) * np.sqrt(3.0 / d_in)).astype(np.float32))
    P = dev((rng.uniform(-1, 1, (1, 3, d, dp)) * np.sqrt(3.0 / dp)).astype(np.float32))
    kw = dict(mask=dev(c["mask"]), gemm_dtype=O.GEMM_BF16, linear=linear)
    lib = sru.lib()

    need_f = sru.forward_workspace_bytes(L, B, d_in, d, O.DIR_FWD, O.GEMM_BF16)
    buf = torch.full((need_f + GUARD,), FILL, dtype=torch.uint8, device="cuda")
    fw = sru.forward(X, dev(c["W"]), *p, ws=buf[:need_f], **kw)
    torch.cuda.synchronize()
    assert bool(torch.all(buf[need_f:] == FILL)), "the forward wrote past its workspace"

    need_lf = lib.sru_forward_lowrank_workspace_bytes(L, B, d_in, d, dp, O.DIR_FWD, O.GEMM_BF16)
    need_lb = lib.sru_backward_lowrank_workspace_bytes(L, B, d_in, d, dp, O.DIR_FWD, O.GEMM_BF16)
    lf = sru.forward_lowrank(X, Q, P, *p, **kw)
    buf = torch.full((need_lb + GUARD,), FILL, dtype=torch.uint8, device="cuda")
    lb = sru.backward_lowrank(X, Q, P, *p, lf["T"], lf["U"], lf["C"], dev(c["dH"]),
                              ws=buf[:need_lb], **kw)
    ref = sru.backward_lowrank(X, Q, P, *p, lf["T"], lf["U"], lf["C"], dev(c["dH"]), **kw)
    torch.cuda.synchronize()
    assert need_lf > 0 and fw["H"] is not None
    assert bool(torch.all(buf[need_lb:] == FILL)), "the low-rank backward wrote past its workspace"
    for k in ("dX", "dQ", "dP", "db_f", "db_r", "dc0"):
        assert torch.equal(lb[k], ref[k]), k


@pytest.mark.parametrize("linear", [False, True])
def test_scans_stay_inside(linear):
    """The scan entry points: the linear recurrence's segment maps and the
    per-sequence v/b partials live in their workspaces."""
    L, B, d = 300, 3, 64   # few lane groups: the linear scans cut time into segments
    print(f"workspace guard scans L={L} B={B} d={d} linear={linear}", flush=True)
    c = random_layer_case(np.random.default_rng(7), L, B, d, d, O.DIR_BI, masked=True,
                          c0=True, dc_last=True, bias_scale=0.5)
    X, W = dev(c["X"]), dev(c["W"])
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    kw = dict(c0=dev(c["c0"]), direction=O.DIR_BI, mask=dev(c["mask"]), linear=linear)
    fw = sru.forward(X, W, *p, **kw)
    lib = sru.lib()
    nf = lib.sru_scan_forward_workspace_bytes(L, B, d, d, O.DIR_BI)
    nb = lib.sru_scan_backward_workspace_bytes(L, B, d, d, O.DIR_BI)
    fbuf = torch.full((nf + GUARD,), FILL, dtype=torch.uint8, device="cuda")
    bbuf = torch.full((nb + GUARD,), FILL, dtype=torch.uint8, device="cuda")
    sf = sru.scan_forward(fw["U"], X, *p, ws=fbuf[:nf], **kw)
    sb = sru.scan_backward(fw["U"], X, fw["C"], dev(c["dH"]), *p, dc_last=dev(c["dc_last"]),
                           ws=bbuf[:nb], **kw)
    torch.cuda.synchronize()
    assert nf > 0 and nb > 0
    assert bool(torch.all(fbuf[nf:] == FILL)), "the forward scan wrote past its workspace"
    assert bool(torch.all(bbuf[nb:] == FILL)), "the backward scan wrote past its workspace"
    assert torch.equal(sf["H"], fw["H"]) and torch.equal(sf["c_last"], fw["c_last"])


def _guarded_out(shape, dtype=torch.float32):
    """An output tensor of `shape` at the start of a buffer whose tail is a guard."""
    n = int(np.prod(shape))
    esz = torch.tensor([], dtype=dtype).element_size()
    buf = torch.full(((n * esz + GUARD_OUT + 15) // 16 * 16,), FILL, dtype=torch.uint8,
                     device="cuda")
    return buf, buf[:n * esz].view(dtype).view(shape), n * esz


GUARD_OUT = 1 << 16


@pytest.mark.parametrize("case", [
    (37, 5, 130, 65, O.DIR_FWD, O.GEMM_FP32),
    (20, 3, 63, 63, O.DIR_BI, O.GEMM_FP32),
    (33, 9, 264, 264, O.DIR_REV, O.GEMM_BF16),
    (40, 13, 256, 256, O.DIR_BI, O.GEMM_BF16),
    (17, 6, 200, 72, O.DIR_BI, O.GEMM_BF16),
])
def test_outputs_written_within_bounds(case):
    """Ragged shapes (partial tiles, partial lane groups): every output is
    the head of a larger buffer, and nothing past it changes."""
    L, B, d_in, d, direction, gemm = case
    print(f"output guard L={L} B={B} d_in={d_in} d={d} dir={direction} gemm={gemm}", flush=True)
    c = random_layer_case(np.random.default_rng(3 * L + d), L, B, d_in, d, direction,
                          masked=True, c0=True, dc_last=True, bias_scale=0.5)
    X, W = dev(c["X"]), dev(c["W"])
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    ndir, k = W.shape[0], W.shape[1]
    nf = ndir * d
    guards = []

    def out(name, shape, dtype=torch.float32):
        buf, t, nbytes = _guarded_out(shape, dtype)
        guards.append((name, buf, nbytes))
        return t
    bf = gemm == O.GEMM_BF16
    fo = dict(U=out("U", (L, B, ndir, k, d)), H=out("H", (L, B, nf)), C=out("C", (L, B, nf)),
              c_last=out("c_last", (B, nf)))
    if bf:
        fo["W_bf16"] = out("W_bf16", tuple(W.shape), torch.bfloat16)
        fo["H_bf16"] = out("H_bf16", (L, B, nf), torch.bfloat16)
    kw = dict(c0=dev(c["c0"]), direction=direction, mask=dev(c["mask"]), gemm_dtype=gemm)
    fw = sru.forward(X, W, *p, out=fo, **kw)
    bo = dict(dX=out("dX", (L, B, d_in)), dW=out("dW", tuple(W.shape)), dv_f=out("dv_f", (ndir, d)),
              dv_r=out("dv_r", (ndir, d)), db_f=out("db_f", (ndir, d)), db_r=out("db_r", (ndir, d)),
              dc0=out("dc0", (B, nf)))
    sru.backward(X, W, *p, fw["U"], fw["C"], dev(c["dH"]), dc_last=dev(c["dc_last"]), out=bo,
                 W_bf16=fo.get("W_bf16"), **kw)
    torch.cuda.synchronize()
    for name, buf, nbytes in guards:
        assert bool(torch.all(buf[nbytes:] == FILL)), f"{name} written past its end"
