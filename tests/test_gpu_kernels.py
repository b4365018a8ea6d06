"""GPU parity of the individual kernels through the C ABI's component entry
points: the MFMA products against numpy's matmul of the same (bf16-rounded)
operands, and the two scans against the oracle fed the same U / C."""

import numpy as np
import pytest
import torch

from helpers import TOL_FP32, check, dev, host
from oracle import sru_oracle as O
from paper_1709_02755_amd import sru
from paper_1709_02755_amd.workloads import random_layer_case

pytestmark = pytest.mark.gpu


def _bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16).double().numpy()


# (1500, 520, 200): six tile rows of 256, i.e. one whole group of four tile
# rows and a partial one in the workgroup -> tile order.  NT in bf16 runs
# (2048, 768, 256) and (700, 480, 72) on 256 x 96 tiles (more of them than
# 256 x 128 tiles give), the latter with a partial tile row and a partial
# K step.
GEMM_SHAPES = [(1, 1, 1), (7, 5, 3), (63, 65, 130), (130, 63, 65), (256, 256, 32),
               (257, 513, 96), (384, 128, 128), (1000, 300, 260), (2048, 768, 256),
               (1500, 520, 200), (700, 480, 72)]


@pytest.mark.parametrize("op", [sru.OP_NT, sru.OP_NN, sru.OP_TN])
@pytest.mark.parametrize("dtype", [sru.GEMM_FP32, sru.GEMM_BF16])
@pytest.mark.parametrize("shape", GEMM_SHAPES)
def test_gemm_matches_matmul(op, dtype, shape):
    M, N, K = shape
    print(f"gemm op={op} dtype={dtype} M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M * 7 + N * 3 + K)
    a_shape = (K, M) if op == sru.OP_TN else (M, K)
    b_shape = (N, K) if op == sru.OP_NT else (K, N)
    A = rng.standard_normal(a_shape).astype(np.float32)
    B = rng.standard_normal(b_shape).astype(np.float32)
    Ar, Br = (_bf16(A), _bf16(B)) if dtype == sru.GEMM_BF16 else (A.astype(np.float64), B.astype(np.float64))
    Am = Ar.T if op == sru.OP_TN else Ar
    Bm = Br.T if op == sru.OP_NT else Br
    ref = Am @ Bm
    C = sru.gemm(op, dev(A), dev(B), M, N, K, dtype)
    torch.cuda.synchronize()
    # products of bf16 values are exact in fp32: only accumulation order differs
    check("C", C, ref, TOL_FP32)


def test_gemm_n96_tiles_at_the_shard_shape():
    """U = X W^T of one GPU's share of the 6-layer d = 1024 batch (2,048
    tokens): 256 tiles of 256 x 96, every workgroup a full tile."""
    M, N, K = 2048, 3072, 1024
    print(f"gemm NT bf16 M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(96)
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = rng.standard_normal((N, K)).astype(np.float32)
    C = sru.gemm(sru.OP_NT, dev(A), dev(B), M, N, K, sru.GEMM_BF16)
    torch.cuda.synchronize()
    check("C", C, _bf16(A) @ _bf16(B).T, TOL_FP32)


@pytest.mark.parametrize("dtype", [sru.GEMM_FP32, sru.GEMM_BF16])
@pytest.mark.parametrize("shape", [(384, 256, 12800), (130, 63, 4100), (257, 100, 3000),
                                   (1500, 100, 3000)])
def test_gemm_long_reduction_split(dtype, shape):
    """dW-shaped product with K = tokens (split over K, fixed-order sum).
    N = 63 sums the splits element by element, N = 100 and 256 in groups of
    four; M = 130, 257 and 1500 leave ragged edge tiles (1500: six tile rows,
    a partial group of tile rows)."""
    M, N, K = shape
    print(f"gemm TN long K dtype={dtype} M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(5)
    A = rng.standard_normal((K, M)).astype(np.float32)
    B = rng.standard_normal((K, N)).astype(np.float32)
    Ar, Br = (_bf16(A), _bf16(B)) if dtype == sru.GEMM_BF16 else (A.astype(np.float64), B.astype(np.float64))
    assert sru.lib().sru_gemm_workspace_bytes(sru.OP_TN, M, N, K, dtype) > 0
    C = sru.gemm(sru.OP_TN, dev(A), dev(B), M, N, K, dtype)
    torch.cuda.synchronize()
    check("C", C, Ar.T @ Br, TOL_FP32)


def _case(seed, L, B, d_in, d, direction, **kw):
    return random_layer_case(np.random.default_rng(seed), L, B, d_in, d, direction, **kw)


SCAN_CASES = [
    # (L, B, d_in, d, direction, masked)
    (1, 1, 1, 1, O.DIR_FWD, False),
    (5, 3, 7, 7, O.DIR_REV, False),
    (17, 2, 65, 65, O.DIR_FWD, True),
    (9, 3, 130, 63, O.DIR_BI, True),
    (33, 4, 128, 128, O.DIR_BI, False),
    (40, 5, 64, 64, O.DIR_FWD, True),
    (23, 2, 96, 48, O.DIR_REV, True),
    # exactly one and two rings of 6 steps (the forward's first ring runs
    # ahead of its loop; no tail)
    (6, 3, 64, 64, O.DIR_FWD, False),
    (12, 2, 128, 64, O.DIR_BI, True),
    # 8,192 lanes: the backward runs time-parallel (chunks of 8 steps per
    # wave, 8 or 16 waves per block): one partial block; two blocks, the
    # second partial; k = 4 in both directions
    (37, 8, 1024, 1024, O.DIR_FWD, True),
    (150, 16, 512, 512, O.DIR_REV, True),
    (21, 4, 512, 1024, O.DIR_BI, False),
    (19, 65, 127, 127, O.DIR_REV, True),  # 8,255 lanes: a partial last lane group
    # a wave on every SIMD (B*ndir*d >= 65536): the backward's shorter ring,
    # with a ragged tail (L % 4 != 0), k = 3 and 4
    (7, 64, 1024, 1024, O.DIR_FWD, True),
    (13, 32, 512, 1024, O.DIR_BI, True),
]


@pytest.mark.parametrize("case", SCAN_CASES)
def test_scan_forward_on_oracle_projection(case):
    L, B, d_in, d, direction, masked = case
    print(f"scan_fwd L={L} B={B} d_in={d_in} d={d} dir={direction} mask={masked}", flush=True)
    c = _case(L * 31 + d, L, B, d_in, d, direction, masked=masked, c0=True, bias_scale=0.5)
    ref = O.forward(c["X"], c["W"], c["v_f"], c["v_r"], c["b_f"], c["b_r"], c["c0"], direction,
                    c["mask"])
    U = ref["U"].astype(np.float32)
    out = sru.scan_forward(dev(U), dev(c["X"]), dev(c["v_f"]), dev(c["v_r"]), dev(c["b_f"]),
                           dev(c["b_r"]), dev(c["c0"]), direction, dev(c["mask"]))
    torch.cuda.synchronize()
    for k in ("H", "C", "c_last"):
        check(k, out[k], ref[k], TOL_FP32)


# Forward scan without a mask at ragged sizes (L below, at and above the
# prefetch ring, a partial last wave, k = 3 and 4, every direction), with
# and without C, writing the bf16 copy of H as well.
LDS_SCAN_CASES = [
    # (L, B, d_in, d, direction)
    (1, 1, 4, 4, O.DIR_FWD),
    (5, 3, 20, 20, O.DIR_REV),
    (27, 3, 40, 20, O.DIR_BI),
    (29, 2, 96, 96, O.DIR_FWD),
    (61, 5, 64, 64, O.DIR_BI),
    (100, 4, 96, 64, O.DIR_REV),
    (130, 3, 128, 128, O.DIR_FWD),
    # 256-unit workgroups streaming through the LDS ring (65,536 lanes):
    # a partial last group of steps, k = 3 reverse, k = 4 bidirectional
    (9, 64, 1024, 1024, O.DIR_REV),
    (6, 32, 512, 1024, O.DIR_BI),
]


@pytest.mark.parametrize("store_c", [True, False])
@pytest.mark.parametrize("case", LDS_SCAN_CASES)
def test_scan_forward_outputs_unmasked(case, store_c):
    L, B, d_in, d, direction = case
    print(f"scan_fwd outputs L={L} B={B} d_in={d_in} d={d} dir={direction} C={store_c}",
          flush=True)
    c = _case(L * 17 + d, L, B, d_in, d, direction, c0=True, bias_scale=0.5)
    ref = O.forward(c["X"], c["W"], c["v_f"], c["v_r"], c["b_f"], c["b_r"], c["c0"], direction,
                    None)
    U = ref["U"].astype(np.float32)
    ndir = 2 if direction == O.DIR_BI else 1
    out = dict(H=torch.full((L, B, ndir * d), float("nan"), device="cuda"),
               C=torch.full((L, B, ndir * d), float("nan"), device="cuda") if store_c else None,
               c_last=torch.full((B, ndir * d), float("nan"), device="cuda"),
               H_bf16=torch.zeros((L, B, ndir * d), dtype=torch.bfloat16, device="cuda"))
    out = sru.scan_forward(dev(U), dev(c["X"]), dev(c["v_f"]), dev(c["v_r"]), dev(c["b_f"]),
                           dev(c["b_r"]), dev(c["c0"]), direction, None, out=out)
    torch.cuda.synchronize()
    keys = ("H", "C", "c_last") if store_c else ("H", "c_last")
    for k in keys:
        check(k, out[k], ref[k], TOL_FP32)
    assert torch.equal(out["H_bf16"].view(torch.int16), out["H"].to(torch.bfloat16).view(torch.int16))
    # the same without the bf16 copy
    out2 = sru.scan_forward(dev(U), dev(c["X"]), dev(c["v_f"]), dev(c["v_r"]), dev(c["b_f"]),
                            dev(c["b_r"]), dev(c["c0"]), direction, None, store_c=store_c)
    torch.cuda.synchronize()
    for k in keys:
        assert torch.equal(out2[k], out[k]), k


@pytest.mark.parametrize("case", SCAN_CASES)
def test_scan_backward_on_oracle_states(case):
    L, B, d_in, d, direction, masked = case
    print(f"scan_bwd L={L} B={B} d_in={d_in} d={d} dir={direction} mask={masked}", flush=True)
    c = _case(L * 17 + d, L, B, d_in, d, direction, masked=masked, c0=True, dc_last=True,
              bias_scale=0.5)
    args = (c["X"], c["W"], c["v_f"], c["v_r"], c["b_f"], c["b_r"])
    fw = O.forward(*args, c["c0"], direction, c["mask"])
    bw = O.backward(*args, c["dH"], c["c0"], direction, c["mask"], O.GEMM_FP32, c["dc_last"])
    # the scan sees exactly the fp32 U and C the forward would hand it
    out = sru.scan_backward(dev(fw["U"].astype(np.float32)), dev(c["X"]),
                            dev(fw["C"].astype(np.float32)), dev(c["dH"]), dev(c["v_f"]),
                            dev(c["v_r"]), dev(c["b_f"]), dev(c["b_r"]), dev(c["c0"]),
                            dev(c["dc_last"]), direction, dev(c["mask"]), d_in=d_in)
    torch.cuda.synchronize()
    check("dU", out["dU"], bw["dU"], TOL_FP32)
    if d_in == d:
        check("dxh", out["dxh"], bw["dxh"], TOL_FP32)
    for k in ("dv_f", "dv_r", "db_f", "db_r", "dc0"):
        check(k, out[k], bw[k], TOL_FP32)


@pytest.mark.parametrize("L,B,d", [(20, 8, 1024), (9, 64, 1024)])
def test_scan_forward_on_unaligned_inputs(L, B, d):
    """U and x need only 4-byte alignment.  The LDS-ring scans (8,192 lanes:
    the narrow ring; 65,536: the wide one) load 16 bytes per lane, so inputs
    that start 4 bytes past a 16-byte boundary take the register-ring scan;
    the results are the same bits."""
    print(f"scan_fwd unaligned L={L} B={B} d={d}", flush=True)
    c = _case(L + B + d, L, B, d, d, O.DIR_FWD, masked=True, c0=True, bias_scale=0.5)
    U = torch.randn(L, B, 1, 3, d, device="cuda")
    X = dev(c["X"])
    p = [dev(c[k]) for k in ("v_f", "v_r", "b_f", "b_r")]
    def shifted(t):
        buf = torch.empty(t.numel() + 1, device="cuda")
        v = buf[1:].view(t.shape)
        v.copy_(t)
        return v
    Us, Xs = shifted(U), shifted(X)
    assert Us.data_ptr() % 16 == 4 and Xs.data_ptr() % 16 == 4
    a = sru.scan_forward(U, X, *p, dev(c["c0"]), O.DIR_FWD, dev(c["mask"]))
    b = sru.scan_forward(Us, Xs, *p, dev(c["c0"]), O.DIR_FWD, dev(c["mask"]))
    torch.cuda.synchronize()
    for k in ("H", "C", "c_last"):
        assert torch.equal(a[k], b[k]), k


def test_scan_saturation_exact_and_finite():
    """b_f = +100 keeps c = c0 exactly; b_f = -100 gives c = u0 exactly;
    b_r = +100 gives h = c exactly; no NaN anywhere (sigma saturates)."""
    L, B, d = 12, 3, 70
    c = _case(1, L, B, d, d, O.DIR_FWD, c0=True)
    U = np.random.default_rng(2).standard_normal((L, B, 1, 3, d)).astype(np.float32) * 3
    big = np.full((1, d), 100.0, np.float32)
    zero = np.zeros((1, d), np.float32)
    o = sru.scan_forward(dev(U), dev(c["X"]), dev(c["v_f"]), dev(c["v_r"]), dev(big), dev(zero),
                         dev(c["c0"]), O.DIR_FWD)
    C = host(o["C"])
    assert np.array_equal(C, np.broadcast_to(c["c0"].astype(np.float64), C.shape))
    o = sru.scan_forward(dev(U), dev(c["X"]), dev(c["v_f"]), dev(c["v_r"]), dev(-big), dev(big),
                         dev(c["c0"]), O.DIR_FWD)
    C, H = host(o["C"]), host(o["H"])
    assert np.array_equal(C, U[:, :, 0, 0].astype(np.float64))
    assert np.array_equal(H, C)
    assert np.all(np.isfinite(H))
