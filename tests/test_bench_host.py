"""Host logic of bench.py (no GPU): the algorithmic work it prices each
kernel's roofline with, the dW split count it reads back from the library's
workspace plan, and the one-GPU contract of its command line."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_1709_02755_amd import sru  # noqa: E402
from paper_1709_02755_amd.workloads import WORKLOADS  # noqa: E402


def _w(name):
    return next(w for w in WORKLOADS if w.name == name)


def test_headline_work_figures():
    """The 6-layer stack at L 256, B 64, d 1024 with bf16 products: each
    product 2 M N K flops (M = 16,384 tokens, N = 3 d, K = d); the forward
    scan 24 B per (t, b, j) plus the bf16 copy of h on 5 of the 6 layers; the
    backward scan 24 B read, dU written in bf16 (3 blocks) and the fp32
    highway gradient (34 B); the split-K sum reads S partials and writes
    the result, and also sums the v/b partials over the batch."""
    w = _w("sru6_L256_B64_d1024_bf16")
    elems = 256 * 64 * 1024
    work = bench.kernel_work(w, 5, True)
    for key in ("gemm_u", "gemm_dx", "gemm_dw"):
        assert work[key]["flops"] == 2.0 * 16384 * 3072 * 1024
    assert work["scan_fwd"]["bytes"] == pytest.approx(elems * (24 + 2 * 5 / 6), rel=1e-15)
    assert work["scan_bwd"]["bytes"] == elems * 34
    # with the v/b sums (4 per feature) of the 64 sequences folded in
    assert work["splitk_reduce"]["bytes"] == 4.0 * 6 * 3072 * 1024 + 4.0 * 4 * 65 * 1024
    assert work["bf16_x"]["bytes"] == 6.0 * 16384 * 1024


def test_fp32_backward_scan_bytes_and_k4():
    """fp32 products keep dU in fp32 (40 B at k = 3); a layer whose input
    width differs from d has k = 4 and no separate highway gradient."""
    w = _w("bisru3_L400_B32_d128_fp32_masked")
    per0 = bench._layer_work(w, 0, 1, False)   # d_in 128 = d: k = 3
    per1 = bench._layer_work(w, 1, 1, False)   # d_in 256 (both directions): k = 4
    elems = 400 * 32 * 2 * 128
    assert per0["scan_bwd"]["bytes"] == elems * 40
    assert per1["scan_bwd"]["bytes"] == elems * (24 + 4 * 4)
    assert per1["gemm_u"]["flops"] == 2.0 * 12800 * (2 * 4 * 128) * 256


def test_dw_split_count_read_from_the_workspace_plan():
    """The headline dW (N 3072, d_in 1024, 16,384 tokens: 48 tiles of
    256 x 256) runs in 5 K splits, 240 workgroups on the 256 CUs."""
    assert bench.dw_splits(sru.lib(), _w("sru6_L256_B64_d1024_bf16")) == 5


@pytest.mark.parametrize("L,B,d", [(1024, 384, 1024), (4096, 1024, 2048), (16384, 256, 1024),
                                   (65536, 64, 512)])
def test_dw_split_panels_fit_buffer_offsets(L, B, d):
    """The direct products address a split's panel of a row-contiguous
    operand (dU [M, N] and X [M, d_in] in bf16, k-rows = tokens) with 32-bit
    offsets from the split's first k-row.  The plan keeps every split's
    panel below 2^31 bytes, raising the split count where the cost model
    alone would not (4M tokens at d = 2048: 12.9 GB per split at its
    preferred 4 splits)."""
    w = bench_workload = type(_w("sru6_L256_B64_d1024_bf16"))(
        f"big_L{L}_B{B}_d{d}", 1, 0, L, B, d, d, 1, True, None, True, 0)
    s = bench.dw_splits(sru.lib(), bench_workload)
    M, N = L * B, 3 * d
    kt = -(-M // 64)
    kps = -(-kt // s) * 64
    for rows in (N, w.d_in):  # dU's and X's row lengths (elements)
        assert (kps - 1) * rows * 2 + rows * 2 < 2 ** 31, (s, kps, rows)
    if M * N * 2 >= 2 ** 31:
        assert s > 1


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
