#!/usr/bin/env python3
"""Throughput of the SRU layer stack (forward + backward) on one MI355X.

Workload: 6 stacked unidirectional SRU layers, L = 256 steps, B = 64
sequences, d_in = d = 1024, bf16-input / fp32-accumulate matrix products,
fp32 scans, synthetic inputs (seeded; the paper's datasets are not used).
One step = forward through all 6 layers, then backward through all 6
(including dX of the first layer).  Metric: tokens/s = L*B / step time.

Besides the headline number the JSON line carries
  * roofline: the kernel that takes the most time per step, its algorithmic
    bytes or flops per launch over its average duration (HIP events recorded
    by the library around every launch, on the launch stream), against the
    MI355X peak;
  * scan_hbm: the same for both scan kernels (the metric's second half);
  * cpu_baseline: the fp64 CPU oracle timed on a bounded sample of the same
    workload on this host.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""

from __future__ import annotations

import argparse
import ctypes
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "fp32": 157.3}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# ------------------------------------------------------------------ HIP events
class HipEvents:
    """A pool of HIP events created through the HIP runtime torch has loaded."""

    def __init__(self, n):
        path = None
        for line in open("/proc/self/maps"):
            if "libamdhip64" in line:
                path = line.split()[-1]
                break
        if path is None:
            raise RuntimeError("HIP runtime not loaded")
        h = ctypes.CDLL(path)
        h.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                          ctypes.c_void_p]
        h.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.h = h
        self.events = (ctypes.c_void_p * n)()
        for i in range(n):
            ev = ctypes.c_void_p()
            if h.hipEventCreate(ctypes.byref(ev)) != 0:
                raise RuntimeError("hipEventCreate failed")
            self.events[i] = ev
        self.n = n

    def elapsed_ms(self, i, j):
        ms = ctypes.c_float()
        rc = self.h.hipEventElapsedTime(ctypes.byref(ms), self.events[i], self.events[j])
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return ms.value

    def close(self):
        for i in range(self.n):
            self.h.hipEventDestroy(self.events[i])


# ------------------------------------------------------------------ work model
class GpuLead:
    """Idle GPU time queued ahead of a bracketed launch sequence.

    The per-launch hook records an event right before each kernel.  When the
    GPU waits on the host (a short step, or the first call after a
    synchronisation), the event completes at once and the kernel arrives
    microseconds later, so that gap would be timed as the kernel's.  A spin
    kernel of torch's (torch.cuda._sleep: it waits a set number of clock
    cycles and touches no memory, so the caches stay as they were) placed in
    front of the sequence lets the host queue every launch and event before
    the GPU reaches them."""

    def __init__(self):
        import torch
        self.torch = torch
        torch.cuda._sleep(1000)
        e0, e1 = (torch.cuda.Event(enable_timing=True) for _ in range(2))
        n = 2_000_000
        e0.record()
        torch.cuda._sleep(n)
        e1.record()
        torch.cuda.synchronize()
        self.cycles_per_ms = n / max(e0.elapsed_time(e1), 1e-3)

    def __call__(self, ms):
        self.torch.cuda._sleep(int(self.cycles_per_ms * ms))


def host_ms(fn):
    """Host time of fn's launches (they are asynchronous), in ms; the GPU
    work is waited for afterwards."""
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    fn()
    ms = (time.perf_counter() - t0) * 1e3
    torch.cuda.synchronize()
    return ms


def kernel_work(w, splits, bf16):
    """Algorithmic bytes / flops per launch of each kernel at workload w,
    averaged over the stack's layers (a layer above a bidirectional one
    takes 2d inputs); the input rounding runs once per step, on the first
    layer's input.  Bytes count each element read or written once: fp32
    4 B, bf16 2 B."""
    per = [_layer_work(w, li, splits, bf16) for li in range(w.layers)]
    out = {}
    for key in per[0]:
        vals = [p[key] for p in per]
        out[key] = {m: sum(v[m] for v in vals) / len(vals) for m in vals[0]}
    out["bf16_x"] = per[0]["bf16_x"]
    return out


def _layer_work(w, li, splits, bf16):
    """Algorithmic bytes / flops per launch of each kernel for layer li."""
    M = w.L * w.B
    nfeat = w.ndir * w.d
    K, k = w.layer_dims(li)
    N = w.ndir * k * w.d
    elems = M * nfeat
    du_b = 2.0 if bf16 else 4.0
    nq = 2 if w.linear else 4  # v/b sums per feature (no v in the linear variant)
    hb = 2.0 * (w.layers - 1) / w.layers if bf16 else 0.0  # bf16 copy of H (not the top's)
    vb_bytes = 4.0 * (nq * w.B * nfeat + nq * nfeat)  # per-sequence partials in, sums out
    if w.dp is not None:  # low-rank layers: Wcat = P Q^T, rank dp
        dp = w.dp
        low = {
            "gemm_t": dict(flops=2.0 * M * dp * K),    # T = X Q
            "gemm_u": dict(flops=2.0 * M * N * dp),    # U = T P^T
            "gemm_dt": dict(flops=2.0 * M * dp * N),   # dT = dU P
            "gemm_dx": dict(flops=2.0 * M * K * dp),   # dX = dT Q^T
            "gemm_dp": dict(flops=2.0 * N * dp * M),   # dP = dU^T T
            "gemm_dq": dict(flops=2.0 * K * dp * M),   # dQ = X^T dT
            "bf16_x": dict(bytes=(4.0 + 2.0) * M * K),
            "bf16_q": dict(bytes=(4.0 + 2.0) * K * dp),   # Q, or Q^T
            "bf16_p": dict(bytes=(4.0 + 2.0) * N * dp),   # P, or P^T
            "splitk_reduce": dict(),  # two reductions of different sizes: time only
        }
    else:
        low = {}
    return {
        "gemm_u": dict(flops=2.0 * M * N * K),     # U = X W^T
        # inference with the projection and the scan fused: the product's flops
        "proj_scan_fwd": dict(flops=2.0 * M * N * K),
        "gemm_dx": dict(flops=2.0 * M * K * N),    # dX = dU W
        "gemm_dw": dict(flops=2.0 * N * K * M),    # dW = dU^T X
        # read U's three blocks and x_hat (x, or U block 3), write h and c
        # (24 B per (t, b, j); 20 B without c); with bf16 products below the
        # top layer also the bf16 copy of h (the next layer's operand)
        "scan_fwd": dict(bytes=elems * (16.0 + 4.0 + (4.0 if w.store_c or w.backward else 0.0)
                                        + hb)),
        # read U's blocks, x_hat, c, dh (24 B); write dU (k blocks, bf16 when
        # the products are bf16) and, for k = 3, dx_hat (4 B): 34 B (bf16) /
        # 40 B (fp32) at k = 3
        "scan_bwd": dict(bytes=elems * (24.0 + du_b * k + (4.0 if k == 3 else 0.0))),
        "reduce_vb": dict(bytes=vb_bytes),
        # the dense backward runs the v/b sums as extra workgroups of the dW
        # product's split-K sum when it has one (else as reduce_vb)
        "splitk_reduce": dict(bytes=4.0 * (splits + 1) * N * K
                              + (vb_bytes if w.dp is None and splits > 1 else 0.0)),
        # fp32 -> bf16 copies of the product operands: Wcat, X (first layer);
        # Wcat^T for dX, transposed from the forward's bf16 Wcat (the stack
        # hands it over: 2 B read, 2 B written per element)
        "bf16_w": dict(bytes=(4.0 + 2.0) * N * K),
        "bf16_x": dict(bytes=(4.0 + 2.0) * M * K),
        "bf16_wt": dict(bytes=(2.0 + 2.0) * N * K),
        **low,
    }


def dw_splits(lib, w):
    """Split count of the dW product as sru_backward plans it.  The backward
    workspace ends with the split partials (fp32 [splits, N, d_in]); the
    buffers before them are laid out as the library does (each 256-aligned:
    dU, dx_hat for k = 3, v/b partials, bf16 Wcat and X in bf16 mode)."""
    a = lambda x: (x + 255) // 256 * 256
    bf16 = w.gemm_dtype == 1
    M, nfeat = w.tokens, w.ndir * w.d
    k = 3 if w.d_in == w.d else 4
    N = w.ndir * k * w.d
    total = lib.sru_backward_workspace_bytes(w.L, w.B, w.d_in, w.d, w.direction, w.gemm_dtype)
    before = a((2 if bf16 else 4) * M * N) + (a(4 * M * nfeat) if k == 3 else 0)
    before += a(16 * w.B * nfeat)
    if bf16:
        before += a(2 * N * w.d_in) + a(2 * M * w.d_in)
    return max(1, (total - before) // (4 * N * w.d_in))


def source_hash():
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(ROOT, "paper_1709_02755_amd", "csrc", "*"))):
        h.update(open(p, "rb").read())
    return h.hexdigest()[:16]


def pmc_traffic(label, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    it was taken on the current kernel sources and this workload; else None."""
    p = os.path.join(ROOT, "profiles", "pmc_traffic.json")
    if not os.path.exists(p):
        return None
    d = json.load(open(p))
    if d.get("source_hash") != source_hash() or d.get("workload") != workload:
        return None
    k = d.get("kernels", {}).get(label)
    return None if k is None else k.get("hbm_bytes_per_launch")


FLUSH_MODES = ("none", "write", "read", "write+read")


def cold_scans(w, st, X, dH, mask, reps, highway_scale, reset_new, mode="write+read"):
    """The two scans of layer 0, timed cold: right before every call a
    512 MiB buffer is overwritten, so none of the scan's input is left in
    L2 or the 256 MB last-level cache, and then a second 512 MiB buffer is
    read, so the caches hold only clean lines when the scan starts.  (The
    overwrite alone leaves up to 288 MB of dirty lines in those caches,
    whose write-back to HBM would then be charged to the scan: 14-25 us per
    scan at L 256, B 64, d 1024.)  The scan kernels are the ones the step runs:
    the forward is the plain scan call with the step's outputs (H, C and, with
    bf16 products, the bf16 copy of H); the backward is the whole layer-0
    backward call, whose first kernel is the gradient scan (bf16 dU with bf16
    products).  Each time is the scan kernel's own, from the per-launch event
    hook, over its algorithmic bytes: forward, U's k blocks, x (k = 3), h, c
    (and bf16 h); backward, U's k blocks, x (k = 3), c, dh, dU's k blocks
    (fp32 or bf16) and dx_hat (k = 3).  The linear recurrence's maps kernel,
    when it runs, is timed with its scan."""
    import torch

    from paper_1709_02755_amd import sru
    f0 = st.fw[0]
    if f0["U"] is None or f0["C"] is None:
        return None
    U, C = f0["U"], f0["C"]
    L, B, ndir, k, d = U.shape
    p = st.layers[0]
    bf16 = w.gemm_dtype == sru.GEMM_BF16
    v = dict(highway_scale=highway_scale, reset_new=reset_new, linear=w.linear)
    par = (p["v_f"], p["v_r"], p["b_f"], p["b_r"])
    elems = L * B * ndir * d
    xb = 4.0 if k == 3 else 0.0
    fbytes = elems * (4.0 * k + xb + 8.0 + (2.0 if bf16 else 0.0))
    bbytes = elems * (4.0 * k + xb + 8.0 + (2.0 if bf16 else 4.0) * k + xb)
    fout = dict(H=torch.empty_like(f0["H"]), C=torch.empty_like(C),
                c_last=torch.empty_like(f0["c_last"]))
    if bf16:
        fout["H_bf16"] = torch.empty(f0["H"].shape, dtype=torch.bfloat16, device=U.device)
    fws = sru.workspace(sru.lib().sru_scan_forward_workspace_bytes(L, B, X.shape[2], d,
                                                                   w.direction), U.device)
    calls = {"scan_fwd": (fbytes, ("scan_fwd", "scan_maps"), lambda: sru.scan_forward(
        U, X, *par, direction=w.direction, mask=mask, out=fout, ws=fws, **v))}
    if w.backward:
        # the layer-0 call of the step's backward (dH has layer 0's output shape)
        if "Q" in p:
            bcall = lambda: sru.backward_lowrank(
                X, p["Q"], p["P"], *par, f0["T"], U, C, dH, None, None, w.direction, mask,
                w.gemm_dtype, want_dc0=False, out=st.bw[0], ws=st.ws, X_bf16=st.xb0,
                T_bf16=f0.get("T_bf16"), **v)
        else:
            bcall = lambda: sru.backward(
                X, p["W"], *par, U, C, dH, None, None, w.direction, mask, w.gemm_dtype,
                want_dc0=False, out=st.bw[0], ws=st.ws, X_bf16=st.xb0,
                W_bf16=f0.get("W_bf16"), **v)
        calls["scan_bwd"] = (bbytes, ("scan_bwd", "scan_maps"), bcall)
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=U.device)
    clean = torch.ones((512 << 20) // 4, dtype=torch.float32, device=U.device)
    sink = torch.empty((), dtype=torch.float32, device=U.device)
    lib = sru.lib()
    ev = HipEvents(2 * 64 + 2)
    lead = GpuLead()
    res = {}
    try:
        for name, (nbytes, labels, call) in calls.items():
            lead_ms = 3.0 * host_ms(call) + 0.2  # also warms the launch path
            times = []
            for i in range(reps):
                if "write" in mode:
                    flush.fill_(i & 0xFF)              # evict the scan's data
                if "read" in mode:
                    torch.sum(clean, dim=0, out=sink)  # write back the dirty lines
                torch.cuda.synchronize()
                lead(lead_ms)  # the call's launches queue before the GPU reaches them
                lib.sru_timing_begin(ev.events, ev.n)
                try:
                    call()
                finally:
                    nk = lib.sru_timing_end()
                torch.cuda.synchronize()
                times.append(sum(ev.elapsed_ms(2 * j, 2 * j + 1) for j in range(nk)
                                 if lib.sru_timing_label(j).decode() in labels) * 1e-3)
            t = sorted(times)[len(times) // 2]
            gbps = nbytes / t / 1e9
            res[name] = {"avg_us": round(t * 1e6, 2), "GBps": round(gbps, 1),
                         "frac": round(gbps / HBM_PEAK_GBPS, 4),
                         "bytes_per_elem": nbytes / elems, "reps": reps, "stat": "median",
                         "flush": {"none": "none", "write": "512 MiB written",
                                   "read": "512 MiB read",
                                   "write+read": "512 MiB written, then 512 MiB read"}[mode]}
    finally:
        ev.close()
    del flush, clean
    return res


def yardstick(w, st, X, dH, mask, eager_step, reps=20):
    """The vendor library (torch.mm, i.e. hipBLASLt, bf16 operands, run
    only) on the first layer's three product shapes, with fp32 and with bf16
    output, beside this library's own product kernels in the step (the
    per-launch event hook): medians of `reps` launches, microseconds."""
    import torch

    from paper_1709_02755_amd import sru
    M = w.tokens
    K, k = w.layer_dims(0)
    N = w.ndir * k * w.d
    g = torch.Generator(device="cuda").manual_seed(0)
    rnd = lambda *shape: torch.randn(*shape, device="cuda", generator=g).to(torch.bfloat16)
    X16, W16, dU16 = rnd(M, K), rnd(N, K), rnd(M, N)
    # transposed operands are materialised (no transposed views)
    Wt16, dUt16 = W16.t().contiguous(), dU16.t().contiguous()
    shapes = {"gemm_u": (lambda od: torch.mm(X16, Wt16, out_dtype=od)),     # U = X W^T
              "gemm_dx": (lambda od: torch.mm(dU16, W16, out_dtype=od)),    # dX = dU W
              "gemm_dw": (lambda od: torch.mm(dUt16, X16, out_dtype=od))}   # dW = dU^T X

    def median_us(fn):
        fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * reps)]
        for i in range(reps):
            ev[2 * i].record()
            fn()
            ev[2 * i + 1].record()
        torch.cuda.synchronize()
        t = sorted(ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(reps))
        return round(t[reps // 2] * 1e3, 2)

    vendor = {name: {"fp32_out": median_us(lambda: fn(torch.float32)),
                     "bf16_out": median_us(lambda: fn(torch.bfloat16))}
              for name, fn in shapes.items()}
    # this library's kernels: one bracketed step
    ev = HipEvents(2 * w.layers * 32 + 2)
    lib = sru.lib()
    lead_ms = 3.0 * host_ms(eager_step) + 0.5
    GpuLead()(lead_ms)
    lib.sru_timing_begin(ev.events, ev.n)
    try:
        eager_step()
    finally:
        nk = lib.sru_timing_end()
    torch.cuda.synchronize()
    ours = {}
    for i in range(nk):
        lab = lib.sru_timing_label(i).decode()
        if lab in shapes and lab not in ours:  # the first layer's launch
            ours[lab] = round(ev.elapsed_ms(2 * i, 2 * i + 1) * 1e3, 2)
    ev.close()
    flops = 2.0 * M * N * K
    for name in shapes:
        log(f"  {name}: vendor fp32-out {vendor[name]['fp32_out']} us, bf16-out "
            f"{vendor[name]['bf16_out']} us; ours (fp32 out) {ours.get(name)} us")
    return {"workload": w.name, "M": M, "N": N, "K": K, "flops": flops, "vendor_us": vendor,
            "ours_us": ours,
            "note": "vendor: torch.mm on bf16 operands, median of %d; ours: the step's "
                    "kernels, first layer" % reps}


# ------------------------------------------------------------------ CPU oracle
def cpu_baseline(w, inp, nseq):
    """The fp64 oracle (test infrastructure, never the product path) on the
    first `nseq` sequences of the same inputs: the full stack, forward and
    (when the workload has one) backward."""
    from oracle import sru_oracle as O
    affinity = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info
        blas = max((i.get("num_threads", 1) for i in threadpool_info()
                    if i.get("user_api") == "blas"), default=1)
    except Exception:  # threadpoolctl missing: the BLAS pool is not known
        blas = None
    threads = blas if blas is not None else affinity
    nseq = min(nseq, w.B)
    sl = slice(0, nseq)
    X = inp["X"][:, sl]
    mask = None if inp["mask"] is None else inp["mask"][:, sl]
    dH = None if inp["dH"] is None else inp["dH"][:, sl]
    # a sample shorter than a second is repeated until a second has passed
    reps, t0 = 0, time.perf_counter()
    while True:
        O.stack_forward_backward(X, inp["layers"], w.direction, mask, w.gemm_dtype, dH,
                                 need_backward=w.backward, linear=w.linear)
        reps += 1
        secs = time.perf_counter() - t0
        if secs >= 1.0:
            break
    tokens = w.L * nseq * reps
    passes = "fwd+bwd" if w.backward else "fwd"
    return {"value": tokens / secs, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "blas_threads": blas, "affinity_cores": affinity, "seconds": secs,
            "sample": f"{w.layers}-layer {passes} stack on {nseq} of {w.B} sequences, "
                      f"{reps} run(s) ({tokens} tokens), fp64 NumPy, per-step projections"}


# ------------------------------------------------------------------ counters
COPY_BYTES = 1 << 30  # calibration copy: 1 GiB read + 1 GiB written


def copy_calibration(reps):
    """A plain elementwise copy of known size (torch's own kernel), run under
    rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE to scale those counters."""
    import torch
    src = torch.ones(COPY_BYTES // 4, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    log(f"copy calibration: {reps} x {COPY_BYTES} bytes")


def _pmc_rows(path):
    import csv
    rows = []
    for f in glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            rows.extend(csv.DictReader(fh))
    if not rows:
        raise SystemExit(f"no *counter_collection.csv under {path}")
    return rows


def _per_kernel(rows, counter):
    """Average counter value per dispatch, by kernel-name key."""
    acc = {}
    for r in rows:
        if r.get("Counter_Name") != counter:
            continue
        name = r.get("Kernel_Name", "")
        a = acc.setdefault(name, [0.0, 0])
        a[0] += float(r["Counter_Value"])
        a[1] += 1
    return {k: v[0] / v[1] for k, v in acc.items()}


# kernel-name substrings (all must occur) -> labels of the per-launch table
KERNEL_KEYS = [(("scan_fwd_kernel",), "scan_fwd"), (("scan_fwd_ring_kernel",), "scan_fwd"),
               (("scan_bwd_kernel",), "scan_bwd"),
               (("scan_fwd_lin_kernel",), "scan_fwd"), (("scan_bwd_lin_kernel",), "scan_bwd"),
               (("reduce_vb_kernel",), "reduce_vb"), (("splitk_reduce_kernel",), "splitk_reduce"),
               (("splitk_reduce4_kernel",), "splitk_reduce"),
               (("to_bf16_kernel",), "bf16_x"),
               # the three products of the dense bf16 path (template args after
               # the 256 x 256 tile configuration: addend count, A row-contiguous,
               # B row-contiguous, bf16 result)
               (("gemm_direct_kernel", "256, 256, 64", ">, 0, false, false, false>"), "gemm_u"),
               (("gemm_direct_kernel", "256, 256, 64", ">, 1, false, false, false>"), "gemm_dx"),
               (("gemm_direct_kernel", "256, 256, 64", ">, 2, false, false, false>"), "gemm_dx"),
               (("gemm_direct_kernel", "256, 256, 64", ">, 0, true, true, false>"), "gemm_dw")]


def summarize_pmc(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, out, workload):
    """Turn four rocprofv3 --pmc runs (FETCH_SIZE and WRITE_SIZE of the bench
    and of the calibration copy) into per-launch HBM bytes for the scans."""
    def one(d, counter, key):
        vals = _per_kernel(_pmc_rows(d), counter)
        keys = (key,) if isinstance(key, str) else key
        hits = {k: v for k, v in vals.items() if all(s in k for s in keys)}
        if not hits:
            raise SystemExit(f"{key} not in {d}")
        return max(hits.values())

    # FETCH_SIZE / WRITE_SIZE are KiB per dispatch
    scale_f = COPY_BYTES / (1024.0 * one(copy_fetch_dir, "FETCH_SIZE", "elementwise"))
    scale_w = COPY_BYTES / (1024.0 * one(copy_write_dir, "WRITE_SIZE", "elementwise"))
    kernels = {}
    for key, label in KERNEL_KEYS:
        try:
            f = one(fetch_dir, "FETCH_SIZE", key) * 1024.0 * scale_f
            w = one(write_dir, "WRITE_SIZE", key) * 1024.0 * scale_w
        except SystemExit:
            continue
        kernels[label] = {"fetch_bytes_per_launch": f, "write_bytes_per_launch": w,
                          "hbm_bytes_per_launch": f + w}
    res = {"source_hash": source_hash(), "workload": workload, "copy_scale_fetch": scale_f,
           "copy_scale_write": scale_w, "kernels": kernels}
    with open(out, "w") as fh:
        json.dump(res, fh, indent=1)
    print(json.dumps(res, indent=1))


# ------------------------------------------------------------------ main
def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=3, help="index into the workload table")
    ap.add_argument("--profile-steps", type=int, default=5,
                    help="steps run with per-kernel event brackets")
    ap.add_argument("--cpu-seqs", type=int, default=64,
                    help="sequences in the CPU-oracle sample (0 = skip)")
    ap.add_argument("--highway-scale", type=float, default=1.0,
                    help="alpha on the highway term (Sec. 3.2 scaling correction; 1 = none)")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of the step recorded into a HIP graph (no launch cost)")
    ap.add_argument("--reset-new", action="store_true",
                    help="reset gate reads c_t (Algorithm 1's order) instead of c_{t-1}")
    ap.add_argument("--cold-reps", type=int, default=7,
                    help="launches of each scan timed cold (0 = skip; the counter runs skip "
                         "them so that only the step's launches are counted)")
    ap.add_argument("--cold-protocols", action="store_true",
                    help="only time the layer-0 scans under each cache-flush protocol "
                         "(none, write, read, write+read) and print one JSON line")
    ap.add_argument("--yardstick", action="store_true",
                    help="only time the vendor library's bf16 products (torch.mm) on the "
                         "workload's three product shapes beside the step's own kernels")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="REPS",
                    help="only run a 1 GiB copy REPS times (counter calibration)")
    ap.add_argument("--summarize-pmc", nargs=5,
                    metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR", "COPY_WRITE_DIR", "OUT"),
                    help="build the per-launch HBM traffic table from rocprofv3 --pmc runs")
    args = ap.parse_args()
    if args.summarize_pmc:
        from paper_1709_02755_amd.workloads import WORKLOADS
        summarize_pmc(*args.summarize_pmc, WORKLOADS[args.workload].name)
        return
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(--gpus must be 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1709_02755_amd import sru
    from paper_1709_02755_amd.workloads import WORKLOADS, make_inputs

    w = WORKLOADS[args.workload]
    log(f"workload {w.name}: L={w.L} B={w.B} d_in={w.d_in} d={w.d} layers={w.layers}")
    inp = make_inputs(w)
    dev = torch.device("cuda:0")
    to = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    layers = [{k: to(v) for k, v in p.items()} for p in inp["layers"]]
    # inference with bf16 products holds its weights in bf16, rounded once
    # (by the library) before the timed steps; training rounds them every
    # step, since the optimizer changes them
    held_bf16 = not w.backward and w.gemm_dtype == sru.GEMM_BF16
    if held_bf16:
        for p in layers:
            if "W" in p:
                p["W"] = sru.round_bf16(p["W"])
    X, dH, mask = to(inp["X"]), to(inp["dH"]), to(inp["mask"])
    st = sru.Stack(layers, w.L, w.B, w.d_in, w.d, w.direction, w.gemm_dtype, dev,
                   backward=w.backward, highway_scale=args.highway_scale,
                   reset_new=args.reset_new, store_c=w.store_c, linear=w.linear)

    def eager_step():
        st.forward(X, mask)
        if w.backward:
            st.backward(X, dH, mask)

    if args.yardstick:
        print(json.dumps(yardstick(w, st, X, dH, mask, eager_step)), flush=True)
        return

    if args.cold_protocols:
        eager_step()
        torch.cuda.synchronize()
        table = {m: cold_scans(w, st, X, dH, mask, max(args.cold_reps, 3), args.highway_scale,
                               args.reset_new, mode=m) for m in FLUSH_MODES}
        for m, r in table.items():
            log("  " + m.ljust(11) + "  ".join(f"{k} {v['avg_us']:8.2f} us ({v['frac']:.3f})"
                                              for k, v in r.items()))
        print(json.dumps({"workload": w.name, "cold_protocols": table}), flush=True)
        return

    step = eager_step
    if args.graph:
        step = st.capture(X, dH, mask).replay
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup {args.warmup} done")

    # the library launches on torch's current stream, so torch's events
    # bracket each step; the wall clock brackets all of them
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t0 = time.perf_counter()
    marks[0].record()
    for i in range(args.steps):
        step()
        marks[i + 1].record()
    torch.cuda.synchronize()
    secs = time.perf_counter() - t0
    step_ms = sorted(marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps))
    ms_per_step = 1e3 * secs / args.steps
    tokens_per_s = w.tokens * args.steps / secs
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step, {tokens_per_s:.4g} tokens/s "
        f"(median {step_ms[len(step_ms) // 2]:.3f}, min {step_ms[0]:.3f} ms)")

    # --- per-kernel durations: the library brackets each launch with events
    per_step = w.layers * 32  # upper bound on kernels per layer and step
    ev = HipEvents(2 * per_step * args.profile_steps + 2)
    lib = sru.lib()
    lead = GpuLead()
    lead_ms = 3.0 * host_ms(eager_step) + 0.5
    lib.sru_timing_begin(ev.events, ev.n)
    try:
        for _ in range(args.profile_steps):
            lead(lead_ms)  # the step's launches queue before the GPU reaches them
            eager_step()  # the hook brackets launches, which a graph replay does not make
    finally:
        nk = lib.sru_timing_end()
    torch.cuda.synchronize()
    if 2 * nk + 2 > ev.n:  # the hook ran out of events: the counts would be short
        raise RuntimeError(f"per-launch timing ran out of events ({nk} kernels)")
    agg = {}
    for i in range(nk):
        lab = lib.sru_timing_label(i).decode()
        ms = ev.elapsed_ms(2 * i, 2 * i + 1)
        a = agg.setdefault(lab, [0.0, 0])
        a[0] += ms
        a[1] += 1
    ev.close()
    splits = dw_splits(lib, w) if w.backward and w.dp is None else 1
    work = kernel_work(w, splits, w.gemm_dtype == sru.GEMM_BF16)
    gemm_peak = MFMA_PEAK_TFLOPS["bf16" if w.gemm_dtype == sru.GEMM_BF16 else "fp32"]
    kernels = {}
    for lab, (tot, cnt) in agg.items():
        avg_ms = tot / cnt
        wk = work.get(lab, {})
        row = {"avg_us": round(avg_ms * 1e3, 2), "launches_per_step": cnt // args.profile_steps,
               "ms_per_step": round(tot / args.profile_steps, 4)}
        if "flops" in wk:
            tf = wk["flops"] / (avg_ms * 1e-3) / 1e12
            row.update(bound="mfma", achieved=round(tf, 1), unit="TFLOP/s", peak=gemm_peak,
                       frac=round(tf / gemm_peak, 4), algorithmic=wk["flops"])
        elif "bytes" in wk:
            gbps = wk["bytes"] / (avg_ms * 1e-3) / 1e9
            row.update(bound="hbm", achieved=round(gbps, 1), unit="GB/s", peak=HBM_PEAK_GBPS,
                       frac=round(gbps / HBM_PEAK_GBPS, 4), algorithmic=wk["bytes"])
        kernels[lab] = row
    dominant = max(kernels, key=lambda k: kernels[k]["ms_per_step"])
    d = kernels[dominant]
    roofline = {"kernel": dominant, "bound": d.get("bound"), "achieved": d.get("achieved"),
                "peak": d.get("peak"), "unit": d.get("unit"), "frac": d.get("frac"),
                "avg_us": d["avg_us"], "traffic": pmc_traffic(dominant, w.name)}
    scan_hbm = {k: {"GBps": kernels[k]["achieved"], "frac": kernels[k]["frac"],
                    "avg_us": kernels[k]["avg_us"], "traffic": pmc_traffic(k, w.name)}
                for k in ("scan_fwd", "scan_bwd") if k in kernels}
    for k, v in sorted(kernels.items(), key=lambda kv: -kv[1]["ms_per_step"]):
        log(f"  {k:14s} {v['avg_us']:9.2f} us x{v['launches_per_step']}  "
            f"{v.get('achieved', '-')} {v.get('unit', '')} ({v.get('frac', '-')})")

    cold = None
    if args.cold_reps > 0:
        cold = cold_scans(w, st, X, dH, mask, args.cold_reps, args.highway_scale,
                          args.reset_new)
    if cold:
        for k, v in cold.items():
            log(f"  cold {k}: {v['avg_us']} us, {v['GBps']} GB/s ({v['frac']})")
    valid = None if inp["mask"] is None else int((inp["mask"] == 0).sum())

    cpu = None
    if args.cpu_seqs > 0:
        log(f"cpu oracle on {args.cpu_seqs} sequences ...")
        cpu = cpu_baseline(w, inp, args.cpu_seqs)
        log(f"cpu oracle: {cpu['value']:.4g} tokens/s in {cpu['seconds']:.1f} s "
            f"({cpu['cores']} threads)")

    out = {
        "metric": ("SRU fwd+bwd tokens/s at L256 B64 d1024; scan-kernel HBM GB/s % of peak"
                   if args.workload == 3 else
                   f"SRU {'fwd+bwd' if w.backward else 'fwd'} tokens/s at {w.name}"),
        "value": tokens_per_s,
        "unit": "tokens/s",
        "valid_tokens_per_s": None if valid is None else valid * args.steps / secs,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "ms_per_step_median": step_ms[len(step_ms) // 2],
        "ms_per_step_min": step_ms[0],
        "tokens_per_s_median": w.tokens / (step_ms[len(step_ms) // 2] * 1e-3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.gemm_dtype == sru.GEMM_BF16 else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "layers": w.layers, "L": w.L, "B": w.B,
                   "d_in": w.d_in, "d": w.d,
                   "direction": ["forward", "reverse", "bidirectional"][w.direction],
                   "passes": "fwd+bwd" if w.backward else "fwd",
                   "gemm": "bf16 operands, fp32 accumulate" if w.gemm_dtype else "fp32",
                   "weights": ("bf16, rounded once before the timed steps (inference)"
                               if held_bf16 else
                               "fp32, rounded to bf16 in every step" if w.gemm_dtype
                               else "fp32"),
                   "scan": "fp32", "tokens_per_step": w.tokens, "global_batch": w.B,
                   "valid_tokens_per_step": valid,
                   "highway_scale": args.highway_scale,
                   "reset_gate": "c_t (Algorithm 1)" if args.reset_new else "c_{t-1} (Eq. 3)",
                   "recurrence": ("linear: v * c removed (ablation (1), Sec. 4.5)" if w.linear
                                  else "gated (Eq. 1-4)"),
                   "seq_len": w.L, "parallelism": "single GPU",
                   "launch": "hip graph replay" if args.graph else "eager"},
        "roofline": roofline,
        "scan_hbm": scan_hbm,
        "scan_cold": cold,
        "kernels": kernels,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
