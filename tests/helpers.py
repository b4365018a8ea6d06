"""Shared helpers for the GPU parity tests (device transfer, tolerances)."""

import numpy as np
import torch

from conftest import rel_err

# Parity tolerances: 1e-5 relative for fp32 GEMMs, 2e-2 for the
# bf16-GEMM path, measured as max |g - r| / max(|r|, rms(r)) per tensor.
TOL_FP32 = 1e-5
TOL_BF16 = 2e-2
# The low-rank projection (Wcat = P Q^T) computes each projection as two
# chained products, so every gradient passes twice as many bf16-rounded
# operands as on the dense path; independent roundings add in quadrature,
# which scales the dense bar by sqrt(2) (2.8e-2), rounded up.
TOL_BF16_LOWRANK = 3e-2


def dev(a, dtype=None):
    if a is None:
        return None
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def host(t):
    return None if t is None else t.detach().cpu().numpy().astype(np.float64)


def check(name, got, ref, tol, report=None):
    e = rel_err(host(got) if isinstance(got, torch.Tensor) else got, ref)
    if report is not None:
        report[name] = e
    assert np.isfinite(e) and e <= tol, f"{name}: rel err {e:.3e} > {tol:.1e}"
    return e


def layer_to_dev(p):
    return {k: dev(v) for k, v in p.items()}
