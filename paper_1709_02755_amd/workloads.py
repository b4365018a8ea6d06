"""Seeded synthetic workloads for the SRU layer (input generation only).

This module draws random tensors and holds the workload table; it contains
none of the layer's arithmetic.  Both the HIP path (through the benchmark and
tests) and the CPU oracle receive the float32 arrays it returns.

The paper trains on public datasets (SST, SQuAD, WMT, Enwik8) that are not
available here; these synthetic tensors stand in for them, with the shapes
below and the value distributions of the initialisation paragraph (Sec. 3.2):
weights uniform on [-sqrt(3/d), +sqrt(3/d)], i.e. variance 1/d.

Draw order (fixed, PCG64 = numpy.random.default_rng(seed)), all in float64
then cast to float32:
  1. lengths, if the workload is masked: integers uniform in [lo, L]
     inclusive, then lengths[0] = L so the full length always occurs;
  2. X ~ N(0, 1) of shape [L, B, d_in] (padded positions included);
  3. per layer: W ~ U(-sqrt(3/d), sqrt(3/d)) of shape [ndir, k, d, d_in]
     (low-rank workloads instead: Q ~ U(-sqrt(3/d_in), sqrt(3/d_in)) of shape
     [d_in, dp], then P ~ U(-sqrt(3/dp), sqrt(3/dp)) of shape [ndir, k, d, dp]),
     v_f, v_r ~ U(-0.5, 0.5), b_f ~ U(-1, 1) or 0, b_r = 0;
  4. dH ~ N(0, 1) on the last layer's H (only when a backward pass runs).
c0 = 0 everywhere.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

DIR_FWD, DIR_REV, DIR_BI = 0, 1, 2
GEMM_FP32, GEMM_BF16 = 0, 1


@dataclass(frozen=True)
class Workload:
    name: str
    layers: int
    direction: int          # DIR_FWD / DIR_REV / DIR_BI
    L: int
    B: int
    d_in: int               # input width of the first layer
    d: int                  # hidden width per direction
    gemm_dtype: int         # GEMM_FP32 / GEMM_BF16
    backward: bool
    len_lo: int | None      # None: all sequences full length
    bf_uniform: bool        # b_f ~ U(-1, 1) (else 0)
    seed: int
    store_c: bool = True    # keep every state C (False: inference, no backward)
    dp: int | None = None   # projection rank: Wcat = P Q^T (Sec. 4.4), else dense
    linear: bool = False    # v * c removed from both gates (ablation (1), Sec. 4.5)

    @property
    def ndir(self) -> int:
        return 2 if self.direction == DIR_BI else 1

    def layer_dims(self, li: int) -> tuple[int, int]:
        """(d_in, k) of layer li: later layers take the previous H."""
        d_in = self.d_in if li == 0 else self.ndir * self.d
        return d_in, (3 if d_in == self.d else 4)

    @property
    def tokens(self) -> int:
        return self.L * self.B


# Five workloads of the SRU layer at the sizes of its common uses (layers,
# direction, L, B, d, product precision, padding), then the inference shape
# of the SRU that replaces a Transformer's feed-forward layer (Sec. 4.3:
# d_model = 512 in, d_sru = 2048, batches of about 5120 tokens; forward only,
# no C), the 6-layer stack with the projection trick, workload 2 with
# the linear recurrence, and one GPU's shard of the headline stack; seeds
# are the workload index.  The linear workload still draws v_f, v_r (same draw
# order as the others); nothing reads them.
WORKLOADS = [
    Workload("sru1_L32_B4_d128_fp32_fwd", 1, DIR_FWD, 32, 4, 128, 128,
             GEMM_FP32, False, None, False, 0),
    Workload("sru2_L64_B32_d256_fp32", 2, DIR_FWD, 64, 32, 256, 256,
             GEMM_FP32, True, None, False, 1),
    Workload("bisru3_L400_B32_d128_fp32_masked", 3, DIR_BI, 400, 32, 128, 128,
             GEMM_FP32, True, 200, False, 2),
    Workload("sru6_L256_B64_d1024_bf16", 6, DIR_FWD, 256, 64, 1024, 1024,
             GEMM_BF16, True, None, True, 3),
    Workload("sru4_L128_B128_d2048_bf16_masked", 4, DIR_FWD, 128, 128, 2048, 2048,
             GEMM_BF16, True, 64, True, 4),
    Workload("ffn_L64_B80_din512_d2048_bf16_infer", 1, DIR_FWD, 64, 80, 512, 2048,
             GEMM_BF16, False, None, True, 5, store_c=False),
    # the headline stack with the projection trick at the paper's rank 512
    Workload("sru6_L256_B64_d1024_dp512_bf16", 6, DIR_FWD, 256, 64, 1024, 1024,
             GEMM_BF16, True, None, True, 6, dp=512),
    # the question-answering shape of workload 2 without the v * c terms: the
    # recurrence is linear in c, so its scans also run parallel over time
    Workload("bisru3_L400_B32_d128_fp32_masked_linear", 3, DIR_BI, 400, 32, 128, 128,
             GEMM_FP32, True, 200, False, 7, linear=True),
    # one GPU's share of the headline stack under 8-way data parallelism:
    # the batch of 64 sequences cut into 8 shards of 8 (sequences never
    # interact, so each GPU runs the whole stack on its shard)
    Workload("sru6_L256_B8_d1024_bf16_dp8_shard", 6, DIR_FWD, 256, 8, 1024, 1024,
             GEMM_BF16, True, None, True, 8),
]


def scaled(w: Workload, *, L=None, B=None, d=None, layers=None, name=None) -> Workload:
    """The same workload structure at other sizes (for parity at small sizes)."""
    L = w.L if L is None else L
    d = w.d if d is None else d
    d_in = d if w.d_in == w.d else (w.d_in * d) // w.d
    len_lo = None if w.len_lo is None else max(1, (w.len_lo * L) // w.L)
    dp = None if w.dp is None else max(8, (w.dp * d) // w.d)
    return Workload(name or f"{w.name}@L{L}_B{B or w.B}_d{d}", layers or w.layers,
                    w.direction, L, B or w.B, d_in, d, w.gemm_dtype, w.backward,
                    len_lo, w.bf_uniform, w.seed, w.store_c, dp, w.linear)


def lengths_to_mask(lengths: np.ndarray, L: int) -> np.ndarray:
    """[L, B] uint8, 1 where t >= length[b] (a padded position)."""
    t = np.arange(L)[:, None]
    return (t >= np.asarray(lengths)[None, :]).astype(np.uint8)


def irregular_mask(rng, L: int, B: int) -> np.ndarray:
    """[L, B] uint8 padding that is not a suffix, cycling over B by sequence:
    no padding, every step padded, random holes (about 40 %), the first third
    padded, a single valid step in the middle.  The layer's mask is any [L, B]
    pattern; these are the degenerate ones beside the usual padded tails."""
    m = np.zeros((L, B), np.uint8)
    for b in range(B):
        kind = b % 5
        if kind == 1:
            m[:, b] = 1
        elif kind == 2:
            m[:, b] = rng.random(L) < 0.4
            m[rng.integers(L), b] = 0
        elif kind == 3:
            m[: L // 3, b] = 1
        elif kind == 4:
            m[:, b] = 1
            m[L // 2, b] = 0
    return m


def draw_layer(rng, ndir: int, k: int, d: int, d_in: int, bf_uniform: bool,
               dp: int | None = None) -> dict:
    if dp is None:
        bound = math.sqrt(3.0 / d)
        mats = dict(W=rng.uniform(-bound, bound, size=(ndir, k, d, d_in)))
    else:
        bq, bp = math.sqrt(3.0 / d_in), math.sqrt(3.0 / dp)
        Q = rng.uniform(-bq, bq, size=(d_in, dp))
        mats = dict(Q=Q, P=rng.uniform(-bp, bp, size=(ndir, k, d, dp)))
    v_f = rng.uniform(-0.5, 0.5, size=(ndir, d))
    v_r = rng.uniform(-0.5, 0.5, size=(ndir, d))
    b_f = rng.uniform(-1.0, 1.0, size=(ndir, d)) if bf_uniform else np.zeros((ndir, d))
    b_r = np.zeros((ndir, d))
    return {k_: np.ascontiguousarray(v.astype(np.float32)) for k_, v in
            dict(mats, v_f=v_f, v_r=v_r, b_f=b_f, b_r=b_r).items()}


def make_inputs(w: Workload, seed: int | None = None) -> dict:
    """All float32 / uint8 arrays of one step of workload `w`."""
    rng = np.random.default_rng(w.seed if seed is None else seed)
    lengths = None
    mask = None
    if w.len_lo is not None:
        lengths = rng.integers(w.len_lo, w.L + 1, size=w.B)
        lengths[0] = w.L
        mask = lengths_to_mask(lengths, w.L)
    X = rng.standard_normal((w.L, w.B, w.d_in)).astype(np.float32)
    layers = []
    for li in range(w.layers):
        d_in, k = w.layer_dims(li)
        layers.append(draw_layer(rng, w.ndir, k, w.d, d_in, w.bf_uniform, w.dp))
    dH = None
    if w.backward:
        dH = rng.standard_normal((w.L, w.B, w.ndir * w.d)).astype(np.float32)
    return dict(X=X, layers=layers, dH=dH, mask=mask, lengths=lengths)


def random_layer_case(rng, L, B, d_in, d, direction, *, masked=False, c0=False,
                      dc_last=False, bias_scale=0.0, v_scale=0.5, x_scale=1.0):
    """One layer's inputs at arbitrary sizes, for tests (float32 arrays)."""
    ndir = 2 if direction == DIR_BI else 1
    k = 3 if d_in == d else 4
    X = (x_scale * rng.standard_normal((L, B, d_in))).astype(np.float32)
    bound = math.sqrt(3.0 / d)
    out = dict(
        X=X,
        W=rng.uniform(-bound, bound, (ndir, k, d, d_in)).astype(np.float32),
        v_f=rng.uniform(-v_scale, v_scale, (ndir, d)).astype(np.float32),
        v_r=rng.uniform(-v_scale, v_scale, (ndir, d)).astype(np.float32),
        b_f=rng.uniform(-bias_scale, bias_scale, (ndir, d)).astype(np.float32)
        if bias_scale else np.zeros((ndir, d), np.float32),
        b_r=rng.uniform(-bias_scale, bias_scale, (ndir, d)).astype(np.float32)
        if bias_scale else np.zeros((ndir, d), np.float32),
        c0=rng.standard_normal((B, ndir * d)).astype(np.float32) if c0 else None,
        dc_last=rng.standard_normal((B, ndir * d)).astype(np.float32) if dc_last else None,
        dH=rng.standard_normal((L, B, ndir * d)).astype(np.float32),
        mask=None,
    )
    if masked:
        lengths = rng.integers(max(1, L // 2), L + 1, size=B)
        lengths[0] = L
        if B > 1:
            lengths[-1] = max(1, L // 2)
        out["mask"] = lengths_to_mask(lengths, L)
        out["lengths"] = lengths
    return out
