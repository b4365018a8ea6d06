"""Plain fp64 CPU oracle for one Simple Recurrent Unit (SRU) layer.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the test suite, the smoke check and the CPU-baseline
leg of the benchmark use it.  It shares no code with the HIP library and
imports nothing from the product package.

What it computes (Lei et al., "Simple Recurrent Units for Highly
Parallelizable Recurrence", Sec. 3, Eq. 1-4):

    f_t = sigma(W_f x_t + v_f * c_{t-1} + b_f)          (Eq. 1)
    c_t = f_t * c_{t-1} + (1 - f_t) * (W x_t)            (Eq. 2)
    r_t = sigma(W_r x_t + v_r * c_{t-1} + b_r)          (Eq. 3)
    h_t = r_t * c_t + (1 - r_t) * x_t                    (Eq. 4)

The forward pass is the plain per-step definition (the "naive
implementation" of Sec. 3.1 that evaluates Eq. 1-4 one step at a time, with
the projections x_t W^T computed inside the time loop).  The batched
reorganisation of Sec. 3.1 (one matrix product for all steps, then the fused
element-wise loop of Algorithm 1) is what the GPU path implements; the oracle
does NOT assume it, and the test suite checks the two organisations agree.

Readings of the paper taken here (each is also listed in the design notes):
  * The reset gate uses c_{t-1}, as Eq. 3 writes it (Algorithm 1 evaluates r
    after updating c; Eq. 3 is taken as the definition).  With
    reset_new=True it uses c_t instead: Algorithm 1's order.
  * Highway scaling alpha = 1 (Eq. 4 as printed, no scaling correction).
    Sec. 3.2 multiplies the highway term by a constant alpha (sqrt(3), or
    sqrt(1 + 2 e^b) for a reset-gate bias b, Appendix A); the alpha
    argument does that:  h_t = r_t * c_t + (1 - r_t) * x_hat * alpha.
  * "b_v" after Eq. 4 is read as b_r.
  * When d_in != d, Eq. 4 has no x_t of width d; the highway term uses a
    fourth learned block W_h (x_hat = W_h x_t), stored as projection block 3.
    With d_in == d, x_hat = x_t and there are k = 3 blocks.
  * Padding: a padded step (t, b) leaves c unchanged and outputs h = 0; its
    upstream gradient is ignored and it contributes no parameter gradient.
  * Bidirectional: the two directions are independent layers (own W, v, b,
    c0); the reverse one visits t = L-1 .. 0.  Features are concatenated
    [forward | reverse].
  * bf16 GEMM mode rounds the operands of the three matrix products (and only
    those) to bfloat16, round-to-nearest-even; state and gates stay wide.
  * linear=True is ablation (1) of the ablation analysis (Sec. 4.5): the
    point-wise terms v_f * c_{t-1} and v_r * c_{t-1} are removed from both
    gates, so f_t and r_t depend on x_t only and c_t = f_t c_{t-1} +
    (1 - f_t) W x_t is a linear recurrence in c.  The removed term is taken
    as zero; v_f and v_r are then not read and have no gradient (None).

The backward pass is not in the paper (training by back-propagation is
implied by the optimisers of Sec. 4).  It is the chain rule of Eq. 1-4 taken
in reverse step order; the formulas are derived in the design notes and
pinned by finite differences in the tests.

Shapes (row-major, same as the C ABI):
  X   [L, B, d_in]           W  [ndir, k, d, d_in]
  v_f, v_r, b_f, b_r [ndir, d]
  c0, c_last, dc0, dc_last [B, ndir*d]
  U   [L, B, ndir, k, d]     H, C, dH [L, B, ndir*d]
  pad_mask [L, B] (nonzero = padded) or None
"""

from __future__ import annotations

import numpy as np

DIR_FWD, DIR_REV, DIR_BI = 0, 1, 2
GEMM_FP32, GEMM_BF16 = 0, 1


def _f64(a):
    return None if a is None else np.asarray(a, dtype=np.float64)


# Precision in which the matrix products accumulate: fp64 (exact for the
# oracle's purposes).  A test may set it to np.float32 to evaluate the same
# method the way an fp32-accumulating implementation does, which measures how
# far accumulation order alone can move a bf16-mode result (each product's
# output then differs by fp32 rounding, and a value that crosses a bf16
# rounding boundary changes the next product's operand by a whole bf16 step).
PRODUCT_ACCUMULATION = np.float64


def _mm(a, b):
    """The matrix product a @ b, accumulated in PRODUCT_ACCUMULATION,
    returned as fp64."""
    if PRODUCT_ACCUMULATION is np.float64:
        return np.asarray(a, np.float64) @ np.asarray(b, np.float64)
    acc = PRODUCT_ACCUMULATION
    return (np.asarray(a, acc) @ np.asarray(b, acc)).astype(np.float64)


def bf16_round(a):
    """Round to the nearest bfloat16 value (ties to even), returned as fp64.

    A bfloat16 keeps the top 16 bits of an IEEE binary32.  The value is first
    rounded to binary32 (the GPU rounds fp32 values), then the low 16 bits are
    rounded away: add 0x7FFF plus the lowest kept bit, truncate.  NaN inputs
    stay NaN; +-Inf stay Inf.
    """
    a32 = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    bits = a32.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    rounded = ((bits + 0x7FFF + lsb) >> 16) << 16
    nan = np.isnan(a32)
    rounded = np.where(nan, bits | 0x00400000, rounded)  # keep NaN quiet NaN
    out = (rounded & 0xFFFFFFFF).astype(np.uint32).view(np.float32)
    return out.astype(np.float64)


def sigmoid(z):
    """Logistic function 1 / (1 + e^{-z}) in fp64 (Eq. 1 and 3)."""
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-z))


def scaling_alpha(b):
    """Highway scaling constant for a reset-gate bias b (Sec. 3.2, derived in
    Appendix A): alpha = sqrt(1 + 2 e^b), sqrt(3) at b = 0."""
    return float(np.sqrt(1.0 + 2.0 * np.exp(b)))


def _ndir(direction):
    if direction not in (DIR_FWD, DIR_REV, DIR_BI):
        raise ValueError(f"unknown direction {direction}")
    return 2 if direction == DIR_BI else 1


def _is_reverse(direction, dirn):
    return direction == DIR_REV or (direction == DIR_BI and dirn == 1)


def _gate_weights(v_f, v_r, ndir, d, linear):
    """v_f, v_r as [ndir, d] fp64, or zeros for the linear variant (the
    removed point-wise term contributes nothing)."""
    if linear:
        return np.zeros((ndir, d)), np.zeros((ndir, d))
    return _f64(v_f).reshape(ndir, d), _f64(v_r).reshape(ndir, d)


def _check_shapes(X, W, direction):
    L, B, d_in = X.shape
    ndir, k, d, d_in_w = W.shape
    if ndir != _ndir(direction):
        raise ValueError("W's first axis must be the number of directions")
    if d_in_w != d_in:
        raise ValueError("W's last axis must be d_in")
    want_k = 3 if d_in == d else 4
    if k != want_k:
        raise ValueError(f"k must be {want_k} for d_in={d_in}, d={d}")
    return L, B, d_in, ndir, k, d


def forward(X, W, v_f, v_r, b_f, b_r, c0=None, direction=DIR_FWD,
            pad_mask=None, gemm_dtype=GEMM_FP32, alpha=1.0, reset_new=False, linear=False):
    """Eq. 1-4 evaluated step by step; returns dict(U, H, C, c_last).

    alpha scales the highway term (Sec. 3.2); reset_new makes the reset gate
    read the updated state c_t (Algorithm 1's order) instead of c_{t-1};
    linear removes the v * c_{t-1} terms of both gates (ablation (1)).

    U holds the per-step projections x_t W^T (one block per gate), assembled
    in the [L, B, ndir, k, d] layout so that it can be compared with the
    batched projection.
    """
    X = _f64(X)
    W = _f64(W)
    L, B, d_in, ndir, k, d = _check_shapes(X, W, direction)
    v_f, v_r = _gate_weights(v_f, v_r, ndir, d, linear)
    b_f, b_r = (_f64(a).reshape(ndir, d) for a in (b_f, b_r))
    c0 = np.zeros((B, ndir, d)) if c0 is None else _f64(c0).reshape(B, ndir, d)
    pad = np.zeros((L, B), bool) if pad_mask is None else (np.asarray(pad_mask) != 0)
    bf16 = gemm_dtype == GEMM_BF16
    Wp = bf16_round(W) if bf16 else W

    U = np.zeros((L, B, ndir, k, d))
    H = np.zeros((L, B, ndir, d))
    C = np.zeros((L, B, ndir, d))
    c_last = np.zeros((B, ndir, d))
    for dirn in range(ndir):
        steps = range(L - 1, -1, -1) if _is_reverse(direction, dirn) else range(L)
        c = c0[:, dirn].copy()
        for t in steps:
            x_t = X[t]
            xp = bf16_round(x_t) if bf16 else x_t
            u = [_mm(xp, Wp[dirn, q].T) for q in range(k)]          # W x_t, W_f x_t, ...
            x_hat = x_t if k == 3 else u[3]
            f = sigmoid(u[1] + v_f[dirn] * c + b_f[dirn])        # Eq. 1
            c_new = f * c + (1.0 - f) * u[0]                      # Eq. 2
            s = c_new if reset_new else c                         # state r reads
            r = sigmoid(u[2] + v_r[dirn] * s + b_r[dirn])        # Eq. 3
            h = r * c_new + (1.0 - r) * x_hat * alpha             # Eq. 4 (Sec. 3.2)
            valid = ~pad[t][:, None]
            c = np.where(valid, c_new, c)
            H[t, :, dirn] = np.where(valid, h, 0.0)
            C[t, :, dirn] = c
            U[t, :, dirn] = np.stack(u, axis=1)
        c_last[:, dirn] = c
    return dict(U=U, H=H.reshape(L, B, ndir * d), C=C.reshape(L, B, ndir * d),
                c_last=c_last.reshape(B, ndir * d))


def backward(X, W, v_f, v_r, b_f, b_r, dH, c0=None, direction=DIR_FWD,
             pad_mask=None, gemm_dtype=GEMM_FP32, dc_last=None, fw=None, alpha=1.0,
             reset_new=False, linear=False):
    """Reverse-step chain rule of Eq. 1-4 (alpha, reset_new and linear as in
    forward; with linear, dv_f and dv_r are None).

    Returns dict(dX, dW, dv_f, dv_r, db_f, db_r, dc0, dU, dxh) where dU is
    the gradient with respect to the projections ([L, B, ndir, k, d]) and dxh
    the gradient reaching x_hat through the highway skip term (zeros when
    k = 4, where it is part of dU block 3).  The forward states come from
    `fw` (the result of `forward` on the same inputs) or are recomputed.
    """
    X = _f64(X)
    W = _f64(W)
    L, B, d_in, ndir, k, d = _check_shapes(X, W, direction)
    v_f, v_r = _gate_weights(v_f, v_r, ndir, d, linear)
    b_f, b_r = (_f64(a).reshape(ndir, d) for a in (b_f, b_r))
    c0_ = np.zeros((B, ndir, d)) if c0 is None else _f64(c0).reshape(B, ndir, d)
    pad = np.zeros((L, B), bool) if pad_mask is None else (np.asarray(pad_mask) != 0)
    dH = _f64(dH).reshape(L, B, ndir, d)
    g_init = np.zeros((B, ndir, d)) if dc_last is None else _f64(dc_last).reshape(B, ndir, d)
    bf16 = gemm_dtype == GEMM_BF16

    if fw is None:
        fw = forward(X, W, v_f, v_r, b_f, b_r, c0_.reshape(B, ndir * d), direction,
                     pad_mask, gemm_dtype, alpha, reset_new)  # v already zero if linear
    U = fw["U"]
    C = fw["C"].reshape(L, B, ndir, d)
    Wp = bf16_round(W) if bf16 else W

    dU = np.zeros((L, B, ndir, k, d))
    dxh = np.zeros((L, B, ndir, d))
    dX = np.zeros((L, B, d_in))
    dW = np.zeros((ndir, k, d, d_in))
    dv_f = np.zeros((ndir, d))
    dv_r = np.zeros((ndir, d))
    db_f = np.zeros((ndir, d))
    db_r = np.zeros((ndir, d))
    dc0 = np.zeros((B, ndir, d))

    for dirn in range(ndir):
        rev = _is_reverse(direction, dirn)
        fwd_steps = list(range(L - 1, -1, -1)) if rev else list(range(L))
        g = g_init[:, dirn].copy()                     # dloss/dc_t from later steps
        for pos in range(L - 1, -1, -1):               # reverse of the forward order
            t = fwd_steps[pos]
            c_p = C[fwd_steps[pos - 1], :, dirn] if pos > 0 else c0_[:, dirn]
            c_t = C[t, :, dirn]
            u0, u1, u2 = U[t, :, dirn, 0], U[t, :, dirn, 1], U[t, :, dirn, 2]
            x_hat = X[t] if k == 3 else U[t, :, dirn, 3]
            valid = ~pad[t][:, None]
            dh = np.where(valid, dH[t, :, dirn], 0.0)

            f = sigmoid(u1 + v_f[dirn] * c_p + b_f[dirn])
            s = c_t if reset_new else c_p             # the state r reads
            r = sigmoid(u2 + v_r[dirn] * s + b_r[dirn])
            dr = dh * (c_t - alpha * x_hat) * r * (1.0 - r)  # through r's pre-activation
            gc = g + dh * r                            # dh/dc_t = r
            if reset_new:
                gc = gc + dr * v_r[dirn]               # r also depends on c_t
            df = gc * (c_p - u0) * f * (1.0 - f)       # through f's pre-activation
            du0 = gc * (1.0 - f)
            dxhat = dh * (1.0 - r) * alpha
            df = np.where(valid, df, 0.0)
            dr = np.where(valid, dr, 0.0)
            du0 = np.where(valid, du0, 0.0)
            dxhat = np.where(valid, dxhat, 0.0)

            dU[t, :, dirn, 0] = du0
            dU[t, :, dirn, 1] = df
            dU[t, :, dirn, 2] = dr
            if k == 3:
                dxh[t, :, dirn] = dxhat
            else:
                dU[t, :, dirn, 3] = dxhat
            dv_f[dirn] += (df * c_p).sum(axis=0)
            dv_r[dirn] += (dr * s).sum(axis=0)
            db_f[dirn] += df.sum(axis=0)
            db_r[dirn] += dr.sum(axis=0)
            g_prev = gc * f + df * v_f[dirn]
            if not reset_new:
                g_prev = g_prev + dr * v_r[dirn]       # r depends on c_{t-1}
            g = np.where(valid, g_prev, g)             # padded step: identity on c

            # Projections: dX gets dU_t W, dW gets dU_t^T x_t (per step).
            x_t = X[t]
            du_t = dU[t, :, dirn]                      # [B, k, d]
            du_p = bf16_round(du_t) if bf16 else du_t
            xp = bf16_round(x_t) if bf16 else x_t
            for q in range(k):
                dX[t] += _mm(du_p[:, q], Wp[dirn, q])
                dW[dirn, q] += _mm(du_p[:, q].T, xp)
            if k == 3:
                dX[t] += dxh[t, :, dirn]
        dc0[:, dirn] = g
    if linear:
        dv_f = dv_r = None
    return dict(dX=dX, dW=dW, dv_f=dv_f, dv_r=dv_r, db_f=db_f, db_r=db_r,
                dc0=dc0.reshape(B, ndir * d), dU=dU, dxh=dxh)


def forward_batched(X, W, v_f, v_r, b_f, b_r, c0=None, direction=DIR_FWD, pad_mask=None,
                    alpha=1.0, reset_new=False, linear=False):
    """Sec. 3.1's organisation of the same layer, as a cross-check of
    forward() (fp32-GEMM mode): the projections of all L*B tokens come from
    one matrix product with the stacked weight [W; W_f; W_r(; W_h)] first,
    and the step loop of Eq. 1-4 then only reads its gate inputs from that
    batched tensor.  forward() instead multiplies inside the step loop, so
    agreement checks the reorganisation rather than assuming it.
    Returns dict(U, H, C, c_last)."""
    X = _f64(X)
    W = _f64(W)
    L, B, d_in, ndir, k, d = _check_shapes(X, W, direction)
    Wcat = W.reshape(ndir * k * d, d_in)                    # rows (dir, block, unit)
    U = _mm(X.reshape(L * B, d_in), Wcat.T).reshape(L, B, ndir, k, d)
    out = _scan_on_u(X, U, v_f, v_r, b_f, b_r, c0, direction, pad_mask, alpha, reset_new,
                     linear)
    out["U"] = U
    return out


def stack_forward_backward(X, layers, direction, pad_mask, gemm_dtype, dH_top,
                           need_backward=True, alpha=1.0, reset_new=False, linear=False):
    """Stacked layers: layer l+1 takes layer l's H as its X.

    `layers` is a list of dicts with W, v_f, v_r, b_f, b_r (c0 = 0).
    Returns dict(Hs=[H per layer], Cs=[...], Us=[...], grads=[per-layer
    backward dicts, bottom first]) ; grads is empty without backward.
    """
    xs = [np.asarray(X, np.float64)]
    fws = []
    for p in layers:
        if "Q" in p:  # low-rank layer (Sec. 4.4)
            fw = forward_lowrank(xs[-1], p["Q"], p["P"], p["v_f"], p["v_r"], p["b_f"], p["b_r"],
                                 None, direction, pad_mask, gemm_dtype, alpha, reset_new, linear)
        else:
            fw = forward(xs[-1], p["W"], p["v_f"], p["v_r"], p["b_f"], p["b_r"], None,
                         direction, pad_mask, gemm_dtype, alpha, reset_new, linear)
        fws.append(fw)
        xs.append(fw["H"])
    grads = []
    if need_backward:
        g = np.asarray(dH_top, np.float64)
        for li in range(len(layers) - 1, -1, -1):
            p = layers[li]
            if "Q" in p:
                bw = backward_lowrank(xs[li], p["Q"], p["P"], p["v_f"], p["v_r"], p["b_f"],
                                      p["b_r"], g, None, direction, pad_mask, gemm_dtype,
                                      fw=fws[li], alpha=alpha, reset_new=reset_new,
                                      linear=linear)
            else:
                bw = backward(xs[li], p["W"], p["v_f"], p["v_r"], p["b_f"], p["b_r"], g,
                              None, direction, pad_mask, gemm_dtype, fw=fws[li], alpha=alpha,
                              reset_new=reset_new, linear=linear)
            grads.append(bw)
            g = bw["dX"]
        grads.reverse()
    return dict(Hs=[fw["H"] for fw in fws], Cs=[fw["C"] for fw in fws],
                Us=[fw["U"] for fw in fws], grads=grads, xs=xs)


# ------------------------------------------------------ low-rank projection
# The projection (bottleneck) trick of Sec. 4.4: the stacked weights are a
# product of two smaller matrices, so the batched product runs as two.  The
# text writes the product as P^T Q with Q of shape [d_in, d'] and P of shape
# [3 d_out, d']; those shapes only compose as P Q^T, which is the reading
# taken here:  Wcat [ndir*k*d, d_in] = P Q^T,  U = (X Q) P^T.
# In bf16 mode the operands of each of the two products are rounded:
# X and Q for T = X Q; T and P for U = T P^T (and likewise backward).

def forward_lowrank(X, Q, P, v_f, v_r, b_f, b_r, c0=None, direction=DIR_FWD,
                    pad_mask=None, gemm_dtype=GEMM_FP32, alpha=1.0, reset_new=False,
                    linear=False):
    """Layer with Wcat = P Q^T.  Q [d_in, dp], P [ndir, k, d, dp].
    Returns dict(T, U, H, C, c_last) with T = X Q [L, B, dp]."""
    X = _f64(X)
    Q = _f64(Q)
    P = _f64(P)
    L, B, d_in = X.shape
    ndir, k, d, dp = P.shape
    bf16 = gemm_dtype == GEMM_BF16
    rnd = bf16_round if bf16 else (lambda a: a)
    T = _mm(rnd(X), rnd(Q))                               # [L, B, dp]
    U = _mm(rnd(T), rnd(P).reshape(ndir * k * d, dp).T).reshape(L, B, ndir, k, d)
    # the scan of Eq. 1-4 on this U: the dense oracle with W chosen so that
    # its per-step projections are exactly U is not available, so the step
    # loop is run here on U directly
    out = _scan_on_u(X, U, v_f, v_r, b_f, b_r, c0, direction, pad_mask, alpha, reset_new,
                     linear)
    out["T"] = T
    out["U"] = U
    return out


def _scan_on_u(X, U, v_f, v_r, b_f, b_r, c0, direction, pad_mask, alpha, reset_new, linear):
    """Eq. 1-4 per step given the projections U [L, B, ndir, k, d]."""
    L, B, ndir, k, d = U.shape
    v_f, v_r = _gate_weights(v_f, v_r, ndir, d, linear)
    b_f, b_r = (_f64(a).reshape(ndir, d) for a in (b_f, b_r))
    c0 = np.zeros((B, ndir, d)) if c0 is None else _f64(c0).reshape(B, ndir, d)
    pad = np.zeros((L, B), bool) if pad_mask is None else (np.asarray(pad_mask) != 0)
    H = np.zeros((L, B, ndir, d))
    C = np.zeros((L, B, ndir, d))
    c_last = np.zeros((B, ndir, d))
    for dirn in range(ndir):
        steps = range(L - 1, -1, -1) if _is_reverse(direction, dirn) else range(L)
        c = c0[:, dirn].copy()
        for t in steps:
            u = U[t, :, dirn]
            x_hat = X[t] if k == 3 else u[:, 3]
            f = sigmoid(u[:, 1] + v_f[dirn] * c + b_f[dirn])
            c_new = f * c + (1.0 - f) * u[:, 0]
            s = c_new if reset_new else c
            r = sigmoid(u[:, 2] + v_r[dirn] * s + b_r[dirn])
            h = r * c_new + (1.0 - r) * x_hat * alpha
            valid = ~pad[t][:, None]
            c = np.where(valid, c_new, c)
            H[t, :, dirn] = np.where(valid, h, 0.0)
            C[t, :, dirn] = c
        c_last[:, dirn] = c
    return dict(H=H.reshape(L, B, ndir * d), C=C.reshape(L, B, ndir * d),
                c_last=c_last.reshape(B, ndir * d))


def backward_lowrank(X, Q, P, v_f, v_r, b_f, b_r, dH, c0=None, direction=DIR_FWD,
                     pad_mask=None, gemm_dtype=GEMM_FP32, dc_last=None, fw=None, alpha=1.0,
                     reset_new=False, linear=False):
    """Gradients of the low-rank layer: dict(dX, dQ, dP, dv_f, dv_r, db_f,
    db_r, dc0, dU, dT).  The scan part is the dense backward's (the recurrence
    only sees U); then dT = dU P, dX = dT Q^T (+ the highway gradient when
    k = 3), dP = dU^T T, dQ = X^T dT, each product on rounded operands in
    bf16 mode."""
    X = _f64(X)
    Q = _f64(Q)
    P = _f64(P)
    L, B, d_in = X.shape
    ndir, k, d, dp = P.shape
    bf16 = gemm_dtype == GEMM_BF16
    rnd = bf16_round if bf16 else (lambda a: a)
    if fw is None:
        fw = forward_lowrank(X, Q, P, v_f, v_r, b_f, b_r, c0, direction, pad_mask, gemm_dtype,
                             alpha, reset_new, linear)
    # The recurrence gradients: run the dense backward with a weight whose
    # products are never used (W = 0) on the forward states of this layer.
    Wz = np.zeros((ndir, k, d, d_in))
    bw = backward(X, Wz, v_f, v_r, b_f, b_r, dH, c0, direction, pad_mask, GEMM_FP32, dc_last,
                  fw=dict(U=fw["U"], C=fw["C"]), alpha=alpha, reset_new=reset_new,
                  linear=linear)
    dU = bw["dU"].reshape(L, B, ndir * k * d)
    Pm = P.reshape(ndir * k * d, dp)
    dT = _mm(rnd(dU), rnd(Pm))                              # [L, B, dp]
    dX = _mm(rnd(dT), rnd(Q).T)
    if k == 3:
        dX = dX + bw["dxh"].sum(axis=2)
    dUm = rnd(dU).reshape(L * B, -1)
    dP = _mm(dUm.T, rnd(fw["T"]).reshape(L * B, dp)).reshape(ndir, k, d, dp)
    dQ = _mm(rnd(X).reshape(L * B, d_in).T, rnd(dT).reshape(L * B, dp))
    return dict(dX=dX, dQ=dQ, dP=dP, dv_f=bw["dv_f"], dv_r=bw["dv_r"], db_f=bw["db_f"],
                db_r=bw["db_r"], dc0=bw["dc0"], dU=bw["dU"], dT=dT, dxh=bw["dxh"])
