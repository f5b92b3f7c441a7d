"""TEST INFRASTRUCTURE ONLY: fp64 CPU oracle of the translator fit.

Section 5 of the paper trains the translator T_theta by minimising a
representation distance D(T_theta(KV_A(C)), KV_B(C)) between translated and
natively prefilled target caches; Section 2.2 recalls closed-form linear maps
between the caches of two models.  For the per-layer affine translator of
the hot path (u = W z + b, target RoPE applied after it) and D the squared
Frobenius distance over the whole target cache, the problem is a linear
least-squares fit per (target layer, K|V).  This oracle adds a ridge term
lam * ||W||_F^2 (the bias is not penalised) so that the fit is well posed for
any number of rows, and solves the normal equations directly.

Because RoPE is a rotation, the distance between the translated cache and the
native cache equals the distance between the pre-rotation outputs u and the
native rows de-rotated by the target RoPE; the fit therefore regresses

    Y = [R_tgt(-t) K_B[l][b][h][t]]_h   (K)   or   [V_B[l][b][h][t]]_h   (V)

on the pooled, source-de-rotated rows Z of the hot path's steps 1-2:

    min_{W, b}  sum_rows ||Y_r - W Z_r - b||^2 + lam ||W||_F^2.

With Zt = [Z, 1] (bias) the minimiser solves (Zt^T Zt + lam D) [W b]^T =
Zt^T Y, D = diag(1, ..., 1, 0).  Everything is fp64 numpy; the only library
step is the dense linear solve.  Nothing here imports the GPU library.
"""
from __future__ import annotations

import numpy as np


def _widen(a, dtype=None) -> np.ndarray:
    """Storage array (float32, or bfloat16 bit patterns as uint16) -> fp64."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def inv_freq(head_dim: int, base: float, table=None) -> np.ndarray:
    """theta_i = base^(-2i/D), i < D/2 (or the override table)."""
    if table is not None:
        return np.asarray(table, dtype=np.float64)
    i = np.arange(head_dim // 2, dtype=np.float64)
    return base ** (-2.0 * i / head_dim)


def rotate(x: np.ndarray, pos: np.ndarray, theta: np.ndarray, sign: float) -> np.ndarray:
    """Rotate-half RoPE of rows x [n, D] at positions pos [n] by sign*pos*theta.

    y_i = x_i cos(a) - x_{i+D/2} sin(a),  y_{i+D/2} = x_{i+D/2} cos(a) + x_i sin(a),
    a = sign * pos * theta_i."""
    half = x.shape[-1] // 2
    ang = sign * np.outer(pos.astype(np.float64), theta)
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[:, :half], x[:, half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=1)


def source_rows(prob, layer: int, which: int, src_theta=None) -> np.ndarray:
    """Pooled, de-rotated source rows Z [R, din] of target layer `layer`
    (which 0 = K, 1 = V), rows concatenated per context."""
    spec = prob.spec
    s = spec.src
    src = prob.src_k if which == 0 else prob.src_v
    T = spec.src_tokens
    use_rope = which == 0 and s.rope_base > 0
    theta = inv_freq(s.head_dim, s.rope_base, src_theta) if use_rope else None
    lmap = np.asarray(prob.layer_map if prob.layer_map is not None else spec.layer_map)
    out = []
    row = 0
    for b in range(spec.batch):
        parts = []
        for j in range(spec.mix):
            ls = int(lmap[layer * spec.mix + j])
            for h in range(s.n_kv_heads):
                x = _widen(src[ls, b, h], spec.dtype)          # [T, Ds]
                if use_rope:
                    x = rotate(x, np.arange(T), theta, -1.0)
                parts.append(x)
        xb = np.concatenate(parts, axis=1) if parts else np.zeros((T, 0))   # [T, din]
        if prob.row_ptr is None:
            out.append(xb)
            continue
        tt = int(prob.tgt_tokens[b])
        zb = np.zeros((tt, xb.shape[1]))
        for t in range(tt):
            e0, e1 = int(prob.row_ptr[row + t]), int(prob.row_ptr[row + t + 1])
            for e in range(e0, e1):
                zb[t] += float(prob.weight[e]) * xb[int(prob.col_idx[e])]
        row += tt
        out.append(zb)
    return np.concatenate(out, axis=0)


def target_rows(prob, tgt, which: int, tgt_theta=None) -> np.ndarray:
    """Regression targets Y [Lt, R, dout] from a native target cache
    tgt [Lt][B][Ht][cap][Dt] (K de-rotated by the target RoPE at the target
    token's own position; V as stored)."""
    spec = prob.spec
    t_ = spec.tgt
    tt = np.asarray(prob.tgt_tokens)
    use_rope = which == 0 and t_.rope_base > 0
    theta = inv_freq(t_.head_dim, t_.rope_base, tgt_theta) if use_rope else None
    layers = []
    for l in range(t_.n_layers):
        rows = []
        for b in range(spec.batch):
            n = int(tt[b])
            heads = []
            for h in range(t_.n_kv_heads):
                y = _widen(tgt[l, b, h, :n], None)
                if use_rope:
                    y = rotate(y, np.arange(n), theta, -1.0)
                heads.append(y)
            rows.append(np.concatenate(heads, axis=1))
        layers.append(np.concatenate(rows, axis=0))
    return np.stack(layers)


def solve(Z: np.ndarray, Y: np.ndarray, lam: float, fit_bias: bool):
    """Ridge least squares: returns (W [dout, din], b [dout] or None)."""
    n, din = Z.shape
    Zt = np.concatenate([Z, np.ones((n, 1))], axis=1) if fit_bias else Z
    D = np.ones(Zt.shape[1])
    if fit_bias:
        D[-1] = 0.0
    A = Zt.T @ Zt + lam * np.diag(D)
    X = np.linalg.solve(A, Zt.T @ Y)          # [din(+1), dout]
    W = X[:din].T.copy()
    b = X[din].copy() if fit_bias else None
    return W, b


def fit(prob, tgt_k, tgt_v, lam: float, fit_bias: bool = True, src_theta=None,
        tgt_theta=None):
    """Per-layer fit of K and V translators from paired caches.

    Returns (w_k, w_v) fp64 [Lt, dout, din] and (b_k, b_v) fp64 [Lt, dout]
    (zeros without a bias)."""
    spec = prob.spec
    Lt = spec.tgt.n_layers
    yk = target_rows(prob, tgt_k, 0, tgt_theta)
    yv = target_rows(prob, tgt_v, 1, tgt_theta)
    ws, bs = [], []
    for which, Y in ((0, yk), (1, yv)):
        wl, bl = [], []
        for l in range(Lt):
            Z = source_rows(prob, l, which, src_theta)
            W, b = solve(Z, Y[l], lam, fit_bias)
            wl.append(W)
            bl.append(b if b is not None else np.zeros(W.shape[0]))
        ws.append(np.stack(wl))
        bs.append(np.stack(bl))
    return ws[0], ws[1], bs[0], bs[1]


def objective(prob, tgt, which: int, W, b, lam: float, src_theta=None, tgt_theta=None):
    """sum over layers of ||Y - Z W^T - b||^2 + lam ||W||^2 (pre-rotation form)."""
    Y = target_rows(prob, tgt, which, tgt_theta)
    total = 0.0
    for l in range(prob.spec.tgt.n_layers):
        Z = source_rows(prob, l, which, src_theta)
        r = Y[l] - Z @ W[l].T - (b[l] if b is not None else 0.0)
        total += float((r * r).sum()) + lam * float((W[l] * W[l]).sum())
    return total
