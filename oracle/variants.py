"""TEST INFRASTRUCTURE ONLY: fp64 CPU oracle of translator variants.

Section 5 of the paper notes that translation may work through compressed
representations or low-dimensional latent adapters, and Section 2.2 recalls a
mixture of translator modules.  Two variants of the affine per-layer
translator follow from that (the rest of the operator -- source RoPE removal,
pooling, target RoPE -- is unchanged):

* low rank:  u = U[l] (V[l] z) + b[l],  U [dout, r], V [r, din];
* mixture:   u = sum_k alpha_k (W_k[l] z + b_k[l]) with fixed weights alpha_k.

Both are computed here literally (the latent vector V z first; every mixture
member applied and weighted), in fp64 numpy, from the pooled, de-rotated
source rows of the fit oracle, followed by the target rotation.  Nothing here
imports the GPU library.
"""
from __future__ import annotations

import numpy as np

from oracle import fit as F


def _finish(prob, U_rows, layer: int, which: int, tgt_theta=None):
    """Target rows u [R, dout] -> per-context head tensors with the target
    RoPE on K: returns [B, Ht, cap, Dt] (NaN past each context's end)."""
    spec = prob.spec
    t_ = spec.tgt
    tt = np.asarray(prob.tgt_tokens)
    cap = int(tt.max()) if len(tt) else 0
    out = np.full((spec.batch, t_.n_kv_heads, cap, t_.head_dim), np.nan)
    use_rope = which == 0 and t_.rope_base > 0
    theta = F.inv_freq(t_.head_dim, t_.rope_base, tgt_theta) if use_rope else None
    r0 = 0
    for b in range(spec.batch):
        n = int(tt[b])
        for h in range(t_.n_kv_heads):
            y = U_rows[r0:r0 + n, h * t_.head_dim:(h + 1) * t_.head_dim]
            if use_rope:
                y = F.rotate(y, np.arange(n), theta, +1.0)
            out[b, h, :n] = y
        r0 += n
    return out


def translate_lowrank(prob, u_k, v_k, u_v, v_v, b_k=None, b_v=None, src_theta=None,
                      tgt_theta=None):
    """Low-rank translators: u_k/u_v [Lt, dout, r], v_k/v_v [Lt, r, din]
    (any storage dtype; bf16 as uint16 bits), b [Lt, dout] or None.
    Returns (tgt_k, tgt_v) fp64 [Lt, B, Ht, cap, Dt]."""
    spec = prob.spec
    outs = []
    for which, U, V, b in ((0, u_k, v_k, b_k), (1, u_v, v_v, b_v)):
        U, V = F._widen(U), F._widen(V)
        layers = []
        for l in range(spec.tgt.n_layers):
            Z = F.source_rows(prob, l, which, src_theta)         # [R, din]
            latent = Z @ V[l].T                                   # [R, r]
            u = latent @ U[l].T                                   # [R, dout]
            if b is not None:
                u = u + np.asarray(b[l], dtype=np.float64)
            layers.append(_finish(prob, u, l, which, tgt_theta))
        outs.append(np.stack(layers))
    return outs[0], outs[1]


def translate_mixture(prob, alpha, w_k, w_v, b_k=None, b_v=None, src_theta=None,
                      tgt_theta=None):
    """Mixture of K translators: alpha [K], w [K, Lt, dout, din], b [K, Lt, dout]
    or None.  Every member is applied to the row and the outputs are
    weighted.  Returns (tgt_k, tgt_v) fp64 [Lt, B, Ht, cap, Dt]."""
    spec = prob.spec
    alpha = np.asarray(alpha, dtype=np.float64)
    outs = []
    for which, W, b in ((0, w_k, b_k), (1, w_v, b_v)):
        W = F._widen(W)
        layers = []
        for l in range(spec.tgt.n_layers):
            Z = F.source_rows(prob, l, which, src_theta)
            u = np.zeros((Z.shape[0], W.shape[2]))
            for k in range(len(alpha)):
                uk = Z @ W[k, l].T
                if b is not None:
                    uk = uk + np.asarray(b[k, l], dtype=np.float64)
                u += alpha[k] * uk
            layers.append(_finish(prob, u, l, which, tgt_theta))
        outs.append(np.stack(layers))
    return outs[0], outs[1]
