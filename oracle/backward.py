"""fp64 CPU oracle of the gradient of the Still compactor forward pass.

TEST INFRASTRUCTURE ONLY.  Only tests may import this module.  It shares no
code with the GPU library.  It covers the training hot path without the base
model: the paper trains each layer's compactor phi by backpropagating a loss
through the compact cache (Section 2.4, training; Appendix E).  The loss
itself stays out of scope.  Given upstream gradients dC_k, dC_v of one
layer's outputs, this module returns the gradient of
    L = <dC_k, C_k> + <dC_v, C_v>
with respect to every compactor tensor: the latent bank, every block's
projections and biases, and the output heads.  The cache K, V is an input of
the frozen base model and gets no gradient.

The forward pass is the one of oracle/compactor.py, evaluated again here with
every intermediate kept.  The backward pass applies the chain rule to each step
in reverse order, one step per function below:
* RMSNorm  y = x r, r = (mean x^2 + eps)^(-1/2):
      dx = r dy - (r^3 / D) x (x . dy)
* QK-norm  y = x / ||x||:  dx = (dy - y (y . dy)) / ||x||
* RoPE     y = R(phi) x:   dx = R(-phi) dy  (a rotation)
* softmax  P = softmax(S) per row:  dS = P * (dP - rowsum(P * dP))
* attention H = P v, S = s q k^T:  dv = P^T dH, dP = dH v^T,
      dq = s dS k, dk = s dS^T q
* linear   y = x W^T + b:  dW = dy^T x, db = sum_rows dy, dx = dy W
* SwiGLU   a = SiLU(g) * u:  dg = da * u * SiLU'(g), du = da * SiLU(g),
      SiLU'(g) = s(g) (1 + g (1 - s(g))), s the logistic function
* GELU     a = gelu(u):  du = da (Phi(u) + u phi(u))
Pinned in tests/test_backward_pins.py by central finite differences of the
oracle's own forward pass and by torch float64 autograd.
"""
from __future__ import annotations

import math

import numpy as np

from .compactor import (FFN_GELU, FFN_NONE, FFN_SWIGLU, _head_width, _scale, gelu, l2_normalize,
                        latent_positions, rms_norm, rope, silu, softmax_rows)


# ----------------------------------------------------------------------------
# Backward of the elementary steps
# ----------------------------------------------------------------------------

def rms_norm_backward(x: np.ndarray, dy: np.ndarray, eps: float) -> np.ndarray:
    D = x.shape[-1]
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return r * dy - (r ** 3 / D) * x * np.sum(x * dy, axis=-1, keepdims=True)


def l2_normalize_backward(x: np.ndarray, dy: np.ndarray, eps: float) -> np.ndarray:
    n = np.sqrt(np.sum(x * x, axis=-1, keepdims=True))
    nn = np.maximum(n, eps)
    y = x / nn
    # below eps the map is x / eps, a plain scaling
    return np.where(n > eps, (dy - y * np.sum(y * dy, axis=-1, keepdims=True)) / nn, dy / eps)


def rope_backward(dy: np.ndarray, positions, base: float) -> np.ndarray:
    """The adjoint of a rotation is the inverse rotation."""
    return rope(dy, positions, base, inverse=True)


def softmax_backward(P: np.ndarray, dP: np.ndarray) -> np.ndarray:
    return P * (dP - np.sum(P * dP, axis=-1, keepdims=True))


def silu_grad(g: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        s = 1.0 / (1.0 + np.exp(-g))
    return s * (1.0 + g * (1.0 - s))


def gelu_grad(u: np.ndarray) -> np.ndarray:
    erf = np.vectorize(math.erf, otypes=[np.float64])
    return 0.5 * (1.0 + erf(u / math.sqrt(2.0))) + u * np.exp(-0.5 * u * u) / math.sqrt(2.0 * math.pi)


def _add(grads: dict, name: str, g: np.ndarray):
    grads[name] = grads[name] + g if name in grads else g.copy()


# ----------------------------------------------------------------------------
# Sublayers: forward with the intermediates the backward needs, then backward
# ----------------------------------------------------------------------------

def _cross_forward(Q, X, p_q, p_k, w, cfg, b):
    nc, dc = cfg.n_cross_heads, _head_width(cfg, "cross")
    s = _scale(cfg, "cross")
    heads, cache = [], []
    for i in range(nc):
        rows = slice(i * dc, (i + 1) * dc)
        qt = Q @ w[f"b{b}.ca_wq"][rows].T + w[f"b{b}.ca_bq"][rows]
        kt = X @ w[f"b{b}.ca_wk"][rows].T + w[f"b{b}.ca_bk"][rows]
        v = X @ w[f"b{b}.ca_wv"][rows].T
        q = rope(l2_normalize(qt, cfg.l2_eps), p_q, cfg.compactor_rope_base)
        k = rope(l2_normalize(kt, cfg.l2_eps), p_k, cfg.compactor_rope_base)
        P = softmax_rows(s * (q @ k.T))
        heads.append(P @ v)
        cache.append((qt, kt, v, q, k, P))
    Hc = np.concatenate(heads, axis=-1)
    return Hc @ w[f"b{b}.ca_wo"].T, (Hc, cache)


def _cross_backward(dout, Q, X, p_q, p_k, w, cfg, b, saved, grads):
    """Returns dQ; adds the block's cross-attention parameter gradients."""
    nc, dc = cfg.n_cross_heads, _head_width(cfg, "cross")
    s = _scale(cfg, "cross")
    Hc, cache = saved
    _add(grads, f"b{b}.ca_wo", dout.T @ Hc)
    dH = dout @ w[f"b{b}.ca_wo"]
    dQ = np.zeros_like(Q)
    for i in range(nc):
        rows = slice(i * dc, (i + 1) * dc)
        qt, kt, v, q, k, P = cache[i]
        dHi = dH[:, rows]
        dv = P.T @ dHi
        dS = s * softmax_backward(P, dHi @ v.T)
        dq = dS @ k
        dk = dS.T @ q
        dqt = l2_normalize_backward(qt, rope_backward(dq, p_q, cfg.compactor_rope_base), cfg.l2_eps)
        dkt = l2_normalize_backward(kt, rope_backward(dk, p_k, cfg.compactor_rope_base), cfg.l2_eps)
        for name, dy, x in (("ca_wq", dqt, Q), ("ca_wk", dkt, X), ("ca_wv", dv, X)):
            full = grads.setdefault(f"b{b}.{name}", np.zeros_like(w[f"b{b}.{name}"]))
            full[rows] += dy.T @ x
        for name, dy in (("ca_bq", dqt), ("ca_bk", dkt)):
            full = grads.setdefault(f"b{b}.{name}", np.zeros_like(w[f"b{b}.{name}"]))
            full[rows] += dy.sum(axis=0)
        dQ += dqt @ w[f"b{b}.ca_wq"][rows]
    return dQ


def _self_forward(Y, w, cfg, b):
    ns, ds = cfg.n_self_heads, _head_width(cfg, "self")
    s = _scale(cfg, "self")
    heads, cache = [], []
    for i in range(ns):
        rows = slice(i * ds, (i + 1) * ds)
        qt = Y @ w[f"b{b}.sa_wq"][rows].T + w[f"b{b}.sa_bq"][rows]
        kt = Y @ w[f"b{b}.sa_wk"][rows].T + w[f"b{b}.sa_bk"][rows]
        v = Y @ w[f"b{b}.sa_wv"][rows].T
        q, k = l2_normalize(qt, cfg.l2_eps), l2_normalize(kt, cfg.l2_eps)
        P = softmax_rows(s * (q @ k.T))
        heads.append(P @ v)
        cache.append((qt, kt, v, q, k, P))
    Hc = np.concatenate(heads, axis=-1)
    return Hc @ w[f"b{b}.sa_wo"].T, (Hc, cache)


def _self_backward(dout, Y, w, cfg, b, saved, grads):
    ns, ds = cfg.n_self_heads, _head_width(cfg, "self")
    s = _scale(cfg, "self")
    Hc, cache = saved
    _add(grads, f"b{b}.sa_wo", dout.T @ Hc)
    dH = dout @ w[f"b{b}.sa_wo"]
    dY = np.zeros_like(Y)
    for i in range(ns):
        rows = slice(i * ds, (i + 1) * ds)
        qt, kt, v, q, k, P = cache[i]
        dHi = dH[:, rows]
        dv = P.T @ dHi
        dS = s * softmax_backward(P, dHi @ v.T)
        dqt = l2_normalize_backward(qt, dS @ k, cfg.l2_eps)
        dkt = l2_normalize_backward(kt, dS.T @ q, cfg.l2_eps)
        for name, dy in (("sa_wq", dqt), ("sa_wk", dkt), ("sa_wv", dv)):
            full = grads.setdefault(f"b{b}.{name}", np.zeros_like(w[f"b{b}.{name}"]))
            full[rows] += dy.T @ Y
        for name, dy in (("sa_bq", dqt), ("sa_bk", dkt)):
            full = grads.setdefault(f"b{b}.{name}", np.zeros_like(w[f"b{b}.{name}"]))
            full[rows] += dy.sum(axis=0)
        dY += dqt @ w[f"b{b}.sa_wq"][rows] + dkt @ w[f"b{b}.sa_wk"][rows] + dv @ w[f"b{b}.sa_wv"][rows]
    return dY


def _ffn_forward(Y, w, cfg, b):
    if cfg.ffn_kind == FFN_SWIGLU:
        g = Y @ w[f"b{b}.ffn_wg"].T
        u = Y @ w[f"b{b}.ffn_wu"].T
        a = silu(g) * u
        return a @ w[f"b{b}.ffn_wd"].T, (g, u, a)
    u = Y @ w[f"b{b}.ffn_wu"].T
    a = gelu(u)
    return a @ w[f"b{b}.ffn_wd"].T, (None, u, a)


def _ffn_backward(dout, Y, w, cfg, b, saved, grads):
    g, u, a = saved
    _add(grads, f"b{b}.ffn_wd", dout.T @ a)
    da = dout @ w[f"b{b}.ffn_wd"]
    if cfg.ffn_kind == FFN_SWIGLU:
        dg = da * u * silu_grad(g)
        du = da * silu(g)
        _add(grads, f"b{b}.ffn_wg", dg.T @ Y)
        _add(grads, f"b{b}.ffn_wu", du.T @ Y)
        return dg @ w[f"b{b}.ffn_wg"] + du @ w[f"b{b}.ffn_wu"]
    du = da * gelu_grad(u)
    _add(grads, f"b{b}.ffn_wu", du.T @ Y)
    return du @ w[f"b{b}.ffn_wu"]


# ----------------------------------------------------------------------------
# One layer
# ----------------------------------------------------------------------------

def compact_layer_backward(K: np.ndarray, V: np.ndarray, positions, rope_theta: float, w: dict, cfg, t: int,
                           dCk: np.ndarray, dCv: np.ndarray, rerotate: bool = True) -> dict:
    """Gradients of <dCk, C_k> + <dCv, C_v> w.r.t. every tensor of ``w``
    (same keys and shapes; float64).  K, V, positions, w as for
    compactor.compact_layer; dCk, dCv [H, t, d]."""
    H = K.shape[0]
    p_k = np.asarray(positions, dtype=np.float64)
    p_q = latent_positions(p_k, t)
    grads: dict = {}
    dlat = np.zeros_like(np.asarray(w["latents"], dtype=np.float64))
    for h in range(H):
        X = np.concatenate([rope(K[h], p_k, rope_theta, inverse=True), V[h]], axis=-1)
        Z = np.array(w["latents"][h], dtype=np.float64)
        tape = []
        for b in range(cfg.n_blocks):
            if cfg.n_cross_heads > 0 and (cfg.cross_every_block or b == 0):
                Q = rms_norm(Z, cfg.rms_eps)
                out, saved = _cross_forward(Q, X, p_q, p_k, w, cfg, b)
                tape.append(("cross", b, Z, Q, saved))
                Z = Z + out
            if cfg.n_self_heads > 0:
                Y = rms_norm(Z, cfg.rms_eps)
                out, saved = _self_forward(Y, w, cfg, b)
                tape.append(("self", b, Z, Y, saved))
                Z = Z + out
            if cfg.ffn_kind != FFN_NONE:
                Y = rms_norm(Z, cfg.rms_eps)
                out, saved = _ffn_forward(Y, w, cfg, b)
                tape.append(("ffn", b, Z, Y, saved))
                Z = Z + out
        Zo = rms_norm(Z, cfg.rms_eps) if cfg.final_norm else Z
        # output heads: C_k = R(p_q) (Zo W_key^T), C_v = Zo W_val^T
        dck = rope_backward(dCk[h], p_q, rope_theta) if rerotate else dCk[h]
        _add(grads, "w_key", dck.T @ Zo)
        _add(grads, "w_val", dCv[h].T @ Zo)
        dZo = dck @ w["w_key"] + dCv[h] @ w["w_val"]
        dZ = rms_norm_backward(Z, dZo, cfg.rms_eps) if cfg.final_norm else dZo
        for kind, b, Zin, Yin, saved in reversed(tape):
            if kind == "cross":
                dY = _cross_backward(dZ, Yin, X, p_q, p_k, w, cfg, b, saved, grads)
            elif kind == "self":
                dY = _self_backward(dZ, Yin, w, cfg, b, saved, grads)
            else:
                dY = _ffn_backward(dZ, Yin, w, cfg, b, saved, grads)
            dZ = dZ + rms_norm_backward(Zin, dY, cfg.rms_eps)
        dlat[h] = dZ
    grads["latents"] = dlat
    for k, v in w.items():   # tensors the forward pass does not use
        grads.setdefault(k, np.zeros_like(np.asarray(v, dtype=np.float64)))
    return grads
