"""fp64 CPU oracle of the Still per-layer compactor forward pass.

TEST INFRASTRUCTURE ONLY.  Only tests, the smoke check and the benchmark's CPU
baseline leg may import this module.  It shares no code with the GPU library
and imports nothing from it; it follows the paper's definitions literally, in
float64, with numpy matmuls as the only library primitive:

* Section 2 (problem statement): g maps per-KV-head (K, V) in R^{T x d} to
  (C_k, C_v) in R^{t x d}.
* Section 2.2 and Appendix B (single-pass recipe): keys are un-rotated into a
  position-free frame, X = [K; V], the compactor runs, compact keys are
  re-rotated at evenly spaced output positions over the compacted range.
* Appendix A (architecture): pre-norm blocks
      Z'   = Z  + CrossAttn(RMSNorm(Z), X)
      Z''  = Z' + SelfAttn(RMSNorm(Z'))
      Z''' = Z''+ FFN(RMSNorm(Z''))
  with the expanded-head convention (each of n_c heads has width d_l),
  q~ = Q W_Q + b_Q, k~ = X W_K + b_K, v = X W_V (no bias), L2 QK-norm, the
  compactor's own RoPE on normalised q/k (latent positions evenly spaced
  between the first and last key positions), logits scaled by d_l,
  head = softmax(d_l q k^T) v, Concat(heads) W_O.  Self-attention: same
  QK-norm and scale, no RoPE.  Output heads C_k = Z_out W_key,
  C_v = Z_out W_val.

Storage convention of weights (the inputs this oracle receives): a projection
written x W with W in R^{in x out} in the paper is stored as the [out][in]
matrix W^T (torch.nn.Linear layout); the oracle therefore evaluates x @ w.T.

Readings where the paper is silent (each is also exercised by a pin test):
* RoPE pairs dimension j with j + w/2 ("rotate-half") and uses angular
  frequency base^(-2j/w) for j < w/2, for both the base model's RoPE and the
  compactor's internal RoPE.
* "first and last supplied key positions" is read as min and max of the
  positions; latent / output positions are fractional (no rounding),
  p_i = p_min + i (p_max - p_min)/(t-1), and p_0 = p_min when t = 1.
* RMSNorm(x) = x / sqrt(mean(x^2) + eps), eps = 1e-6, no gain;
  Norm_L2(x) = x / max(||x||, 1e-12).
* Self-attention mixes the t latents of one KV head's bank (not across
  heads); its q and k projections carry biases like cross-attention's; no
  bias on value, output, FFN or output-head projections.
* FFN: SwiGLU, (SiLU(x W_g) * (x W_u)) W_d, as the benchmark workloads
  specify; the paper's two-layer GELU MLP (exact erf GELU) is the other kind.
* Optional final RMSNorm before the heads is off unless the config sets it.

Every function below is pinned in tests/test_oracle_pins.py; the full-layer
composition is pinned by the identity-style initialisation of Appendix C and
by an independent pure-Python loop evaluation on tiny inputs.
"""
from __future__ import annotations

import math

import numpy as np

FFN_NONE, FFN_SWIGLU, FFN_GELU = 0, 1, 2


# ----------------------------------------------------------------------------
# Elementary operations
# ----------------------------------------------------------------------------

def rope_angles(positions, base: float, width: int) -> np.ndarray:
    """phi[n, j] = p_n * base^(-2j/width), j < width/2 (Section 2.2, Appendix A)."""
    j = np.arange(width // 2, dtype=np.float64)
    inv_freq = np.power(float(base), -2.0 * j / width)
    return np.multiply.outer(np.asarray(positions, dtype=np.float64), inv_freq)


def rope(x: np.ndarray, positions, base: float, inverse: bool = False) -> np.ndarray:
    """Rotary embedding over the last axis: rotate pair (x_j, x_{j+w/2}) by +phi
    (or -phi when ``inverse``, the RoPE-fix un-rotation of Section 2.2)."""
    w = x.shape[-1]
    phi = rope_angles(positions, base, w)
    if inverse:
        phi = -phi
    c, s = np.cos(phi), np.sin(phi)
    a, b = x[..., : w // 2], x[..., w // 2:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def rms_norm(x: np.ndarray, eps: float) -> np.ndarray:
    """Non-parametric RMSNorm (Appendix A, compactor blocks)."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def l2_normalize(x: np.ndarray, eps: float) -> np.ndarray:
    """QK-norm: x / max(||x||_2, eps) (Appendix A, cross-attention)."""
    return x / np.maximum(np.sqrt(np.sum(x * x, axis=-1, keepdims=True)), eps)


def softmax_rows(S: np.ndarray) -> np.ndarray:
    e = np.exp(S - S.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def silu(x: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        return x / (1.0 + np.exp(-x))


def gelu(x: np.ndarray) -> np.ndarray:
    erf = np.vectorize(math.erf, otypes=[np.float64])
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def latent_positions(positions, t: int) -> np.ndarray:
    """Evenly spaced positions over [min p, max p] (Appendix A; Appendix B step 5)."""
    p = np.asarray(positions, dtype=np.float64)
    lo, hi = float(p.min()), float(p.max())
    if t == 1:
        return np.array([lo])
    return lo + np.arange(t, dtype=np.float64) * ((hi - lo) / (t - 1))


# ----------------------------------------------------------------------------
# Sublayers (one KV head's latent bank)
# ----------------------------------------------------------------------------

def _head_width(cfg, kind: str) -> int:
    w = cfg.cross_head_dim if kind == "cross" else cfg.self_head_dim
    return w or cfg.latent_dim


def _scale(cfg, kind: str) -> float:
    s = cfg.logit_scale_cross if kind == "cross" else cfg.logit_scale_self
    return float(s) if s else float(_head_width(cfg, kind))


def cross_attention(Q: np.ndarray, X: np.ndarray, p_q, p_k, w: dict, cfg, block: int,
                    trace: dict | None = None) -> np.ndarray:
    """CrossAttn(Q, X) = Concat(head_1..head_nc) W_O (Appendix A).

    Q = RMSNorm(Z) in R^{t x d_l} (one KV head), X = [K_free; V] in R^{T x 2d}.
    """
    nc, dc = cfg.n_cross_heads, _head_width(cfg, "cross")
    s = _scale(cfg, "cross")
    wq, bq = w[f"b{block}.ca_wq"], w[f"b{block}.ca_bq"]
    wk, bk = w[f"b{block}.ca_wk"], w[f"b{block}.ca_bk"]
    wv, wo = w[f"b{block}.ca_wv"], w[f"b{block}.ca_wo"]
    heads = []
    for i in range(nc):
        rows = slice(i * dc, (i + 1) * dc)
        q_t = Q @ wq[rows].T + bq[rows]            # q~_i = Q W_Qi + b_Qi
        k_t = X @ wk[rows].T + bk[rows]            # k~_i = X W_Ki + b_Ki
        v = X @ wv[rows].T                         # v_i  = X W_Vi
        q = rope(l2_normalize(q_t, cfg.l2_eps), p_q, cfg.compactor_rope_base)
        k = rope(l2_normalize(k_t, cfg.l2_eps), p_k, cfg.compactor_rope_base)
        P = softmax_rows(s * (q @ k.T))
        heads.append(P @ v)
    H = np.concatenate(heads, axis=-1)
    if trace is not None:
        trace.setdefault("ca_heads", []).append(H)
    return H @ wo.T


def self_attention(Y: np.ndarray, w: dict, cfg, block: int) -> np.ndarray:
    """SelfAttn(Y) = Concat(head_1..head_ns) W_O^(sa); QK-norm, d_l scale, no RoPE."""
    ns, ds = cfg.n_self_heads, _head_width(cfg, "self")
    s = _scale(cfg, "self")
    wq, bq = w[f"b{block}.sa_wq"], w[f"b{block}.sa_bq"]
    wk, bk = w[f"b{block}.sa_wk"], w[f"b{block}.sa_bk"]
    wv, wo = w[f"b{block}.sa_wv"], w[f"b{block}.sa_wo"]
    heads = []
    for i in range(ns):
        rows = slice(i * ds, (i + 1) * ds)
        q = l2_normalize(Y @ wq[rows].T + bq[rows], cfg.l2_eps)
        k = l2_normalize(Y @ wk[rows].T + bk[rows], cfg.l2_eps)
        v = Y @ wv[rows].T
        heads.append(softmax_rows(s * (q @ k.T)) @ v)
    return np.concatenate(heads, axis=-1) @ wo.T


def ffn(Y: np.ndarray, w: dict, cfg, block: int) -> np.ndarray:
    if cfg.ffn_kind == FFN_SWIGLU:
        return (silu(Y @ w[f"b{block}.ffn_wg"].T) * (Y @ w[f"b{block}.ffn_wu"].T)) @ w[f"b{block}.ffn_wd"].T
    if cfg.ffn_kind == FFN_GELU:
        return gelu(Y @ w[f"b{block}.ffn_wu"].T) @ w[f"b{block}.ffn_wd"].T
    raise ValueError("no FFN")


# ----------------------------------------------------------------------------
# One layer
# ----------------------------------------------------------------------------

def compact_layer(K: np.ndarray, V: np.ndarray, positions, rope_theta: float, w: dict, cfg,
                  t: int, rerotate: bool = True, heads=None, trace: dict | None = None):
    """Compact one layer's cache.

    K, V: float64 [H, N, d] (RoPE'd keys, values); positions: float64 [N];
    w: float64 weights keyed like the layer's tensor list ([out][in] matrices).
    Returns (C_k [H,t,d], C_v [H,t,d], out_positions [t]).  ``heads`` restricts
    the evaluation to a subset of KV heads (outputs hold only those heads).
    """
    H, N, d = K.shape
    assert w["latents"].shape[1] == t, "latent bank size must equal t"
    p_k = np.asarray(positions, dtype=np.float64)
    p_q = latent_positions(p_k, t)
    hs = range(H) if heads is None else heads
    Ck, Cv = [], []
    for h in hs:
        # Section 2.2 / Appendix B step 3-4: un-rotate keys, X = [K; V].
        X = np.concatenate([rope(K[h], p_k, rope_theta, inverse=True), V[h]], axis=-1)
        Z = np.array(w["latents"][h], dtype=np.float64)
        for b in range(cfg.n_blocks):
            if cfg.n_cross_heads > 0 and (cfg.cross_every_block or b == 0):
                Z = Z + cross_attention(rms_norm(Z, cfg.rms_eps), X, p_q, p_k, w, cfg, b, trace)
            if trace is not None:
                trace.setdefault("Z1", []).append(Z.copy())
            if cfg.n_self_heads > 0:
                Z = Z + self_attention(rms_norm(Z, cfg.rms_eps), w, cfg, b)
            if trace is not None:
                trace.setdefault("Z2", []).append(Z.copy())
            if cfg.ffn_kind != FFN_NONE:
                Z = Z + ffn(rms_norm(Z, cfg.rms_eps), w, cfg, b)
            if trace is not None:
                trace.setdefault("Z3", []).append(Z.copy())
        Zo = rms_norm(Z, cfg.rms_eps) if cfg.final_norm else Z
        if trace is not None:
            trace.setdefault("Zo", []).append(Zo.copy())
        ck = Zo @ w["w_key"].T                    # C_k = Z_out W_key
        cv = Zo @ w["w_val"].T                    # C_v = Z_out W_val
        if rerotate:                              # Appendix B step 5
            ck = rope(ck, p_q, rope_theta)
        Ck.append(ck)
        Cv.append(cv)
    return np.stack(Ck), np.stack(Cv), p_q


# ----------------------------------------------------------------------------
# Compositions around one compaction call (Appendix B)
# ----------------------------------------------------------------------------

def compact_subrange(K: np.ndarray, V: np.ndarray, positions, rope_theta: float, w: dict, cfg, t: int,
                     start: int, end: int, rerotate: bool = True):
    """Appendix B recipe with a selected subrange [start, end): only those
    entries are compacted (to t); the preserved prefix [0, start) and suffix
    [end, N) are spliced back unchanged around the compact entries, which sit
    at the evenly spaced output positions of the compacted range.

    Returns (K', V', positions') with N - (end - start) + t entries.
    """
    N = K.shape[1]
    assert 0 <= start < end <= N
    p = np.asarray(positions, dtype=np.float64)
    Ck, Cv, pq = compact_layer(K[:, start:end], V[:, start:end], p[start:end], rope_theta, w, cfg, t,
                               rerotate=rerotate)
    return (np.concatenate([K[:, :start], Ck, K[:, end:]], axis=1),
            np.concatenate([V[:, :start], Cv, V[:, end:]], axis=1),
            np.concatenate([p[:start], pq, p[end:]]))


def compact_chunks(K: np.ndarray, V: np.ndarray, positions, rope_theta: float, w: dict, cfg, t: int,
                   chunk: int, rerotate: bool = True):
    """Appendix B independent chunk compaction: the range is split into
    consecutive chunks of `chunk` entries (the last one may be shorter), each
    compacted to t entries on its own, and the compact chunks concatenated."""
    N = K.shape[1]
    assert chunk >= 1
    p = np.asarray(positions, dtype=np.float64)
    outs = [compact_layer(K[:, a:a + chunk], V[:, a:a + chunk], p[a:a + chunk], rope_theta, w, cfg, t,
                          rerotate=rerotate) for a in range(0, N, chunk)]
    return (np.concatenate([o[0] for o in outs], axis=1), np.concatenate([o[1] for o in outs], axis=1),
            np.concatenate([o[2] for o in outs]))
