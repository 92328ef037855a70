"""fp64 CPU oracle of the optional bias channel and of attention over a
compacted prefix.

TEST INFRASTRUCTURE ONLY.  Only tests, the smoke check and the benchmark's CPU
baseline leg may import this module.  It shares no code with the GPU library.

* Appendix A (output projections, optional beta shaping): a third linear head
  beta = Z_out w_beta on the final latent state (after the final RMSNorm when
  that is enabled); optional saturation beta_max * tanh(beta / beta_max) and
  optional mass matching, which adds log(T / t) (learnable variant: plus
  log x).  Appendix "Sweeping beta" scales the log term by a factor alpha.
* Appendix B (bias semantics in attention): a query attends over the compact
  prefix followed by the uncompacted suffix; the compact logits get beta
  added, the suffix entries get 0; one softmax over both parts.

Readings where the paper is silent:
* With both reparameterisations on, saturation is applied first and the
  mass-matching offset added after it (the offset is a prior outside the
  clipped learned part).
* Causal prefill over the suffix: query i of n_q sits at suffix index
  S - n_q + i and sees suffix entries up to and including that index; every
  compact entry is visible to every query (the compact prefix precedes the
  suffix in logical position).
* Grouped-query attention: query head j uses KV head j // group (the usual
  grouped layout, group query heads per KV head).
"""
from __future__ import annotations

import math

import numpy as np

from . import compactor


def beta_head(Zo: np.ndarray, w_beta: np.ndarray, beta_max: float = 0.0, mass_alpha: float = 0.0,
              log_x: float = 0.0, T: int = 1, t: int = 1) -> np.ndarray:
    """Appendix A: beta = Z_out w_beta, then the optional shaping.

    Zo: float64 [..., t, D] final latent state (already normed if the
    configuration normalises); w_beta: float64 [D].  Returns [..., t]."""
    b = np.asarray(Zo, dtype=np.float64) @ np.asarray(w_beta, dtype=np.float64)
    if beta_max > 0.0:                                  # saturation
        b = beta_max * np.tanh(b / beta_max)
    return b + (mass_alpha * math.log(T / t) + log_x)   # mass matching (0 when off)


def compact_layer_beta(K, V, positions, rope_theta: float, w: dict, cfg, t: int, w_beta,
                       beta_max: float = 0.0, mass_alpha: float = 0.0, log_x: float = 0.0,
                       rerotate: bool = True):
    """One layer's compaction plus the bias head: (C_k, C_v, out_positions, beta [H, t])."""
    tr: dict = {}
    Ck, Cv, pq = compactor.compact_layer(K, V, positions, rope_theta, w, cfg, t, rerotate=rerotate, trace=tr)
    beta = beta_head(np.stack(tr["Zo"]), w_beta, beta_max, mass_alpha, log_x, K.shape[1], t)
    return Ck, Cv, pq, beta


def attend(q: np.ndarray, Ck: np.ndarray, Cv: np.ndarray, beta, K: np.ndarray, V: np.ndarray,
           group: int = 1, causal: bool = False, scale: float | None = None,
           q_positions=None, rope_theta: float | None = None) -> np.ndarray:
    """Appendix B: Attn(q; [C_k; K_fix], [C_v; V_fix], [beta; 0]).

    q: [H*group, n_q, d]; Ck, Cv: [H, t, d]; beta: [H, t] or None (zeros);
    K, V: [H, S, d].  With q_positions ([n_q], logical positions: physical
    position plus the compacted cache's offset T - physical prefix length,
    Appendix B "logical vs physical cache length") the queries are first
    rotated by the base model's RoPE there.  Returns [H*group, n_q, d] in
    float64."""
    q = np.asarray(q, dtype=np.float64)
    if q_positions is not None:
        q = np.stack([compactor.rope(qh, np.asarray(q_positions, np.float64), rope_theta) for qh in q])
    Hq, nq, d = q.shape
    H, t = Ck.shape[0], Ck.shape[1]
    S = K.shape[1]
    assert Hq == H * group
    s = (1.0 / math.sqrt(d)) if not scale else float(scale)
    out = np.empty_like(q)
    for hq in range(Hq):
        h = hq // group
        keys = np.concatenate([Ck[h], K[h]], axis=0)                       # [t + S, d]
        vals = np.concatenate([Cv[h], V[h]], axis=0)
        bias = np.concatenate([np.zeros(t) if beta is None else np.asarray(beta[h], np.float64),
                               np.zeros(S)])                               # [beta; 0]
        for i in range(nq):
            logit = s * (keys @ q[hq, i]) + bias
            if causal:
                logit[t + (S - nq + i) + 1:] = -np.inf                     # later suffix entries
            e = np.exp(logit - logit.max())
            out[hq, i] = (e @ vals) / e.sum()
    return out
