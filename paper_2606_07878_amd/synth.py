"""Seeded synthetic inputs: KV caches and compactor weights.

This module only *draws* inputs; it contains none of the compactor's
arithmetic.  It stands in for the frozen base model's prefill (Section 2,
first paragraph): per-layer caches K, V in R^{H x N x d} whose keys carry the
base model's rotary embedding at their cache positions, with value
distributions chosen to resemble real caches (unit-Gaussian entries plus a few
large "outlier" key channels per head).  Compactor weights are random
N(0, 0.02) draws, since the paper's trained checkpoints are not available.

Every tensor is rounded to bfloat16 (round-to-nearest-even) once, here, so the
oracle and the GPU path receive identical bits.

Random streams: numpy PCG64 seeded by SeedSequence([seed, layer, stream]);
stream 0 = position-free keys, 1 = values, 2 = outlier channel choice,
3 = weights (fixed enumeration order: latents, block tensors in
``configs.BLOCK_TENSORS`` order, then w_key, w_val), 4 = the bias head's
w_beta, 5 = consumer-attention operands (queries, compact entries, biases,
suffix), 10+r = fresh tokens of iterative round r.
"""
from __future__ import annotations

import numpy as np

from .configs import BLOCK_TENSORS, Workload, block_shapes

WEIGHT_STD = 0.02


def _rng(seed: int, layer: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, layer, stream])))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round to bfloat16 (RNE via float32) and return the raw uint16 bit patterns."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_value(bits: np.ndarray) -> np.ndarray:
    """Exact float64 value of bfloat16 bit patterns."""
    u = bits.astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def base_rope_rotate(k_free: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """The base model's rotary embedding (rotate-half pairs (j, j + d/2)).

    Input synthesis only: plays the role of the base model writing RoPE'd keys
    into its cache at the given positions.
    """
    d = k_free.shape[-1]
    half = d // 2
    inv = np.power(float(theta), -np.arange(0, d, 2, dtype=np.float64) / d)
    ang = np.multiply.outer(np.asarray(positions, dtype=np.float64), inv)   # [N, half]
    c, s = np.cos(ang), np.sin(ang)
    a, b = k_free[..., :half], k_free[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def make_cache(w: Workload, layer: int, n_tokens: int | None = None,
               positions: np.ndarray | None = None, keep_free: bool = False) -> dict:
    """Synthetic RoPE'd cache for one layer.

    Returns dict(K=uint16 bf16 bits [H,N,d], V=..., positions=float64 [N]) and,
    with keep_free, the float64 position-free keys before rotation/rounding.
    """
    cfg = w.cfg
    H, d = cfg.n_kv_heads, cfg.head_dim
    N = n_tokens if n_tokens is not None else w.n_tokens
    if positions is None:
        positions = np.arange(N, dtype=np.float64)
    k_free = _rng(w.seed, layer, 0).standard_normal((H, N, d))
    if w.outlier_channels:
        r2 = _rng(w.seed, layer, 2)
        for h in range(H):
            ch = r2.choice(d, w.outlier_channels, replace=False)
            k_free[h][:, ch] *= w.outlier_scale
    K = bf16_bits(base_rope_rotate(k_free, positions, w.rope_theta))
    V = bf16_bits(_rng(w.seed, layer, 1).standard_normal((H, N, d)))
    out = dict(K=K, V=V, positions=np.asarray(positions, dtype=np.float64))
    if keep_free:
        out["k_free"] = k_free
    return out


def make_fresh_tokens(w: Workload, layer: int, rnd: int, start_pos: float) -> dict:
    """Fresh tokens appended before iterative round ``rnd`` (1-based)."""
    cfg = w.cfg
    H, d, n = cfg.n_kv_heads, cfg.head_dim, w.fresh_tokens
    pos = start_pos + np.arange(n, dtype=np.float64)
    r = _rng(w.seed, layer, 10 + rnd)
    k_free = r.standard_normal((H, n, d))
    v = r.standard_normal((H, n, d))
    return dict(K=bf16_bits(base_rope_rotate(k_free, pos, w.rope_theta)),
                V=bf16_bits(v), positions=pos)


def make_weights(w: Workload, layer: int, t: int | None = None) -> dict:
    """Random compactor weights (bf16 bits), keyed like ``configs.layer_shapes``."""
    cfg = w.cfg
    t = t if t is not None else w.t
    r = _rng(w.seed, layer, 3)
    out = {"latents": bf16_bits(r.normal(0.0, WEIGHT_STD, (cfg.n_kv_heads, t, cfg.latent_dim)))}
    for b in range(cfg.n_blocks):
        shapes = block_shapes(cfg, b)
        for name in BLOCK_TENSORS:
            if name in shapes:
                out[f"b{b}.{name}"] = bf16_bits(r.normal(0.0, WEIGHT_STD, shapes[name]))
    out["w_key"] = bf16_bits(r.normal(0.0, WEIGHT_STD, (cfg.head_dim, cfg.latent_dim)))
    out["w_val"] = bf16_bits(r.normal(0.0, WEIGHT_STD, (cfg.head_dim, cfg.latent_dim)))
    return out


def make_beta_weight(w: Workload, layer: int) -> np.ndarray:
    """w_beta [latent_dim] of the optional bias head (bf16 bits).  Drawn with
    std 1/sqrt(latent_dim) so that beta = Z_out w_beta is O(1) on unit-RMS
    latent states and the bias visibly moves attention."""
    D = w.cfg.latent_dim
    return bf16_bits(_rng(w.seed, layer, 4).normal(0.0, 1.0 / np.sqrt(D), D))


def make_attend_inputs(seed: int, H: int, group: int, n_q: int, t: int, S: int, d: int,
                       beta: bool = True) -> dict:
    """Operands of attention over [C_k; K] with bias [beta; 0] (bf16 bits,
    beta float32): q [H*group, n_q, d], C_k / C_v [H, t, d], beta [H, t],
    K / V [H, S, d].  Unit-Gaussian entries (logits q.k/sqrt(d) ~ N(0, 1));
    beta ~ N(0, 1)."""
    r = _rng(seed, 0, 5)
    out = dict(q=bf16_bits(r.standard_normal((H * group, n_q, d))),
               C_k=bf16_bits(r.standard_normal((H, t, d))), C_v=bf16_bits(r.standard_normal((H, t, d))),
               K=bf16_bits(r.standard_normal((H, S, d))), V=bf16_bits(r.standard_normal((H, S, d))))
    out["beta"] = r.standard_normal((H, t)).astype(np.float32) if beta else None
    return out


def as_f64(d: dict) -> dict:
    """float64 views of every uint16 (bf16) entry; other entries passed through."""
    return {k: (bf16_value(v) if isinstance(v, np.ndarray) and v.dtype == np.uint16 else v)
            for k, v in d.items()}


# ----------------------------------------------------------------------------
# On-device generator for benchmark-sized stacks (same recipe, torch Philox
# streams instead of numpy PCG64, so values differ from the numpy generator).
# ----------------------------------------------------------------------------

def _tgen(device, seed: int, layer: int, stream: int):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1_000_003 + layer) * 101 + stream)
    return g


def make_layer_torch(w: Workload, layer: int, device, dtype=None, n_tokens: int | None = None,
                     positions=None, weights: bool = True):
    """(K, V, positions, weights) for one layer as device tensors (bf16 by default);
    weights is None when not requested (fresh tokens of an iterative round)."""
    import torch
    dtype = dtype or torch.bfloat16
    cfg = w.cfg
    H, d = cfg.n_kv_heads, cfg.head_dim
    N = n_tokens if n_tokens is not None else w.n_tokens
    if positions is None:
        positions = torch.arange(N, dtype=torch.float64, device=device)
    k_free = torch.randn(H, N, d, generator=_tgen(device, w.seed, layer, 0), device=device, dtype=torch.float32)
    if w.outlier_channels:
        g2 = _tgen(device, w.seed, layer, 2)
        for h in range(H):
            ch = torch.randperm(d, generator=g2, device=device)[: w.outlier_channels]
            k_free[h][:, ch] *= w.outlier_scale
    half = d // 2
    inv = torch.pow(torch.tensor(float(w.rope_theta), dtype=torch.float64, device=device),
                    -torch.arange(0, d, 2, dtype=torch.float64, device=device) / d)
    ang = positions[:, None] * inv[None, :]
    c, s = torch.cos(ang).float(), torch.sin(ang).float()
    a, b = k_free[..., :half], k_free[..., half:]
    K = torch.cat([a * c - b * s, b * c + a * s], dim=-1).to(dtype)
    V = torch.randn(H, N, d, generator=_tgen(device, w.seed, layer, 1), device=device).to(dtype)
    if not weights:
        return K, V, positions, None
    g3 = _tgen(device, w.seed, layer, 3)
    from .configs import layer_shapes
    W = {k: (torch.randn(*shape, generator=g3, device=device) * WEIGHT_STD).to(dtype)
         for k, shape in layer_shapes(cfg, w.t).items()}
    return K, V, positions, W
