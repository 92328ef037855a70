"""Pins of the fp64 oracle backward (oracle/backward.py), CPU only.

* Central finite differences of the oracle's own forward pass
  (oracle/compactor.py): for every compactor tensor and a random direction u,
  (L(phi + e u) - L(phi - e u)) / 2e must equal <grad, u>, with
  L = <dC_k, C_k> + <dC_v, C_v>.  This uses nothing of the backward code.
* torch float64 autograd through a forward pass written here with torch
  operations (checked equal to the oracle's forward first).
* Planted mistakes in the backward steps each break the finite-difference pin.
"""
import math

import numpy as np
import pytest
import torch

from oracle import backward as B
from oracle import compactor as O
from paper_2606_07878_amd import configs

RNG = np.random.default_rng(77)


def tiny_cfg(**kw):
    base = dict(n_kv_heads=2, head_dim=4, latent_dim=8, n_blocks=1, n_cross_heads=2, n_self_heads=2,
                ffn_kind=configs.FFN_SWIGLU, ffn_hidden=6)
    base.update(kw)
    return configs.CompactorConfig(**base)


VARIANTS = {
    "swiglu": dict(),
    "gelu_final_norm": dict(ffn_kind=configs.FFN_GELU, final_norm=1),
    "two_blocks": dict(n_blocks=2),
    "resampler": dict(n_blocks=2, cross_every_block=0),
    "no_self_no_ffn": dict(n_self_heads=0, ffn_kind=configs.FFN_NONE, ffn_hidden=0),
    "inv_sqrt_scale": dict(logit_scale_cross=1 / math.sqrt(8), logit_scale_self=1 / math.sqrt(8)),
}


def problem(cfg, N=7, t=3, rng=RNG, theta=1e4):
    shapes = configs.layer_shapes(cfg, t)
    w = {k: rng.normal(0, 0.5, s) for k, s in shapes.items()}
    H, d = cfg.n_kv_heads, cfg.head_dim
    pos = np.sort(rng.uniform(0, 50, N))
    K = O.rope(rng.normal(size=(H, N, d)), pos, theta)
    V = rng.normal(size=(H, N, d))
    dCk, dCv = rng.normal(size=(H, t, d)), rng.normal(size=(H, t, d))
    return K, V, pos, theta, w, t, dCk, dCv


def loss(K, V, pos, theta, w, cfg, t, dCk, dCv, rerotate=True):
    Ck, Cv, _ = O.compact_layer(K, V, pos, theta, w, cfg, t, rerotate=rerotate)
    return float(np.sum(dCk * Ck) + np.sum(dCv * Cv))


def fd_check(cfg, rerotate=True, t=3, rtol=2e-6, grads_fn=None):
    K, V, pos, theta, w, t, dCk, dCv = problem(cfg, t=t)
    grads = (grads_fn or B.compact_layer_backward)(K, V, pos, theta, w, cfg, t, dCk, dCv, rerotate=rerotate)
    assert set(grads) == set(w)
    worst = 0.0
    for name in w:
        u = RNG.normal(size=w[name].shape)
        eps = 1e-5
        wp = {**w, name: w[name] + eps * u}
        wm = {**w, name: w[name] - eps * u}
        fd = (loss(K, V, pos, theta, wp, cfg, t, dCk, dCv, rerotate)
              - loss(K, V, pos, theta, wm, cfg, t, dCk, dCv, rerotate)) / (2 * eps)
        an = float(np.sum(grads[name] * u))
        scale = max(abs(fd), abs(an), 1e-3)
        err = abs(fd - an) / scale
        worst = max(worst, err)
        assert err < rtol, f"{name}: finite difference {fd:.10g} vs gradient {an:.10g}"
    return worst


@pytest.mark.parametrize("variant", sorted(VARIANTS))
def test_backward_matches_finite_differences(variant):
    fd_check(tiny_cfg(**VARIANTS[variant]))


def test_backward_finite_differences_no_rerotate_single_latent():
    fd_check(tiny_cfg(), rerotate=False, t=1)


# ----------------------------------------------------------------------------
# torch float64 autograd through an independently written forward pass
# ----------------------------------------------------------------------------

def _t_rope(x, pos, base, inverse=False):
    w = x.shape[-1]
    j = torch.arange(w // 2, dtype=torch.float64)
    phi = torch.as_tensor(pos, dtype=torch.float64)[:, None] * torch.pow(torch.tensor(float(base), dtype=torch.float64),
                                                                          -2.0 * j / w)[None, :]
    if inverse:
        phi = -phi
    c, s = torch.cos(phi), torch.sin(phi)
    a, b = x[..., : w // 2], x[..., w // 2:]
    return torch.cat([a * c - b * s, b * c + a * s], dim=-1)


def _t_layer(K, V, pos, theta, w, cfg, t, rerotate=True):
    F = torch.nn.functional
    p = torch.as_tensor(pos, dtype=torch.float64)
    lo, hi = float(p.min()), float(p.max())
    pq = torch.tensor([lo]) if t == 1 else lo + torch.arange(t, dtype=torch.float64) * ((hi - lo) / (t - 1))
    rms = lambda x: F.rms_norm(x, (x.shape[-1],), eps=cfg.rms_eps)  # noqa: E731
    l2n = lambda x: x / torch.clamp(torch.linalg.vector_norm(x, dim=-1, keepdim=True), min=cfg.l2_eps)  # noqa: E731
    outs_k, outs_v = [], []
    for h in range(K.shape[0]):
        X = torch.cat([_t_rope(K[h], p, theta, inverse=True), V[h]], dim=-1)
        Z = w["latents"][h]
        for b in range(cfg.n_blocks):
            if cfg.cross_every_block or b == 0:
                Q = rms(Z)
                dc = cfg.dc
                hs = []
                for i in range(cfg.n_cross_heads):
                    r = slice(i * dc, (i + 1) * dc)
                    q = _t_rope(l2n(F.linear(Q, w[f"b{b}.ca_wq"][r], w[f"b{b}.ca_bq"][r])), pq, cfg.compactor_rope_base)
                    k = _t_rope(l2n(F.linear(X, w[f"b{b}.ca_wk"][r], w[f"b{b}.ca_bk"][r])), p, cfg.compactor_rope_base)
                    v = F.linear(X, w[f"b{b}.ca_wv"][r])
                    hs.append(torch.softmax(cfg.scale_cross * q @ k.T, dim=-1) @ v)
                Z = Z + F.linear(torch.cat(hs, -1), w[f"b{b}.ca_wo"])
            if cfg.n_self_heads:
                Y = rms(Z)
                ds = cfg.ds
                hs = []
                for i in range(cfg.n_self_heads):
                    r = slice(i * ds, (i + 1) * ds)
                    q = l2n(F.linear(Y, w[f"b{b}.sa_wq"][r], w[f"b{b}.sa_bq"][r]))
                    k = l2n(F.linear(Y, w[f"b{b}.sa_wk"][r], w[f"b{b}.sa_bk"][r]))
                    hs.append(torch.softmax(cfg.scale_self * q @ k.T, dim=-1) @ F.linear(Y, w[f"b{b}.sa_wv"][r]))
                Z = Z + F.linear(torch.cat(hs, -1), w[f"b{b}.sa_wo"])
            if cfg.ffn_kind == configs.FFN_SWIGLU:
                Y = rms(Z)
                Z = Z + F.linear(F.silu(F.linear(Y, w[f"b{b}.ffn_wg"])) * F.linear(Y, w[f"b{b}.ffn_wu"]),
                                 w[f"b{b}.ffn_wd"])
            elif cfg.ffn_kind == configs.FFN_GELU:
                Y = rms(Z)
                Z = Z + F.linear(F.gelu(F.linear(Y, w[f"b{b}.ffn_wu"])), w[f"b{b}.ffn_wd"])
        Zo = rms(Z) if cfg.final_norm else Z
        ck = F.linear(Zo, w["w_key"])
        outs_k.append(_t_rope(ck, pq, theta) if rerotate else ck)
        outs_v.append(F.linear(Zo, w["w_val"]))
    return torch.stack(outs_k), torch.stack(outs_v)


@pytest.mark.parametrize("variant", sorted(VARIANTS))
def test_backward_matches_torch_autograd(variant):
    cfg = tiny_cfg(**VARIANTS[variant])
    K, V, pos, theta, w, t, dCk, dCv = problem(cfg)
    tw = {k: torch.tensor(v, requires_grad=True) for k, v in w.items()}
    Ck, Cv = _t_layer(torch.tensor(K), torch.tensor(V), pos, theta, tw, cfg, t)
    rk, rv, _ = O.compact_layer(K, V, pos, theta, w, cfg, t)
    np.testing.assert_allclose(Ck.detach().numpy(), rk, rtol=1e-11, atol=1e-12)   # same forward
    np.testing.assert_allclose(Cv.detach().numpy(), rv, rtol=1e-11, atol=1e-12)
    L = (Ck * torch.tensor(dCk)).sum() + (Cv * torch.tensor(dCv)).sum()
    L.backward()
    grads = B.compact_layer_backward(K, V, pos, theta, w, cfg, t, dCk, dCv)
    for name, tv in tw.items():
        ref = tv.grad.numpy() if tv.grad is not None else np.zeros_like(w[name])
        np.testing.assert_allclose(grads[name], ref, rtol=1e-9, atol=1e-11 * max(1.0, np.abs(ref).max()),
                                   err_msg=name)


# ----------------------------------------------------------------------------
# Planted mistakes in the backward steps must break the finite-difference pin
# ----------------------------------------------------------------------------

MUTATIONS = {
    "rms_drops_projection": ("rms_norm_backward",
                             lambda x, dy, eps: dy / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)),
    "l2n_drops_projection": ("l2_normalize_backward",
                             lambda x, dy, eps: dy / np.sqrt(np.sum(x * x, axis=-1, keepdims=True))),
    "rope_wrong_direction": ("rope_backward", lambda dy, pos, base: O.rope(dy, pos, base)),
    "softmax_drops_rowsum": ("softmax_backward", lambda P, dP: P * dP),
    "silu_grad_drops_term": ("silu_grad", lambda g: 1.0 / (1.0 + np.exp(-g))),
    "gelu_grad_drops_term": ("gelu_grad", lambda u: 0.5 * (1.0 + np.vectorize(math.erf)(u / math.sqrt(2.0)))),
}


@pytest.mark.parametrize("mutation", sorted(MUTATIONS))
def test_planted_backward_mistakes_are_caught(mutation, monkeypatch):
    fn, bad = MUTATIONS[mutation]
    monkeypatch.setattr(B, fn, bad)
    cfg = tiny_cfg(ffn_kind=configs.FFN_GELU) if "gelu" in mutation else tiny_cfg()
    with pytest.raises(AssertionError):
        fd_check(cfg)
