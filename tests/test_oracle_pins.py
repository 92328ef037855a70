"""Pins of the fp64 oracle against facts other than itself.

* the rotary embedding against complex multiplication z e^{i phi} (a different
  formulation) and against the synthetic cache generator's forward rotation;
* rotation identities (inverse, norm, relative-position property);
* elementwise operations against torch's float64 library routines;
* attention special cases with closed forms (one key, identical keys);
* invariances (joint permutation of cache tokens, scale of W_K/W_Q);
* the identity-style initialisation of Appendix C at t = T (the paper's only
  end-to-end closed form: compact cache == original cache);
* an independent pure-Python loop evaluation of a whole layer on tiny inputs;
* Appendix D's parameter count and Appendix B's KV-size figures as printed
  (fixtures under tests/golden, each citing where the paper gives it).
"""
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import compactor as O
from oracle import sizing
from paper_2606_07878_amd import configs, synth

RNG = np.random.default_rng(1234)


def tiny_cfg(**kw):
    base = dict(n_kv_heads=2, head_dim=4, latent_dim=8, n_blocks=1, n_cross_heads=2,
                n_self_heads=2, ffn_kind=configs.FFN_SWIGLU, ffn_hidden=6)
    base.update(kw)
    return configs.CompactorConfig(**base)


def rand_weights(cfg, t, std=0.5, rng=RNG):
    shapes = configs.layer_shapes(cfg, t)
    return {k: rng.normal(0, std, s) for k, s in shapes.items()}


# --------------------------------------------------------------------------- RoPE

@pytest.mark.parametrize("width", [4, 8, 64])
def test_rope_is_complex_rotation(width):
    x = RNG.normal(size=(5, width))
    p = np.array([0.0, 1.0, 7.5, 1000.0, 131071.0])
    base = 10.0
    y = O.rope(x, p, base)
    h = width // 2
    z = x[:, :h] + 1j * x[:, h:]
    freq = np.array([base ** (-2.0 * j / width) for j in range(h)])
    zr = z * np.exp(1j * np.outer(p, freq))
    np.testing.assert_allclose(y[:, :h], zr.real, rtol=0, atol=1e-10)  # angle ulps at p~1e5
    np.testing.assert_allclose(y[:, h:], zr.imag, rtol=0, atol=1e-10)


def test_rope_identities():
    x = RNG.normal(size=(6, 16))
    p = RNG.uniform(0, 5e4, 6)
    base = 1e6
    np.testing.assert_allclose(O.rope(O.rope(x, p, base), p, base, inverse=True), x, atol=1e-12)
    np.testing.assert_allclose(np.linalg.norm(O.rope(x, p, base), axis=-1),
                               np.linalg.norm(x, axis=-1), rtol=1e-13)
    np.testing.assert_array_equal(O.rope(x, np.zeros(6), base), x)
    q, k = RNG.normal(size=16), RNG.normal(size=16)
    a, b = 123.0, 4567.0
    lhs = O.rope(q[None], [a], base)[0] @ O.rope(k[None], [b], base)[0]
    rhs = q @ O.rope(k[None], [b - a], base)[0]
    assert abs(lhs - rhs) < 1e-10


def test_unrope_inverts_generator_rotation():
    """The oracle's RoPE-fix must undo the (independent) generator's base RoPE."""
    w = configs.shrink(configs.get_workload(2), n_tokens=64)
    c = synth.make_cache(w, 0, keep_free=True)
    rot = synth.base_rope_rotate(c["k_free"], c["positions"], w.rope_theta)
    back = O.rope(rot, c["positions"], w.rope_theta, inverse=True)
    np.testing.assert_allclose(back, c["k_free"], atol=1e-11)
    # and the bf16 cache is that rotation rounded once
    np.testing.assert_allclose(synth.bf16_value(c["K"]), rot, rtol=2 ** -8, atol=1e-30)


def test_latent_positions():
    p = np.arange(37, dtype=np.float64)
    np.testing.assert_array_equal(O.latent_positions(p, 37), p)
    np.testing.assert_array_equal(O.latent_positions(p, 1), [0.0])
    q = O.latent_positions(p, 4)
    np.testing.assert_allclose(q, [0, 12, 24, 36])
    shuffled = RNG.permutation(p)
    np.testing.assert_array_equal(O.latent_positions(shuffled, 4), q)


# --------------------------------------------------------------------------- elementwise

def test_elementwise_vs_torch():
    x = RNG.normal(size=(7, 33)) * 3
    tx = torch.from_numpy(x)
    np.testing.assert_allclose(O.rms_norm(x, 1e-6), F.rms_norm(tx, (33,), eps=1e-6).numpy(), rtol=1e-13)
    np.testing.assert_allclose(O.l2_normalize(x, 1e-12), F.normalize(tx, dim=-1, eps=1e-12).numpy(), rtol=1e-13)
    np.testing.assert_allclose(O.silu(x), F.silu(tx).numpy(), rtol=1e-13, atol=1e-300)
    np.testing.assert_allclose(O.gelu(x), F.gelu(tx).numpy(), rtol=1e-12, atol=1e-300)
    np.testing.assert_allclose(O.softmax_rows(x), torch.softmax(tx, -1).numpy(), rtol=1e-12)
    assert O.silu(np.array([-1000.0]))[0] == 0.0


# --------------------------------------------------------------------------- attention

def _cross_only_cfg(**kw):
    return tiny_cfg(n_self_heads=0, ffn_kind=configs.FFN_NONE, **kw)


def test_cross_attention_matches_sdpa():
    """softmax(s q k^T) v of one head equals torch SDPA (float64) with scale=s."""
    cfg = _cross_only_cfg(n_cross_heads=1)
    t, N = 3, 11
    w = rand_weights(cfg, t)
    Y = RNG.normal(size=(t, 8))
    X = RNG.normal(size=(N, 8))
    pk = RNG.uniform(0, 50, N)
    pq = O.latent_positions(pk, t)
    tr = {}
    O.cross_attention(Y, X, pq, pk, w, cfg, 0, trace=tr)
    q = O.rope(O.l2_normalize(Y @ w["b0.ca_wq"].T + w["b0.ca_bq"], 1e-12), pq, 10.0)
    k = O.rope(O.l2_normalize(X @ w["b0.ca_wk"].T + w["b0.ca_bk"], 1e-12), pk, 10.0)
    v = X @ w["b0.ca_wv"].T
    ref = F.scaled_dot_product_attention(torch.from_numpy(q)[None], torch.from_numpy(k)[None],
                                         torch.from_numpy(v)[None], scale=8.0)[0].numpy()
    np.testing.assert_allclose(tr["ca_heads"][0], ref, rtol=1e-12, atol=1e-14)


def test_single_key_returns_projected_value():
    cfg = _cross_only_cfg()
    w = rand_weights(cfg, 3)
    X = RNG.normal(size=(1, 8))
    tr = {}
    O.cross_attention(RNG.normal(size=(3, 8)), X, np.zeros(3), np.zeros(1), w, cfg, 0, trace=tr)
    expect = np.broadcast_to(X @ w["b0.ca_wv"].T, (3, 16))
    np.testing.assert_allclose(tr["ca_heads"][0], expect, rtol=1e-13)


def test_identical_keys_give_mean_of_values():
    """Equal positions, equal keys and W_K blind to the value half => uniform attention."""
    cfg = _cross_only_cfg()
    t, N, d = 3, 9, 4
    w = rand_weights(cfg, t)
    w["b0.ca_wk"][:, d:] = 0.0
    k_row = RNG.normal(size=d)
    X = np.concatenate([np.tile(k_row, (N, 1)), RNG.normal(size=(N, d))], axis=1)
    pk = np.full(N, 17.0)
    tr = {}
    O.cross_attention(RNG.normal(size=(t, 8)), X, O.latent_positions(pk, t), pk, w, cfg, 0, trace=tr)
    expect = np.broadcast_to(X.mean(axis=0) @ w["b0.ca_wv"].T, (t, 16))
    np.testing.assert_allclose(tr["ca_heads"][0], expect, rtol=1e-12)


def _layer_inputs(cfg, N, t, theta=1e4, rng=RNG):
    K = rng.normal(size=(cfg.n_kv_heads, N, cfg.head_dim))
    V = rng.normal(size=(cfg.n_kv_heads, N, cfg.head_dim))
    pos = np.arange(N, dtype=np.float64) * 3.0 + 5.0
    return K, V, pos, theta


def test_joint_permutation_invariance():
    cfg = tiny_cfg()
    t, N = 3, 10
    w = rand_weights(cfg, t, std=0.4)
    K, V, pos, th = _layer_inputs(cfg, N, t)
    a = O.compact_layer(K, V, pos, th, w, cfg, t)
    perm = RNG.permutation(N)
    b = O.compact_layer(K[:, perm], V[:, perm], pos[perm], th, w, cfg, t)
    for x, y in zip(a, b):
        np.testing.assert_allclose(x, y, rtol=1e-11, atol=1e-13)


@pytest.mark.parametrize("which", ["ca_wk", "ca_wq", "sa_wk", "sa_wq"])
def test_qk_projection_scale_invariance(which):
    cfg = tiny_cfg()
    t, N = 3, 7
    w = rand_weights(cfg, t, std=0.4)
    K, V, pos, th = _layer_inputs(cfg, N, t)
    a = O.compact_layer(K, V, pos, th, w, cfg, t)
    w2 = dict(w)
    w2[f"b0.{which}"] = w[f"b0.{which}"] * 3.7
    w2[f"b0.{which.replace('w', 'b', 1)}"] = w[f"b0.{which.replace('w', 'b', 1)}"] * 3.7
    b = O.compact_layer(K, V, pos, th, w2, cfg, t)
    for x, y in zip(a, b):
        np.testing.assert_allclose(x, y, rtol=1e-10, atol=1e-13)


# --------------------------------------------------------------------------- Appendix C

def identity_init_weights(cfg, t):
    """Appendix C identity-style initialisation (d_l = 2d, identity path in head 0)."""
    D, d = cfg.latent_dim, cfg.head_dim
    assert D == 2 * d
    w = {k: np.zeros(s) for k, s in configs.layer_shapes(cfg, t).items()}
    u = np.full(D, 1.0 / math.sqrt(D))
    for c in range(cfg.n_cross_heads):
        w["b0.ca_bq"][c * D:(c + 1) * D] = u
        w["b0.ca_bk"][c * D:(c + 1) * D] = u
    w["b0.ca_wv"][:D, :] = np.eye(D)          # head 0: v = X
    w["b0.ca_wo"][:, :D] = np.eye(D)          # only head 0 reaches the latents
    w["b0.ca_wv"][D:, :] = RNG.normal(size=(w["b0.ca_wv"].shape[0] - D, 2 * d))
    for k in ("sa_wq", "sa_wk", "sa_wv", "ffn_wg", "ffn_wu"):
        w[f"b0.{k}"] = RNG.normal(0, 0.1, w[f"b0.{k}"].shape)
    w["w_key"][:, :d] = np.eye(d)             # W_key = [I 0]
    w["w_val"][:, d:] = np.eye(d)             # W_val = [0 I]
    return w


@pytest.mark.parametrize("theta", [1e6, 1e4])
def test_identity_init_is_near_pass_through(theta):
    cfg = configs.get_workload(1).cfg          # d=64, D=128, n_c=2
    N = t = 48
    w = identity_init_weights(cfg, t)
    K = RNG.normal(size=(cfg.n_kv_heads, N, cfg.head_dim))
    V = RNG.normal(size=(cfg.n_kv_heads, N, cfg.head_dim))
    pos = np.arange(N, dtype=np.float64)
    Krot = O.rope(K, pos, theta)
    Ck, Cv, pq = O.compact_layer(Krot, V, pos, theta, w, cfg, t)
    np.testing.assert_array_equal(pq, pos)
    np.testing.assert_allclose(Ck, Krot, rtol=0, atol=2e-5 * np.abs(Krot).max())
    np.testing.assert_allclose(Cv, V, rtol=0, atol=2e-5 * np.abs(V).max())
    # the d_l logit scale is what makes the pattern sharp: 1/sqrt(d_l) breaks it
    cfg2 = configs.CompactorConfig(**{**cfg.__dict__, "logit_scale_cross": 1.0 / math.sqrt(128)})
    Ck2, _, _ = O.compact_layer(Krot, V, pos, theta, w, cfg2, t)
    assert np.abs(Ck2 - Krot).max() > 0.1


# --------------------------------------------------------------------------- loop evaluation

def _loop_layer(K, V, pos, theta, w, cfg, t, rerotate=True):
    """Whole layer with explicit Python loops (tiny sizes), written independently."""
    H, N, d = K.shape
    nc, dc, ns, ds = cfg.n_cross_heads, cfg.dc, cfg.n_self_heads, cfg.ds

    def lin(x, W, b=None):
        return [sum(x[i] * W[o][i] for i in range(len(x))) + (b[o] if b is not None else 0.0)
                for o in range(len(W))]

    def rot(x, p, base, sgn):
        n2 = len(x) // 2
        y = list(x)
        for j in range(n2):
            a = sgn * p * base ** (-2.0 * j / len(x))
            y[j] = x[j] * math.cos(a) - x[j + n2] * math.sin(a)
            y[j + n2] = x[j + n2] * math.cos(a) + x[j] * math.sin(a)
        return y

    def rms(x):
        r = math.sqrt(sum(v * v for v in x) / len(x) + cfg.rms_eps)
        return [v / r for v in x]

    def unit(x):
        r = max(math.sqrt(sum(v * v for v in x)), cfg.l2_eps)
        return [v / r for v in x]

    def attend(qs, ks, vs, s):
        out = []
        for q in qs:
            lg = [s * sum(a * b for a, b in zip(q, k)) for k in ks]
            m = max(lg)
            e = [math.exp(v - m) for v in lg]
            z = sum(e)
            out.append([sum(e[n] * vs[n][f] for n in range(len(vs))) / z for f in range(len(vs[0]))])
        return out

    def add(Z, rows):
        return [[a + b for a, b in zip(z, r)] for z, r in zip(Z, rows)]

    lo, hi = min(pos), max(pos)
    pq = [lo + i * (hi - lo) / (t - 1) for i in range(t)] if t > 1 else [lo]
    Ck = np.zeros((H, t, d))
    Cv = np.zeros((H, t, d))
    for h in range(H):
        X = [rot(list(K[h, n]), pos[n], theta, -1) + list(V[h, n]) for n in range(N)]
        Z = [list(w["latents"][h, i]) for i in range(t)]
        for b in range(cfg.n_blocks):
            B = f"b{b}."
            if nc and (b == 0 or cfg.cross_every_block):
                Q = [rms(z) for z in Z]
                cat = [[] for _ in range(t)]
                for c in range(nc):
                    r = slice(c * dc, (c + 1) * dc)
                    qs = [rot(unit(lin(q, w[B + "ca_wq"][r], w[B + "ca_bq"][r])), pq[i],
                              cfg.compactor_rope_base, 1) for i, q in enumerate(Q)]
                    ks = [rot(unit(lin(x, w[B + "ca_wk"][r], w[B + "ca_bk"][r])), pos[n],
                              cfg.compactor_rope_base, 1) for n, x in enumerate(X)]
                    vs = [lin(x, w[B + "ca_wv"][r]) for x in X]
                    for i, o in enumerate(attend(qs, ks, vs, dc)):
                        cat[i] += o
                Z = add(Z, [lin(c_, w[B + "ca_wo"]) for c_ in cat])
            if ns:
                Y = [rms(z) for z in Z]
                cat = [[] for _ in range(t)]
                for c in range(ns):
                    r = slice(c * ds, (c + 1) * ds)
                    qs = [unit(lin(y, w[B + "sa_wq"][r], w[B + "sa_bq"][r])) for y in Y]
                    ks = [unit(lin(y, w[B + "sa_wk"][r], w[B + "sa_bk"][r])) for y in Y]
                    vs = [lin(y, w[B + "sa_wv"][r]) for y in Y]
                    for i, o in enumerate(attend(qs, ks, vs, ds)):
                        cat[i] += o
                Z = add(Z, [lin(c_, w[B + "sa_wo"]) for c_ in cat])
            if cfg.ffn_kind != configs.FFN_NONE:
                Y = [rms(z) for z in Z]
                upd = []
                for y in Y:
                    u = lin(y, w[B + "ffn_wu"])
                    if cfg.ffn_kind == configs.FFN_SWIGLU:
                        g = lin(y, w[B + "ffn_wg"])
                        hdn = [gv / (1 + math.exp(-gv)) * uv for gv, uv in zip(g, u)]
                    else:
                        hdn = [0.5 * uv * (1 + math.erf(uv / math.sqrt(2))) for uv in u]
                    upd.append(lin(hdn, w[B + "ffn_wd"]))
                Z = add(Z, upd)
        if cfg.final_norm:
            Z = [rms(z) for z in Z]
        for i in range(t):
            ck = lin(Z[i], w["w_key"])
            Ck[h, i] = rot(ck, pq[i], theta, 1) if rerotate else ck
            Cv[h, i] = lin(Z[i], w["w_val"])
    return Ck, Cv, np.array(pq)


LOOP_VARIANTS = {
    "base": {},
    "gelu_final_norm": dict(ffn_kind=configs.FFN_GELU, final_norm=1),
    "two_blocks": dict(n_blocks=2),
    "resampler": dict(n_blocks=2, cross_every_block=0, n_cross_heads=1),
    "cross_only_one_head": dict(n_self_heads=0, ffn_kind=configs.FFN_NONE, n_cross_heads=1),
}


@pytest.mark.parametrize("variant", list(LOOP_VARIANTS))
def test_layer_matches_loop_evaluation(variant, rerotate=True):
    cfg = tiny_cfg(**LOOP_VARIANTS[variant])
    t, N = 3, 6
    w = rand_weights(cfg, t, std=0.6, rng=np.random.default_rng(11))
    K, V, pos, th = _layer_inputs(cfg, N, t, rng=np.random.default_rng(12))
    ref = _loop_layer(K, V, pos, th, w, cfg, t, rerotate=rerotate)
    got = O.compact_layer(K, V, pos, th, w, cfg, t, rerotate=rerotate)
    for a, b in zip(got, ref):
        np.testing.assert_allclose(a, b, rtol=1e-11, atol=1e-12)


def test_layer_matches_loop_evaluation_no_rerotate_single_latent():
    test_layer_matches_loop_evaluation("base", rerotate=False)
    cfg = tiny_cfg()
    w = rand_weights(cfg, 1, std=0.6, rng=np.random.default_rng(13))
    K, V, pos, th = _layer_inputs(cfg, 5, 1, rng=np.random.default_rng(14))
    for a, b in zip(O.compact_layer(K, V, pos, th, w, cfg, 1), _loop_layer(K, V, pos, th, w, cfg, 1)):
        np.testing.assert_allclose(a, b, rtol=1e-11, atol=1e-12)


# --------------------------------------------------------------------------- sizes

def _count(cfg, t):
    n = 0
    for name, shape in configs.layer_shapes(cfg, t).items():
        if len(shape) == 1:        # biases are ignored by the paper's count
            continue
        n += int(np.prod(shape))
    return n + cfg.latent_dim      # + the optional beta head w_beta in R^{d_l}


GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_rows(name):
    """Whitespace-separated rows of a fixture under tests/golden (comments dropped)."""
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].split()
            if line:
                rows.append(line)
    return rows


_PARAM_ROWS = [r for r in _golden_rows("appendix_d_parameter_counts.txt") if r[0] != "bf16_canonical"]
_L, _H, _D, _DL = 36, 8, 128, 256   # Qwen3-4B-shaped base model and d_l of the printed configurations


def _formula(row):
    t, B, Bc, nc, ns, r = (int(v) for v in row[:6])
    return sizing.compactor_params_per_layer(_H, t, _D, _DL, B, Bc, nc, ns, r, ffn=bool(r))


@pytest.mark.parametrize("row", _PARAM_ROWS, ids=[r[6] for r in _PARAM_ROWS])
def test_parameter_count_appendix_d(row):
    """App. D totals: the formula, the oracle's own tensor shapes and the printed figure agree."""
    t, B, Bc, nc, ns, r = (int(v) for v in row[:6])
    printed, tol = float(row[6]), float(row[7])
    cfg = configs.CompactorConfig(n_kv_heads=_H, head_dim=_D, latent_dim=_DL, n_blocks=B,
                                  cross_every_block=int(Bc == B), n_cross_heads=nc, n_self_heads=ns,
                                  ffn_kind=configs.FFN_GELU if r else configs.FFN_NONE,
                                  ffn_hidden=r * _DL)
    formula = _formula(row)
    assert _count(cfg, t) == formula
    assert abs(_L * formula - printed) / printed < tol


def test_canonical_bf16_bytes_appendix_b():
    """App. B: the canonical compactor's bf16 storage, from its App. D count."""
    (mib_row,) = [r for r in _golden_rows("appendix_d_parameter_counts.txt") if r[0] == "bf16_canonical"]
    printed, tol = float(mib_row[1]), float(mib_row[2])
    canonical = _PARAM_ROWS[0]
    assert abs(_L * _formula(canonical) * 2 / 2 ** 20 - printed) / printed < tol


def test_kv_bytes_appendix_b():
    """App. B: M_KV(S) = 2 L H_kv d b S for the Qwen3-4B-shaped cache, against the printed sizes."""
    unit = {"KiB": 2 ** 10, "MiB": 2 ** 20, "GiB": 2 ** 30}
    rows = _golden_rows("appendix_b_kv_footprint.txt")
    assert len(rows) == 6
    for _, S, printed, u, tol in rows:
        got = sizing.kv_bytes(36, 8, 128, 2, int(S)) / unit[u]
        want = float(printed)
        if float(tol) == 0:
            assert got == want
        else:
            assert abs(got - want) / want < float(tol)


# --------------------------------------------------------------------------- Appendix B compositions

def test_subrange_and_chunks_reduce_to_one_call():
    cfg = tiny_cfg()
    t, N = 3, 9
    w = rand_weights(cfg, t, std=0.5, rng=np.random.default_rng(21))
    K, V, pos, th = _layer_inputs(cfg, N, t, rng=np.random.default_rng(22))
    ref = O.compact_layer(K, V, pos, th, w, cfg, t)
    for got in (O.compact_subrange(K, V, pos, th, w, cfg, t, 0, N), O.compact_chunks(K, V, pos, th, w, cfg, t, N),
                O.compact_chunks(K, V, pos, th, w, cfg, t, 5 * N)):
        for a, b in zip(got, ref):
            np.testing.assert_array_equal(a, b)


def test_subrange_identity_init_is_near_pass_through():
    """Appendix B splice with the Appendix C identity-style compactor at
    t = end - start: the spliced cache reproduces the original one."""
    cfg = configs.get_workload(1).cfg
    N, s, e = 80, 17, 65
    t = e - s
    w = identity_init_weights(cfg, t)
    rng = np.random.default_rng(23)
    K = O.rope(rng.normal(size=(cfg.n_kv_heads, N, cfg.head_dim)), np.arange(N, dtype=np.float64), 1e4)
    V = rng.normal(size=(cfg.n_kv_heads, N, cfg.head_dim))
    pos = np.arange(N, dtype=np.float64)
    K2, V2, p2 = O.compact_subrange(K, V, pos, 1e4, w, cfg, t, s, e)
    np.testing.assert_array_equal(p2, pos)
    np.testing.assert_array_equal(K2[:, :s], K[:, :s])          # preserved entries untouched
    np.testing.assert_array_equal(V2[:, e:], V[:, e:])
    np.testing.assert_allclose(K2, K, rtol=0, atol=2e-5 * np.abs(K).max())
    np.testing.assert_allclose(V2, V, rtol=0, atol=2e-5 * np.abs(V).max())


def test_chunks_identity_init_is_near_pass_through():
    cfg = configs.get_workload(1).cfg
    N, chunk = 96, 32
    w = identity_init_weights(cfg, chunk)
    rng = np.random.default_rng(24)
    pos = np.arange(N, dtype=np.float64) * 2.0
    K = O.rope(rng.normal(size=(cfg.n_kv_heads, N, cfg.head_dim)), pos, 1e6)
    V = rng.normal(size=(cfg.n_kv_heads, N, cfg.head_dim))
    K2, V2, p2 = O.compact_chunks(K, V, pos, 1e6, w, cfg, chunk, chunk)
    np.testing.assert_array_equal(p2, pos)
    np.testing.assert_allclose(K2, K, rtol=0, atol=2e-5 * np.abs(K).max())
    np.testing.assert_allclose(V2, V, rtol=0, atol=2e-5 * np.abs(V).max())
