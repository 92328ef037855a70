"""GPU parity where the design is most fragile, against the fp64 oracle.

* Near ties: every cache row repeated 8 to 128 times at one position, so
  each latent's heaviest key comes with exact twins inside the refinement
  margin (the ill-conditioned case of the d_l logit scale, App. A
  cross-attention), in both modes; 512-fold duplication, beyond the
  candidate capacity, is recorded, not gated.
* A whole 36-layer Qwen-shaped call: bit-identical on replay and equal, layer
  by layer, to single-layer calls (the workspace is reused layer after
  layer), with its first and last layers checked against the oracle.
* Multi-block compactors (App. A "Compactor blocks", B = 2 with
  cross-attention in every block) and the paper's canonical compactor
  (App. A canonical configuration: d_l = 256, B = 2, n_c = n_s = 1, no FFN);
  at the d_l logit scale, where fp32 arithmetic cannot reach 1e-4, the fp32
  mode is gated against the oracle's own spread under unit-roundoff input
  perturbations.
* The App. C identity-style initialisation at t = N on the GPU: the compact
  cache reproduces the input cache.
* A workspace filled with NaN bit patterns before the call, at ragged N and t
  (key tiles past N and past t are padding), for the cfg-1 compactor and the
  Qwen-8B-shaped one: nothing stale may reach the outputs.
"""
import math

import numpy as np
import pytest

from paper_2606_07878_amd import configs, synth
from tests.helpers import (BF16_TOL, FP32_TOL, assert_parity, dev_tensor, log, run_gpu, run_oracle,
                           slice_errors)

pytestmark = pytest.mark.gpu

W1 = configs.get_workload(1)
W2 = configs.get_workload(2)
MODES = [(configs.MODE_BF16, BF16_TOL), (configs.MODE_FP32, FP32_TOL)]


def _duplicated_cache(w, layer, distinct, copies):
    """`distinct` cache rows at positions 0, copies, 2 copies, ..., each row
    (key, value, position) repeated `copies` times in a row."""
    pos = np.arange(distinct, dtype=np.float64) * copies
    c = synth.make_cache(w, layer, n_tokens=distinct, positions=pos)
    return dict(K=np.repeat(c["K"], copies, axis=1), V=np.repeat(c["V"], copies, axis=1),
                positions=np.repeat(pos, copies))


def _duplication_case(copies, mode, tol):
    w = W2
    cache = _duplicated_cache(w, 7, w.n_tokens // copies, copies)
    wts = synth.make_weights(w, 7)
    heads = [0, 5]
    log(f"case near ties: {w.n_tokens // copies} rows x {copies} copies, mode {mode}, heads {heads}")
    ref = run_oracle(w.cfg, cache, wts, w.rope_theta, w.t, heads=heads)
    got = run_gpu(w.cfg, cache, wts, w.rope_theta, w.t, mode=mode)
    assert_parity((got[0][heads], got[1][heads], got[2]), ref, tol, what=f"near ties x{copies} mode{mode}")


@pytest.mark.parametrize("copies,mode,tol", [(8, configs.MODE_BF16, BF16_TOL), (16, configs.MODE_BF16, BF16_TOL),
                                             (32, configs.MODE_BF16, BF16_TOL), (128, configs.MODE_BF16, BF16_TOL),
                                             (16, configs.MODE_FP32, FP32_TOL), (128, configs.MODE_FP32, FP32_TOL)])
def test_near_ties_duplicated_rows_qwen_shape(copies, mode, tol):
    """Qwen-8B-shaped compactor (D = 1024, 8 + 8 heads), N = 8192 made of
    8192 / copies distinct rows each repeated `copies` times: every candidate
    key has copies - 1 exact ties, so tens to over a thousand keys per latent
    sit inside the refinement margin, and early key blocks (compared with a
    smaller running maximum) put many more into the candidate lists."""
    _duplication_case(copies, mode, tol)


HEAVY_DUPLICATION_XFAIL = pytest.mark.xfail(
    reason="rows repeated 512 times put more keys per latent inside the refinement margin than the candidate "
           "capacity (1536 overflow entries per row, 256 refined keys per latent): measured bf16 3.4e-2 / 3.7e-2, "
           "fp32 1.2e-4 / 1.2e-4 (recorded, not gated)", strict=False)


@HEAVY_DUPLICATION_XFAIL
@pytest.mark.parametrize("mode,tol", MODES)
def test_heavy_duplication_recorded(mode, tol):
    """The near-tie case beyond the refinement capacity: 16 distinct rows
    each repeated 512 times."""
    _duplication_case(512, mode, tol)


def test_model_36_layers_replay_and_oracle():
    """One still_compact_model call over the 36-layer 8k -> 1024 stack (the
    benchmark's launch configuration), inputs drawn on the device: two calls
    give bit-identical outputs, every checked layer equals a single-layer
    call bit for bit, and layers 0 and 35 match the oracle."""
    import torch
    from paper_2606_07878_amd import binding
    w = W2
    dev = torch.device("cuda")
    L = w.n_layers
    log(f"case 36-layer model: generating {L} layers")
    layers = [synth.make_layer_torch(w, l, dev) for l in range(L)]
    Ks = [x[0] for x in layers]
    Vs = [x[1] for x in layers]
    pos = layers[0][2]
    Ws = [x[3] for x in layers]
    runs = []
    for rep in range(2):
        Ck, Cv, p = binding.compact_model(w.cfg, Ws, Ks, Vs, pos, w.rope_theta, w.t)
        torch.cuda.synchronize()
        runs.append((Ck, Cv, p))
        log(f"model call {rep} done")
    for l in range(L):
        assert torch.equal(runs[0][0][l], runs[1][0][l]) and torch.equal(runs[0][1][l], runs[1][1][l]), \
            f"layer {l}: replay differs"
    assert torch.equal(runs[0][2], runs[1][2])
    for l in (0, 17, 35):
        Ck1, Cv1, _ = binding.compact_layer(w.cfg, Ws[l], Ks[l], Vs[l], pos, w.rope_theta, w.t)
        torch.cuda.synchronize()
        assert torch.equal(Ck1, runs[0][0][l]) and torch.equal(Cv1, runs[0][1][l]), \
            f"layer {l}: model call differs from the single-layer call"
    log("replay and single-layer equality ok")
    f64 = lambda x: x.double().cpu().numpy()  # noqa: E731
    for l, heads in ((0, [1]), (35, [6])):
        cache = dict(K=f64(Ks[l]), V=f64(Vs[l]), positions=pos.cpu().numpy())
        wts = {k: f64(v) for k, v in Ws[l].items()}
        ref = run_oracle(w.cfg, cache, wts, w.rope_theta, w.t, heads=heads)
        got = (f64(runs[0][0][l])[heads], f64(runs[0][1][l])[heads], runs[0][2].cpu().numpy())
        assert_parity(got, ref, BF16_TOL, what=f"36-layer model, layer {l}")


# ----------------------------------------------------------------------------
# Multi-block and canonical compactors
# ----------------------------------------------------------------------------

def _inv_sqrt_scale(cfg):
    """The 1/sqrt(d_l) logit scale of the paper's scale ablation, for cross-
    and self-attention."""
    return dict(logit_scale_cross=1.0 / math.sqrt(cfg.dc), logit_scale_self=1.0 / math.sqrt(cfg.ds))


def _modes_case(w, name, heads=None, modes=MODES):
    cache = synth.make_cache(w, 0)
    wts = synth.make_weights(w, 0)
    log(f"case {name}: N={w.n_tokens} t={w.t}")
    ref = run_oracle(w.cfg, cache, wts, w.rope_theta, w.t, heads=heads)
    errs = []
    for mode, tol in modes:
        got = run_gpu(w.cfg, cache, wts, w.rope_theta, w.t, mode=mode)
        if heads is not None:
            got = (got[0][heads], got[1][heads], got[2])
        errs.append(assert_parity(got, ref, tol, what=f"{name} mode{mode}"))
    return errs


@pytest.mark.parametrize("ffn", [configs.FFN_SWIGLU, configs.FFN_GELU])
def test_two_blocks_cross_every_block_inv_sqrt_scale(ffn):
    """B = 2 with cross-attention in both blocks (block 2 re-tiles its own
    W_K, projects the keys again and refines and merges a second time) at the
    1/sqrt(d_l) logit scale, where the map is well conditioned."""
    c = configs.shrink(W1, n_blocks=2, cross_every_block=1, ffn_kind=ffn, final_norm=int(ffn == configs.FFN_GELU))
    c = configs.shrink(c, **_inv_sqrt_scale(c.cfg))
    _modes_case(c, f"B=2 cross every block, 1/sqrt(d_l) scale, ffn {ffn}")


def _canonical(w):
    """App. A canonical compactor: d_l = 256, B = 2 blocks each with cross- and
    self-attention (one head of width d_l), no FFN."""
    return configs.shrink(w, latent_dim=256, n_blocks=2, cross_every_block=1, n_cross_heads=1,
                          n_self_heads=1, ffn_kind=configs.FFN_NONE, ffn_hidden=0)


def test_canonical_compactor_qwen_cache_inv_sqrt_scale():
    """The canonical compactor on a Qwen-shaped 8k cache (H = 8, d = 128,
    N = 8192 -> t = 1024) at the 1/sqrt(d_l) logit scale."""
    c = _canonical(W2)
    c = configs.shrink(c, **_inv_sqrt_scale(c.cfg))
    _modes_case(c, "canonical d_l=256 B=2, 1/sqrt(d_l) scale", heads=[0, 3])


CANONICAL_DL_XFAIL = pytest.mark.xfail(
    reason="B=2 at the d_l logit scale is ill-conditioned: on the fp64 oracle a random relative perturbation "
           "of 1e-7 (fp32 rounding) of the inputs and weights moves C_k / C_v by 5.1e-4 / 4.8e-4, above the "
           "fp32 mode's 1e-4 bar, and block 1's fp16-operand error is amplified likewise in bf16 mode "
           "(measured: bf16 1.4e-1 / 1.3e-1, fp32 1.4e-4 / 1.6e-4; the fp32 mode is gated against that spread by "
           "test_canonical_compactor_dl_scale_fp32_conditioning_bound)", strict=False)


@CANONICAL_DL_XFAIL
@pytest.mark.parametrize("mode,tol", MODES)
def test_canonical_compactor_qwen_cache_dl_scale(mode, tol):
    """The canonical compactor at the paper's d_l logit scale (both blocks
    run, each with its own refinement and merge; recorded, not gated)."""
    _modes_case(_canonical(W2), "canonical d_l=256 B=2, d_l scale", heads=[0, 3], modes=[(mode, tol)])


def _perturbed(a, u, rng):
    """a (1 + u xi) with xi uniform on [-1, 1]: a random relative perturbation
    of size u of every element (bf16 bit patterns are decoded first)."""
    a = synth.as_f64({"x": a})["x"]
    return a * (1.0 + u * rng.uniform(-1.0, 1.0, a.shape))


def test_canonical_compactor_dl_scale_fp32_conditioning_bound():
    """Gated companion of the recorded d_l-scale canonical case, fp32 mode.
    A computation in fp32 arithmetic can be expected to be as accurate as the
    exact map evaluated at inputs perturbed by fp32's unit roundoff (2^-24),
    no more: the fp64 oracle is run on three such perturbed copies of the
    cache and of every weight (positions exact), and the GPU's deviation from
    the unperturbed oracle must stay within twice the largest deviation they
    show.  A fault in either block's kernels moves the output by orders of
    magnitude more than this spread (about 2e-4 here)."""
    w = _canonical(W2)
    heads = [0, 3]
    cache = synth.make_cache(w, 0)
    wts = synth.make_weights(w, 0)
    log(f"case canonical d_l scale, fp32 conditioning bound: N={w.n_tokens} t={w.t}")
    ref = run_oracle(w.cfg, cache, wts, w.rope_theta, w.t, heads=heads)
    u = 2.0 ** -24
    spread = 0.0
    for draw in range(3):
        rng = np.random.default_rng(900 + draw)
        cp = dict(K=_perturbed(cache["K"], u, rng), V=_perturbed(cache["V"], u, rng), positions=cache["positions"])
        wp = {k: _perturbed(v, u, rng) for k, v in wts.items()}
        rp = run_oracle(w.cfg, cp, wp, w.rope_theta, w.t, heads=heads)
        spread = max(spread, slice_errors(rp[0], ref[0]).max(), slice_errors(rp[1], ref[1]).max())
    log(f"oracle spread under 2^-24 input perturbations: {spread:.3e}")
    assert 0.0 < spread < 1e-2
    got = run_gpu(w.cfg, cache, wts, w.rope_theta, w.t, mode=configs.MODE_FP32)
    assert_parity((got[0][heads], got[1][heads], got[2]), ref, 2.0 * spread,
                  what="canonical d_l scale fp32 vs conditioning bound")


# ----------------------------------------------------------------------------
# App. C identity-style initialisation on the GPU
# ----------------------------------------------------------------------------

def _identity_weights(cfg, t, rng):
    """App. C identity-style initialisation (d_l = 2d): zero latents, W_Q = W_K
    = 0 with b_Q = b_K = the unit vector 1/sqrt(d_l), head 0's value path the
    identity and the only head reaching the latents through W_O, the
    self-attention output and FFN down projections 0, W_key = [I 0],
    W_val = [0 I].  Other matrices random.  Returned as bf16 bits."""
    D, d = cfg.latent_dim, cfg.head_dim
    assert D == 2 * d
    w = {k: np.zeros(s) for k, s in configs.layer_shapes(cfg, t).items()}
    u = np.full(D, 1.0 / math.sqrt(D))
    for c in range(cfg.n_cross_heads):
        w["b0.ca_bq"][c * D:(c + 1) * D] = u
        w["b0.ca_bk"][c * D:(c + 1) * D] = u
    w["b0.ca_wv"][:D, :] = np.eye(D)
    w["b0.ca_wo"][:, :D] = np.eye(D)
    w["b0.ca_wv"][D:, :] = rng.normal(size=(w["b0.ca_wv"].shape[0] - D, 2 * d))
    for k in ("sa_wq", "sa_wk", "sa_wv", "ffn_wg", "ffn_wu"):
        w[f"b0.{k}"] = rng.normal(0, 0.1, w[f"b0.{k}"].shape)
    w["w_key"][:, :d] = np.eye(d)
    w["w_val"][:, d:] = np.eye(d)
    return {k: synth.bf16_bits(v) for k, v in w.items()}


@pytest.mark.parametrize("theta", [1e6, 1e4])
def test_identity_init_reproduces_cache(theta):
    """t = N = 256 with the identity-style compactor: out positions are the
    input positions and (C_k, C_v) reproduce (K, V), in both modes; the GPU
    also matches the oracle on the same weights."""
    import dataclasses
    w = dataclasses.replace(configs.shrink(W1, n_tokens=256, t=256), rope_theta=theta)
    wts = _identity_weights(w.cfg, w.t, np.random.default_rng(5))
    cache = synth.make_cache(w, 0)
    K, V = synth.bf16_value(cache["K"]), synth.bf16_value(cache["V"])
    ref = run_oracle(w.cfg, cache, wts, w.rope_theta, w.t)
    np.testing.assert_array_equal(ref[2], cache["positions"])
    # the oracle itself is a pass-through here (App. C)
    assert slice_errors(ref[0], K).max() < 1e-5 and slice_errors(ref[1], V).max() < 1e-5
    for mode, tol in MODES:
        got = run_gpu(w.cfg, cache, wts, w.rope_theta, w.t, mode=mode)
        assert_parity(got, ref, tol, what=f"identity init theta={theta:g} mode{mode}")
        ek, ev = slice_errors(got[0], K).max(), slice_errors(got[1], V).max()
        log(f"identity init theta={theta:g} mode{mode}: |C_k - K| {ek:.3e}  |C_v - V| {ev:.3e}")
        assert ek <= tol and ev <= tol


# ----------------------------------------------------------------------------
# Cache magnitudes beyond the fp16 operands' range (bf16 I/O allows 3.4e38)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("wid,outlier,vscale,N,t", [(1, 1e5, 1.0, 2048, 256), (1, 10.0, 1e5, 2048, 256),
                                                     (2, 1e4, 1.0, 2240, 256)])
def test_large_cache_magnitudes(wid, outlier, vscale, N, t):
    """Keys with 4 outlier channels per head of standard deviation 1e5
    (cfg 1, max ~5e5) or 1e4 (Qwen shape, max ~5e4), or values of standard
    deviation 1e5: bf16 represents them, fp16 (max 65504) does not, or only
    with no headroom.  The bf16 path stages each KV head scaled by a power of
    two and must match the oracle like any other cache."""
    import dataclasses
    w = dataclasses.replace(configs.get_workload(wid), outlier_channels=4, outlier_scale=outlier)
    cache = synth.make_cache(w, 0, n_tokens=N)
    if vscale != 1.0:
        cache["V"] = synth.bf16_bits(synth.bf16_value(cache["V"]) * vscale)
    kmax, vmax = np.abs(synth.bf16_value(cache["K"])).max(), np.abs(synth.bf16_value(cache["V"])).max()
    log(f"case large magnitudes: cfg{wid} max|K| {kmax:.3g} max|V| {vmax:.3g}")
    assert max(kmax, vmax) > 16384
    wts = synth.make_weights(w, 0, t=t)
    heads = [0, 1] if wid == 1 else [0, 5]
    ref = run_oracle(w.cfg, cache, wts, w.rope_theta, t, heads=heads)
    for mode, tol in MODES:
        got = run_gpu(w.cfg, cache, wts, w.rope_theta, t, mode=mode)
        assert_parity((got[0][heads], got[1][heads], got[2]), ref, tol,
                      what=f"large magnitudes cfg{wid} K x{outlier:g} V x{vscale:g} mode{mode}")


def _poisoned_case(w, N, t, mode, tol, heads=None):
    """One layer with the workspace filled with all-ones bytes (NaN in fp16
    and fp32) before the call, against the oracle."""
    import torch
    from paper_2606_07878_amd import binding
    cache = synth.make_cache(w, 0, n_tokens=N)
    wts = synth.make_weights(w, 0, t=t)
    log(f"case poisoned workspace: {w.name} N={N} t={t} mode {mode}")
    need = binding.still_workspace_size(binding.make_config(w.cfg, mode), N, t, 1)
    ws = torch.full((need,), 255, dtype=torch.uint8, device="cuda")
    K = dev_tensor(cache["K"], mode)
    V = dev_tensor(cache["V"], mode)
    pos = torch.from_numpy(cache["positions"]).cuda()
    W = {k: dev_tensor(v, mode) for k, v in wts.items()}
    Ck, Cv, p = binding.compact_layer(w.cfg, W, K, V, pos, w.rope_theta, t, mode=mode, workspace=ws)
    torch.cuda.synchronize()
    got = (Ck.double().cpu().numpy(), Cv.double().cpu().numpy(), p.cpu().numpy())
    if heads is not None:
        got = (got[0][heads], got[1][heads], got[2])
    ref = run_oracle(w.cfg, cache, wts, w.rope_theta, t, heads=heads)
    assert_parity(got, ref, tol, what=f"N={N} t={t} poisoned workspace mode{mode}")


@pytest.mark.parametrize("mode,tol", MODES)
def test_poisoned_workspace_ragged_shapes(mode, tol):
    """cfg-1 compactor (flash self-attention, d_s = 128) at N = 1000, t = 300:
    the cross-attention's last key tile and the self-attention's last latent
    tile are partly padding; the workspace starts as all-ones bytes (NaN in
    fp16 and fp32)."""
    _poisoned_case(W1, 1000, 300, mode, tol)


@pytest.mark.parametrize("N,t", [(1000, 300), (4097, 129)])
@pytest.mark.parametrize("mode,tol", MODES)
def test_poisoned_workspace_ragged_qwen_shape(N, t, mode, tol):
    """The Qwen-8B-shaped compactor (8 KV heads of width 128, D = 1024, 8 + 8
    heads of width 1024) at ragged N and t: the key projection's workgroups of
    16 keys x 8 KV heads end inside the cache, the 256-key blocks of the
    cross-attention (2d = 256) end in padding, the wide self-attention's
    score rows end in padding; the workspace starts as NaN bit patterns."""
    _poisoned_case(W2, N, t, mode, tol, heads=[0, 7])


@pytest.mark.parametrize("mode,tol", MODES)
def test_poisoned_workspace_ragged_wide_heads(mode, tol):
    """The 64k-cache stack's compactor (8 KV heads of width 256, so 2d = 512:
    64-latent cross-attention tiles, the d = 256 refinement and key
    projection; D = 2048) at N = 1000, t = 300, NaN-poisoned workspace."""
    _poisoned_case(configs.get_workload(5), 1000, 300, mode, tol, heads=[0, 7])
