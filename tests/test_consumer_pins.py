"""Pins of the bias-channel and consumer-attention oracle (CPU only).

Each pin checks the oracle against something other than itself: torch's
scaled-dot-product attention with an additive mask, the identity between a
log-count bias and duplicated cache entries, causality and grouping
invariants, and the bias head against the value head on the same final
latent state.
"""
import math

import numpy as np
import pytest
import torch

from oracle import compactor
from oracle import consumer as O
from paper_2606_07878_amd import configs, synth


def _inputs(seed, H=2, group=2, nq=3, t=5, S=4, d=16):
    a = synth.make_attend_inputs(seed, H, group, nq, t, S, d)
    f = synth.as_f64(a)
    f["beta"] = a["beta"].astype(np.float64)
    return f


def _sdpa(f, group, causal, scale=None):
    """torch SDPA (float64) over [C_k; K] with an additive mask [beta; 0] (+ causal -inf)."""
    q = torch.from_numpy(f["q"])
    H, t = f["C_k"].shape[:2]
    S, nq = f["K"].shape[1], q.shape[1]
    keys = torch.from_numpy(np.concatenate([f["C_k"], f["K"]], axis=1)).repeat_interleave(group, 0)
    vals = torch.from_numpy(np.concatenate([f["C_v"], f["V"]], axis=1)).repeat_interleave(group, 0)
    bias = np.concatenate([f["beta"] if f["beta"] is not None else np.zeros((H, t)), np.zeros((H, S))], axis=1)
    mask = torch.from_numpy(bias).repeat_interleave(group, 0)[:, None, :].expand(-1, nq, -1).clone()
    if causal:
        for i in range(nq):
            mask[:, i, t + S - nq + i + 1:] = -math.inf
    return torch.nn.functional.scaled_dot_product_attention(q, keys, vals, attn_mask=mask, scale=scale).numpy()


@pytest.mark.parametrize("group,causal", [(1, False), (2, False), (2, True), (3, True)])
def test_attend_matches_sdpa_with_additive_mask(group, causal):
    f = _inputs(1, group=group)
    got = O.attend(f["q"], f["C_k"], f["C_v"], f["beta"], f["K"], f["V"], group=group, causal=causal)
    np.testing.assert_allclose(got, _sdpa(f, group, causal), rtol=1e-12, atol=1e-12)


def test_attend_explicit_scale_matches_sdpa():
    f = _inputs(2)
    got = O.attend(f["q"], f["C_k"], f["C_v"], f["beta"], f["K"], f["V"], group=2, scale=0.3)
    np.testing.assert_allclose(got, _sdpa(f, 2, False, scale=0.3), rtol=1e-12, atol=1e-12)


def test_log_count_bias_equals_duplicated_entries():
    """beta_j = log m_j acts exactly like m_j copies of compact entry j with
    beta = 0 (the attention-mass reading behind mass matching)."""
    f = _inputs(3, H=1, group=1, nq=2, t=4, S=3)
    m = np.array([1, 3, 2, 5])
    beta = np.log(m)[None, :].astype(np.float64)
    got = O.attend(f["q"], f["C_k"], f["C_v"], beta, f["K"], f["V"])
    dup_k = np.repeat(f["C_k"], m, axis=1)
    dup_v = np.repeat(f["C_v"], m, axis=1)
    ref = O.attend(f["q"], dup_k, dup_v, None, f["K"], f["V"])
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-13)


def test_uniform_bias_on_empty_suffix_cancels():
    """With no suffix a constant bias on every compact entry cancels in the softmax."""
    f = _inputs(4, S=0)
    a = O.attend(f["q"], f["C_k"], f["C_v"], None, f["K"], f["V"], group=2)
    b = O.attend(f["q"], f["C_k"], f["C_v"], np.full(f["C_k"].shape[:2], 7.5), f["K"], f["V"], group=2)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-13)


def test_single_visible_entry_returns_its_value():
    """t = 1, no suffix: every query returns the one compact value row."""
    f = _inputs(5, H=2, group=2, nq=2, t=1, S=0)
    got = O.attend(f["q"], f["C_k"], f["C_v"], f["beta"], f["K"], f["V"], group=2)
    for hq in range(4):
        np.testing.assert_allclose(got[hq], np.broadcast_to(f["C_v"][hq // 2, 0], got[hq].shape), rtol=1e-14)


def test_causal_queries_ignore_later_suffix_entries():
    f = _inputs(6, nq=4, S=6)
    a = O.attend(f["q"], f["C_k"], f["C_v"], f["beta"], f["K"], f["V"], group=2, causal=True)
    K2, V2 = f["K"].copy(), f["V"].copy()
    K2[:, -1] += 3.0      # only the last query may see the last suffix entry
    V2[:, -1] -= 2.0
    b = O.attend(f["q"], f["C_k"], f["C_v"], f["beta"], K2, V2, group=2, causal=True)
    np.testing.assert_allclose(a[:, :-1], b[:, :-1], rtol=1e-14)
    assert np.abs(a[:, -1] - b[:, -1]).max() > 1e-3
    full = O.attend(f["q"], f["C_k"], f["C_v"], f["beta"], f["K"], f["V"], group=2, causal=False)
    np.testing.assert_allclose(a[:, -1], full[:, -1], rtol=1e-13)


def test_beta_head_shaping_closed_forms():
    Zo = np.random.default_rng(0).standard_normal((2, 6, 8))
    w = np.random.default_rng(1).standard_normal(8)
    raw = np.einsum("htd,d->ht", Zo, w)
    np.testing.assert_allclose(O.beta_head(Zo, w), raw, rtol=1e-14)
    sat = O.beta_head(Zo, w, beta_max=0.5)
    assert np.abs(sat).max() < 0.5 and np.all(np.sign(sat) == np.sign(raw))
    np.testing.assert_allclose(O.beta_head(Zo * 1e-6, w, beta_max=3.0), raw * 1e-6, rtol=1e-10)
    np.testing.assert_allclose(O.beta_head(Zo, w, mass_alpha=1.0, T=800, t=100), raw + math.log(8.0), rtol=1e-14)
    np.testing.assert_allclose(O.beta_head(Zo, w, mass_alpha=0.5, log_x=math.log(1e-3), T=800, t=100),
                               raw + 0.5 * math.log(8.0) + math.log(1e-3), rtol=1e-13)
    both = O.beta_head(Zo, w, beta_max=0.5, mass_alpha=1.0, T=20, t=5)
    np.testing.assert_allclose(both, 0.5 * np.tanh(raw / 0.5) + math.log(4.0), rtol=1e-14)


@pytest.mark.parametrize("final_norm", [1, 0])
def test_beta_head_reads_the_value_heads_state(final_norm):
    """w_beta equal to row k of W_val makes beta equal to C_v[..., k]: the bias
    head sees the same final latent state (and norm) as the value head."""
    w = configs.shrink(configs.get_workload(1), n_tokens=48, t=6, final_norm=final_norm)
    cfg = w.cfg
    c = synth.as_f64(synth.make_cache(w, 0, n_tokens=48))
    wts = synth.as_f64(synth.make_weights(w, 0, t=6))
    k = 3
    Ck, Cv, pq, beta = O.compact_layer_beta(c["K"], c["V"], c["positions"], w.rope_theta, wts, cfg, 6,
                                            wts["w_val"][k])
    np.testing.assert_allclose(beta, Cv[..., k], rtol=1e-12, atol=1e-14)
    ref = compactor.compact_layer(c["K"], c["V"], c["positions"], w.rope_theta, wts, cfg, 6)
    np.testing.assert_allclose(Ck, ref[0], rtol=0, atol=0)
    np.testing.assert_allclose(Cv, ref[1], rtol=0, atol=0)


def test_query_rope_at_logical_positions_is_shift_invariant():
    """Keys stored rotated at their positions, queries rotated at their logical
    positions: moving every position by the same offset leaves the output
    unchanged (RoPE's relative-position property), and dropping the query
    rotation changes it."""
    f = _inputs(7, H=2, group=2, nq=3, t=5, S=4, d=16)
    theta = 1e4
    pc = np.array([0.0, 3.5, 7.0, 10.5, 14.0])          # compact entries at their output positions
    ps = 20.0 + np.arange(4.0)                             # suffix tokens
    pq = 24.0 + np.arange(3.0)                             # queries (logical)

    def run(shift, rotate_q=True):
        Ck = np.stack([compactor.rope(x, pc + shift, theta) for x in f["C_k"]])
        K = np.stack([compactor.rope(x, ps + shift, theta) for x in f["K"]])
        return O.attend(f["q"], Ck, f["C_v"], f["beta"], K, f["V"], group=2,
                        q_positions=(pq + shift) if rotate_q else None, rope_theta=theta)
    base = run(0.0)
    np.testing.assert_allclose(run(131072.0 - 14.0), base, rtol=1e-9, atol=1e-11)
    assert np.abs(run(0.0, rotate_q=False) - base).max() > 1e-2
