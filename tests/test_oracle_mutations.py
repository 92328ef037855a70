"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake in a copy of the oracle's source (a dropped term,
a wrong sign or index, a transposed operand, a swapped weight), loads the copy
as a separate module, points the pin tests at it and requires at least one pin
to fail.  Everything runs on the CPU; the real oracle is never modified.
"""
import inspect
import types

import pytest

import oracle.compactor as oracle_compactor
from tests import test_oracle_pins as pins

SOURCE = inspect.getsource(oracle_compactor)

# (name, text in the oracle source, replacement)
MUTATIONS = [
    ("rope_rotation_sign", "[a * c - b * s, b * c + a * s]", "[a * c + b * s, b * c - a * s]"),
    ("rope_frequency_exponent", "-2.0 * j / width", "-1.0 * j / width"),
    ("rope_inverse_is_forward", "phi = -phi", "phi = phi"),
    ("rms_sum_not_mean", "np.mean(x * x, axis=-1, keepdims=True)", "np.sum(x * x, axis=-1, keepdims=True)"),
    ("l2_missing_sqrt", "np.maximum(np.sqrt(np.sum(x * x, axis=-1, keepdims=True)), eps)",
     "np.maximum(np.sum(x * x, axis=-1, keepdims=True), eps)"),
    ("softmax_global_normaliser", "e / e.sum(axis=-1, keepdims=True)", "e / e.sum()"),
    ("gelu_argument", "x / math.sqrt(2.0)", "x / 2.0"),
    ("latent_positions_step", "((hi - lo) / (t - 1))", "((hi - lo) / t)"),
    ("cross_logits_transposed", "P = softmax_rows(s * (q @ k.T))", "P = softmax_rows(s * (k @ q.T)).T"),
    ("cross_value_uses_wk", "v = X @ wv[rows].T", "v = X @ wk[rows].T"),
    ("cross_query_bias_dropped", "q_t = Q @ wq[rows].T + bq[rows]", "q_t = Q @ wq[rows].T"),
    ("cross_key_not_rotated", "k = rope(l2_normalize(k_t, cfg.l2_eps), p_k,",
     "k = rope(l2_normalize(k_t, cfg.l2_eps), 0 * p_k,"),
    ("cross_heads_share_rows", "rows = slice(i * dc, (i + 1) * dc)", "rows = slice(0, dc)"),
    ("cross_scale_sqrt", "return float(s) if s else float(_head_width(cfg, kind))",
     "return float(s) if s else float(_head_width(cfg, kind)) ** 0.5"),
    ("self_scale_dropped", "heads.append(softmax_rows(s * (q @ k.T)) @ v)",
     "heads.append(softmax_rows(q @ k.T) @ v)"),
    ("self_key_bias_dropped", "k = l2_normalize(Y @ wk[rows].T + bk[rows], cfg.l2_eps)",
     "k = l2_normalize(Y @ wk[rows].T, cfg.l2_eps)"),
    ("swiglu_gate_up_swapped", 'silu(Y @ w[f"b{block}.ffn_wg"].T) * (Y @ w[f"b{block}.ffn_wu"].T)',
     'silu(Y @ w[f"b{block}.ffn_wu"].T) * (Y @ w[f"b{block}.ffn_wg"].T)'),
    ("cross_residual_dropped", "Z = Z + cross_attention(", "Z = cross_attention("),
    ("ffn_residual_dropped", "Z = Z + ffn(", "Z = ffn("),
    ("self_input_not_normed", "self_attention(rms_norm(Z, cfg.rms_eps), w", "self_attention(Z, w"),
    ("cross_every_block_ignored", "(cfg.cross_every_block or b == 0)", "(b == 0)"),
    ("final_norm_inverted", "if cfg.final_norm else Z", "if not cfg.final_norm else Z"),
    ("keys_not_unrotated", "rope(K[h], p_k, rope_theta, inverse=True)", "K[h]"),
    ("output_heads_swapped", 'ck = Zo @ w["w_key"].T', 'ck = Zo @ w["w_val"].T'),
    ("rerotation_inverted", "ck = rope(ck, p_q, rope_theta)", "ck = rope(ck, p_q, rope_theta, inverse=True)"),
]

# Pins that exercise the compactor oracle, with their parameters.
PIN_CALLS = [
    (pins.test_rope_is_complex_rotation, dict(width=8)),
    (pins.test_rope_identities, {}),
    (pins.test_unrope_inverts_generator_rotation, {}),
    (pins.test_latent_positions, {}),
    (pins.test_elementwise_vs_torch, {}),
    (pins.test_cross_attention_matches_sdpa, {}),
    (pins.test_single_key_returns_projected_value, {}),
    (pins.test_identical_keys_give_mean_of_values, {}),
    (pins.test_joint_permutation_invariance, {}),
    *[(pins.test_qk_projection_scale_invariance, dict(which=w)) for w in ("ca_wk", "ca_wq", "sa_wk", "sa_wq")],
    (pins.test_identity_init_is_near_pass_through, dict(theta=1e4)),
    *[(pins.test_layer_matches_loop_evaluation, dict(variant=v)) for v in pins.LOOP_VARIANTS],
    (pins.test_layer_matches_loop_evaluation_no_rerotate_single_latent, {}),
]


def _mutant(old, new):
    assert SOURCE.count(old) == 1, f"mutation anchor must occur once: {old!r}"
    mod = types.ModuleType("oracle_mutant")
    exec(compile(SOURCE.replace(old, new), "oracle_mutant", "exec"), mod.__dict__)
    return mod


def test_unmutated_oracle_passes_every_pin(monkeypatch):
    monkeypatch.setattr(pins, "O", oracle_compactor)
    for fn, kw in PIN_CALLS:
        fn(**kw)


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(monkeypatch, name, old, new):
    monkeypatch.setattr(pins, "O", _mutant(old, new))
    caught = []
    for fn, kw in PIN_CALLS:
        try:
            fn(**kw)
        except Exception as e:  # an assertion, or a shape error the mistake causes
            caught.append(f"{fn.__name__}{kw}: {type(e).__name__}")
    assert caught, f"no pin catches the planted mistake {name}"


# ----------------------------------------------------------------------------
# Bias channel and consumer attention
# ----------------------------------------------------------------------------
import oracle.consumer as oracle_consumer  # noqa: E402
from tests import test_consumer_pins as cpins  # noqa: E402

CONSUMER_SOURCE = inspect.getsource(oracle_consumer)

CONSUMER_MUTATIONS = [
    ("bias_ignored", "np.zeros(t) if beta is None else np.asarray(beta[h], np.float64)", "np.zeros(t)"),
    ("bias_on_suffix_too", "np.zeros(S)])", "np.ones(S)])"),
    ("causal_excludes_diagonal", "logit[t + (S - nq + i) + 1:] = -np.inf", "logit[t + (S - nq + i):] = -np.inf"),
    ("causal_counts_from_prefix", "logit[t + (S - nq + i) + 1:] = -np.inf", "logit[(S - nq + i) + 1:] = -np.inf"),
    ("scale_without_sqrt", "(1.0 / math.sqrt(d))", "(1.0 / d)"),
    ("kv_head_interleaved", "h = hq // group", "h = hq % H"),
    ("softmax_max_normaliser", "(e @ vals) / e.sum()", "(e @ vals) / e.max()"),
    ("saturation_unscaled", "b = beta_max * np.tanh(b / beta_max)", "b = np.tanh(b)"),
    ("mass_ratio_inverted", "math.log(T / t)", "math.log(t / T)"),
    ("mass_alpha_ignored", "(mass_alpha * math.log(T / t) + log_x)", "(math.log(T / t) + log_x)"),
    ("query_rope_inverted", "compactor.rope(qh, np.asarray(q_positions, np.float64), rope_theta)",
     "compactor.rope(qh, np.asarray(q_positions, np.float64), rope_theta, inverse=True)"),
]

CONSUMER_PIN_CALLS = [
    *[(cpins.test_attend_matches_sdpa_with_additive_mask, dict(group=g, causal=c))
      for g, c in [(1, False), (2, False), (2, True), (3, True)]],
    (cpins.test_attend_explicit_scale_matches_sdpa, {}),
    (cpins.test_log_count_bias_equals_duplicated_entries, {}),
    (cpins.test_uniform_bias_on_empty_suffix_cancels, {}),
    (cpins.test_single_visible_entry_returns_its_value, {}),
    (cpins.test_causal_queries_ignore_later_suffix_entries, {}),
    (cpins.test_beta_head_shaping_closed_forms, {}),
    *[(cpins.test_beta_head_reads_the_value_heads_state, dict(final_norm=f)) for f in (1, 0)],
    (cpins.test_query_rope_at_logical_positions_is_shift_invariant, {}),
]


def _consumer_mutant(old, new):
    assert CONSUMER_SOURCE.count(old) == 1, f"mutation anchor must occur once: {old!r}"
    mod = types.ModuleType("oracle_consumer_mutant")
    mod.__dict__["__package__"] = "oracle"
    exec(compile(CONSUMER_SOURCE.replace(old, new), "oracle_consumer_mutant", "exec"), mod.__dict__)
    return mod


def test_unmutated_consumer_oracle_passes_every_pin(monkeypatch):
    monkeypatch.setattr(cpins, "O", oracle_consumer)
    for fn, kw in CONSUMER_PIN_CALLS:
        fn(**kw)


@pytest.mark.parametrize("name,old,new", CONSUMER_MUTATIONS, ids=[m[0] for m in CONSUMER_MUTATIONS])
def test_planted_consumer_mistake_is_caught(monkeypatch, name, old, new):
    monkeypatch.setattr(cpins, "O", _consumer_mutant(old, new))
    caught = []
    for fn, kw in CONSUMER_PIN_CALLS:
        try:
            fn(**kw)
        except Exception as e:
            caught.append(f"{fn.__name__}{kw}: {type(e).__name__}")
    assert caught, f"no pin catches the planted mistake {name}"
