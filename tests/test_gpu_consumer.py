"""GPU parity of the bias head (still_compact_model_beta) and of attention over
a compacted prefix with bias (still_attend) against the fp64 oracle.

Bars:
* bias head: per (layer, KV head) slice, max|beta - beta_oracle| /
  max|beta_oracle| <= 2e-2 (bf16 I/O) or 1e-4 (fp32 mode), the compaction's
  own bars, since beta reads the same final latent state as C_v.
* attention: the kernel takes its operands as given and accumulates in fp32,
  so in bf16 mode the output's rounding to bf16 (relative 2^-9 per element)
  dominates: per query-head slice max|o - o_oracle| / max|o_oracle| <= 8e-3;
  fp32 mode <= 1e-5.
"""
import math

import numpy as np
import pytest

from paper_2606_07878_amd import configs, synth
from tests.helpers import BF16_TOL, FP32_TOL, dev_tensor, log, slice_errors, weights_to_device

pytestmark = pytest.mark.gpu

ATT_TOL = {configs.MODE_BF16: 8e-3, configs.MODE_FP32: 1e-5}


def _attend_case(H, group, nq, t, S, d, causal, mode, beta=True, scale=0.0, seed=11, qpos0=None, theta=1e6):
    import torch
    from oracle import consumer
    from paper_2606_07878_amd import binding
    name = (f"attend H={H} group={group} nq={nq} t={t} S={S} d={d} causal={causal} beta={beta} mode={mode} "
            f"qpos0={qpos0}")
    log(name)
    a = synth.make_attend_inputs(seed, H, group, nq, t, S, d, beta=beta)
    f = synth.as_f64(a)
    qpos = None if qpos0 is None else qpos0 + np.arange(nq, dtype=np.float64)
    ref = consumer.attend(f["q"], f["C_k"], f["C_v"], None if a["beta"] is None else a["beta"].astype(np.float64),
                          f["K"], f["V"], group=group, causal=causal, scale=scale or None,
                          q_positions=qpos, rope_theta=theta)
    dv = {k: (dev_tensor(v, mode) if v is not None else None) for k, v in a.items()}
    out = binding.attend(dv["q"], dv["C_k"] if t else None, dv["C_v"] if t else None, dv["beta"] if t else None,
                         dv["K"] if S else None, dv["V"] if S else None, group=group, causal=causal, scale=scale,
                         q_positions=None if qpos is None else torch.from_numpy(qpos).cuda(), rope_theta=theta)
    torch.cuda.synchronize()
    got = out.double().cpu().numpy()
    assert np.all(np.isfinite(got)), "non-finite output"
    err = slice_errors(got, ref).max()
    log(f"  max slice rel err {err:.3e} (tol {ATT_TOL[mode]:g})")
    assert err <= ATT_TOL[mode], f"{name}: slice error {err:.3e}"


@pytest.mark.parametrize("mode", [configs.MODE_BF16, configs.MODE_FP32])
def test_attend_decode_gqa(mode):
    """Decode step of a Qwen3-8B-shaped layer (8 KV heads, 4 query heads each, d=128)
    over a 200x-compacted 128k prefix (t=655) plus 37 fresh tokens."""
    _attend_case(8, 4, 1, 655, 37, 128, False, mode)


@pytest.mark.parametrize("mode", [configs.MODE_BF16, configs.MODE_FP32])
def test_attend_causal_prefill(mode):
    _attend_case(2, 4, 8, 300, 200, 64, True, mode)


def test_attend_max_rows_no_suffix_no_bias():
    """32 query rows per KV head (the maximum), d=256 (Gemma-3 width), compact part only."""
    _attend_case(4, 2, 16, 1000, 0, 256, False, configs.MODE_BF16, beta=False)


def test_attend_no_compact_part_causal():
    _attend_case(2, 1, 32, 0, 513, 128, True, configs.MODE_BF16)


def test_attend_many_splits_explicit_scale():
    _attend_case(8, 8, 4, 5000, 17, 128, False, configs.MODE_BF16, scale=0.05)


def test_attend_single_entry():
    _attend_case(1, 1, 1, 1, 0, 64, False, configs.MODE_FP32)


@pytest.mark.parametrize("mode,final_norm", [(configs.MODE_BF16, 0), (configs.MODE_BF16, 1),
                                             (configs.MODE_FP32, 1)])
def test_beta_head_two_layers(mode, final_norm):
    """Two layers through still_compact_model_beta with saturation and learnable
    mass matching on (beta_max=2, mass_alpha=0.5, x=1e-3)."""
    import torch
    from oracle import consumer
    from paper_2606_07878_amd import binding
    w = configs.shrink(configs.get_workload(1), final_norm=final_norm)
    N, t, L = 1500, 150, 2
    opts = dict(beta_max=2.0, mass_alpha=0.5, log_x=math.log(1e-3))
    log(f"beta head cfg1 N={N} t={t} layers={L} mode={mode} final_norm={final_norm} {opts}")
    caches = [synth.make_cache(w, l, n_tokens=N) for l in range(L)]
    wts = [synth.make_weights(w, l, t=t) for l in range(L)]
    wb = [synth.make_beta_weight(w, l) for l in range(L)]
    K = [dev_tensor(c["K"], mode) for c in caches]
    V = [dev_tensor(c["V"], mode) for c in caches]
    pos = torch.from_numpy(caches[0]["positions"]).cuda()
    Ck, Cv, _, betas = binding.compact_model_beta(w.cfg, [weights_to_device(x, mode) for x in wts], K, V, pos,
                                                  w.rope_theta, t, [dev_tensor(b, mode) for b in wb], mode=mode,
                                                  **opts)
    torch.cuda.synchronize()
    tol = BF16_TOL if mode == configs.MODE_BF16 else FP32_TOL
    for l in range(L):
        c64, w64 = synth.as_f64(caches[l]), synth.as_f64(wts[l])
        _, rv, _, rb = consumer.compact_layer_beta(c64["K"], c64["V"], c64["positions"], w.rope_theta, w64, w.cfg,
                                                   t, synth.bf16_value(wb[l]), **opts)
        off = opts["mass_alpha"] * math.log(N / t) + opts["log_x"]
        got = betas[l].double().cpu().numpy()
        # error relative to the learned (shaped, pre-offset) part, so the constant offset cannot hide it
        eb = (np.abs(got - rb).max(axis=1) / np.abs(rb - off).max(axis=1)).max()
        ev = slice_errors(Cv[l].double().cpu().numpy(), rv).max()
        log(f"  layer {l}: beta max slice rel err {eb:.3e}, C_v {ev:.3e}, |beta - offset| max "
            f"{np.abs(rb - off).max():.3f}")
        assert np.all(np.isfinite(got))
        assert np.abs(rb - off).max() > 0.1, "the learned part of the bias should not be negligible"
        assert eb <= tol, f"layer {l}: beta slice error {eb:.3e} > {tol}"
        assert ev <= tol


@pytest.mark.parametrize("group,nq,d", [(2, 4, 128), (4, 4, 64), (8, 2, 256), (3, 3, 128)])
def test_attend_row_bands_causal(group, nq, d):
    """Query-row counts R = group * n_queries in each register band (<= 4, 8, 16, 32)."""
    _attend_case(3, group, nq, 777, 129, d, True, configs.MODE_BF16)


@pytest.mark.parametrize("group,nq,t,S,d,mode", [
    (2, 1, 1024, 64, 256, configs.MODE_BF16),     # Gemma-shaped decode: 2 query heads per KV head, d=256
    (2, 1, 1024, 64, 256, configs.MODE_FP32),
    (8, 1, 5000, 3, 64, configs.MODE_BF16),       # 8 rows, many chunks and splits
    (1, 2, 37, 5, 128, configs.MODE_BF16),        # fewer entries than one chunk in each part
])
def test_attend_decode_rows(group, nq, t, S, d, mode):
    _attend_case(4, group, nq, t, S, d, False, mode)


def test_attend_graph_replays_match_eager():
    """The decode calls captured in a HIP graph (as the benchmark times them) give,
    on every replay, the eager result bit for bit."""
    import torch
    from paper_2606_07878_amd import binding
    a = synth.make_attend_inputs(21, 8, 4, 1, 655, 64, 128)
    dv = {k: dev_tensor(v, configs.MODE_BF16) for k, v in a.items()}
    ws = torch.empty(1 << 22, dtype=torch.uint8, device="cuda")
    qs = [dv["q"] * (1.0 + 0.25 * i) for i in range(3)]
    eager = [binding.attend(qs[i], dv["C_k"], dv["C_v"], dv["beta"], dv["K"], dv["V"], group=4, workspace=ws)
             for i in range(3)]
    outs = [torch.empty_like(q) for q in qs]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for i in range(3):
                binding.attend(qs[i], dv["C_k"], dv["C_v"], dv["beta"], dv["K"], dv["V"], group=4, workspace=ws,
                               out=outs[i])
    torch.cuda.current_stream().wait_stream(s)
    for rep in range(3):
        for o in outs:
            o.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        other = binding.attend(qs[0], dv["C_k"], dv["C_v"], None, dv["K"], dv["V"], group=4, workspace=ws)
        torch.cuda.synchronize()
        assert torch.isfinite(other.float()).all()
        for i in range(3):
            assert torch.equal(outs[i], eager[i]), f"replay {rep}, call {i} differs from eager"


@pytest.mark.parametrize("group,nq,d,mode", [(4, 1, 128, configs.MODE_BF16), (4, 1, 128, configs.MODE_FP32),
                                             (2, 3, 256, configs.MODE_BF16), (4, 8, 64, configs.MODE_FP32),
                                             (3, 5, 128, configs.MODE_BF16)])
def test_attend_query_rope_at_logical_positions(group, nq, d, mode):
    """Queries rotated inside the kernel at logical positions past a 128k
    original prefix (offset T - t carried by the compact cache); both kernels
    (<= 8 and > 8 query rows)."""
    _attend_case(2, group, nq, 655, 40, d, True, mode, qpos0=131072.0 + 40 - nq)
