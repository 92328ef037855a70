"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on the
same seeded inputs.  Bar: per (layer, KV head, C_k|C_v) slice,
max|y - y_oracle| / max|y_oracle| <= 2e-2 (bf16 I/O) or 1e-4 (fp32 mode)."""
import numpy as np
import pytest

from paper_2606_07878_amd import configs, synth
from tests.helpers import BF16_TOL, FP32_TOL, assert_parity, log, run_gpu, run_oracle

pytestmark = pytest.mark.gpu

W1 = configs.get_workload(1)


def _case(w, layer=0, N=None, t=None, positions=None, mode=configs.MODE_BF16, rerotate=True, heads=None,
          name=""):
    N = N if N is not None else w.n_tokens
    t = t if t is not None else w.t
    log(f"case {name}: cfg={w.name} layer={layer} N={N} t={t} mode={mode} rerotate={rerotate}")
    cache = synth.make_cache(w, layer, n_tokens=N, positions=positions)
    wts = synth.make_weights(w, layer, t=t)
    got = run_gpu(w.cfg, cache, wts, w.rope_theta, t, mode=mode, rerotate=rerotate)
    ref = run_oracle(w.cfg, cache, wts, w.rope_theta, t, rerotate=rerotate, heads=heads)
    if heads is not None:
        got = (got[0][heads], got[1][heads], got[2])
    tol = BF16_TOL if mode == configs.MODE_BF16 else FP32_TOL
    return assert_parity(got, ref, tol, what=name)


@pytest.mark.parametrize("mode", [configs.MODE_BF16, configs.MODE_FP32])
def test_config1_full(mode):
    _case(W1, mode=mode, name=f"cfg1 mode{mode}")


@pytest.mark.parametrize("N,t", [(1000, 100), (129, 7), (1, 1), (64, 1), (300, 300), (2048, 655)])
def test_config1_ragged_shapes(N, t):
    _case(W1, N=N, t=t, name=f"cfg1 N={N} t={t}")


def test_config1_positions_unsorted_fractional():
    rng = np.random.default_rng(7)
    pos = rng.permutation(np.arange(2048, dtype=np.float64)) * 0.75 + 3.25
    _case(W1, positions=pos, name="cfg1 shuffled fractional positions")


def test_config1_no_rerotate():
    _case(W1, rerotate=False, name="cfg1 no re-rotation")


@pytest.mark.parametrize("variant", ["gelu", "final_norm", "no_self", "no_ffn", "two_blocks", "resampler",
                                     "one_head"])
def test_config1_variants(variant):
    ch = {"gelu": dict(ffn_kind=configs.FFN_GELU),
          "final_norm": dict(final_norm=1),
          "no_self": dict(n_self_heads=0),
          "no_ffn": dict(ffn_kind=configs.FFN_NONE),
          "two_blocks": dict(n_blocks=2),
          "resampler": dict(n_blocks=2, cross_every_block=0),
          "one_head": dict(n_cross_heads=1, n_self_heads=1)}[variant]
    _case(configs.shrink(W1, **ch), name=f"cfg1 {variant}")


@pytest.mark.parametrize("mode", [configs.MODE_BF16, configs.MODE_FP32])
def test_config1_variants_fp32_two_blocks(mode):
    _case(configs.shrink(W1, n_blocks=2, ffn_kind=configs.FFN_GELU, final_norm=1), mode=mode,
          name=f"cfg1 two blocks gelu final-norm mode{mode}")


@pytest.mark.parametrize("wid", [2, 3])
def test_qwen_shapes_reduced_length(wid):
    """Qwen-8B-shaped compactor (D=1024, 8+8 heads, F=4096) at a reduced cache length."""
    _case(configs.get_workload(wid), N=2048 + 64 * 3, t=256, heads=[0, 5], name=f"cfg{wid} N=2240 t=256")
