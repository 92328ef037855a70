"""still_attend_scratch (the allocation-free entry point: split partials in a
static device array) against still_attend with a caller workspace on the
same inputs: bit-identical outputs, on two calls in a row, the second with a
smaller input (the array keeps the first call's contents)."""
import pytest

from paper_2606_07878_amd import configs, synth
from tests.helpers import dev_tensor, log

pytestmark = pytest.mark.gpu


def _both(H, group, nq, t, S, d, causal, seed, rope_theta=0.0):
    import numpy as np
    import torch
    from paper_2606_07878_amd import binding
    log(f"no-alloc attend H={H} group={group} nq={nq} t={t} S={S} d={d} causal={causal} theta={rope_theta}")
    a = synth.make_attend_inputs(seed, H, group, nq, t, S, d)
    dv = {k: dev_tensor(v, configs.MODE_BF16) for k, v in a.items()}
    qpos = None
    if rope_theta:
        qpos = torch.from_numpy(1000.0 + np.arange(nq, dtype=np.float64)).cuda()
    ref = binding.attend(dv["q"], dv["C_k"], dv["C_v"], dv["beta"], dv["K"], dv["V"], group=group,
                         causal=bool(causal), q_positions=qpos, rope_theta=rope_theta)
    acfg = binding.still_attend_config(H, group, d, nq, t, S, causal, 0.0, configs.MODE_BF16, rope_theta)
    out = torch.full_like(dv["q"], float("nan"))
    stream = torch.cuda.current_stream().cuda_stream
    st = binding.still_attend_scratch(acfg, dv["q"], qpos, dv["C_k"], dv["C_v"], dv["beta"], dv["K"], dv["V"],
                                      out, stream)
    assert st == 0, binding.still_last_error()
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all()
    assert torch.equal(out, ref), f"max diff {(out.float() - ref.float()).abs().max().item():.3e}"


def test_scratch_attend_matches_workspace_attend_twice():
    _both(8, 4, 2, 1024, 64, 128, 1, seed=21)                 # decode-shaped, causal suffix
    _both(2, 2, 1, 300, 17, 64, 0, seed=22, rope_theta=1e6)   # smaller, queries rotated in-kernel


def test_scratch_attend_prefill_rows():
    _both(4, 4, 8, 655, 128, 256, 1, seed=23)                 # 32 rows per KV head (LDS kernel)
