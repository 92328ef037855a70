"""C-ABI contract checks that need no GPU: the library loads, exports every
function include/still.h declares, and rejects invalid arguments with the
documented status codes before enqueuing any work."""
import ctypes
import os
import re

import pytest

from paper_2606_07878_amd import binding, configs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "still.h")

FAKE = 0x10000   # never dereferenced: validation fails before any device access


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(still_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert {"still_compact_layer", "still_compact_model", "still_workspace_size"} <= set(names)
    lib = binding.lib()
    for n in names:
        assert hasattr(lib, n), f"{n} not exported"


def test_status_strings_and_version():
    for code, name in binding.STATUS.items():
        assert binding.still_status_string(code) == name
    assert "gfx950" in binding.still_version()


def _cfg(**kw):
    base = configs.get_workload(1).cfg
    c = binding.make_config(base)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


class FakeWeights:
    """still_layer_weights with fake (aligned, never dereferenced) device pointers."""

    def __init__(self, cfg, t_bank, drop=None, misalign=None):
        self.blocks = (binding.still_block_weights * cfg.n_blocks)()
        for b in range(cfg.n_blocks):
            for f, _ in binding.still_block_weights._fields_:
                setattr(self.blocks[b], f, FAKE)
        if drop:
            setattr(self.blocks[0], drop, None)
        if misalign:
            setattr(self.blocks[0], misalign, FAKE + 2)
        self.struct = binding.still_layer_weights(FAKE, t_bank, self.blocks, FAKE, FAKE)


def call(cfg, w, N=2048, t=256, K=FAKE, ws_bytes=1 << 40, flags=1, positions=FAKE, ws=FAKE):
    return binding.lib().still_compact_layer(ctypes.byref(cfg), ctypes.byref(w.struct), K, FAKE, positions, N,
                                             1e6, t, flags, FAKE, FAKE, None, ws, ws_bytes, None)


def test_workspace_size():
    c = _cfg()
    n = binding.still_workspace_size(c, 2048, 256, 1)
    assert n > 0
    assert binding.still_workspace_size(c, 4096, 256, 1) > n
    assert binding.still_workspace_size(_cfg(head_dim=96), 2048, 256, 1) == 0
    assert binding.still_workspace_size(c, 0, 256, 1) == 0
    assert binding.still_workspace_size(c, 2048, 256, 0) == 0


@pytest.mark.parametrize("kw,status", [
    (dict(mode=7), -3),
    (dict(head_dim=63), -2),
    (dict(head_dim=96), -5),
    (dict(n_kv_heads=0), -1),
    (dict(n_cross_heads=0), -1),
    (dict(ffn_kind=9), -1),
    (dict(cross_head_dim=96), -5),
    (dict(compactor_rope_base=0.0), -1),
])
def test_bad_config(kw, status):
    c = _cfg(**kw)
    assert call(c, FakeWeights(c, 256)) == status
    assert binding.still_last_error()


def test_bank_size_mismatch():
    c = _cfg()
    assert call(c, FakeWeights(c, 128)) == -2
    assert "latent bank" in binding.still_last_error()


def test_null_and_misaligned_pointers():
    c = _cfg()
    assert call(c, FakeWeights(c, 256), K=None) == -1
    assert call(c, FakeWeights(c, 256), positions=None) == -1
    assert call(c, FakeWeights(c, 256, drop="ca_wq")) == -1
    assert call(c, FakeWeights(c, 256, misalign="sa_wo")) == -1
    assert call(c, FakeWeights(c, 256), K=FAKE + 4) == -1
    # a NULL bias is allowed (zero bias): fails only later, at the workspace check
    assert call(c, FakeWeights(c, 256, drop="ca_bq"), ws_bytes=16) == -4


def test_bad_sizes_and_flags():
    c = _cfg()
    assert call(c, FakeWeights(c, 256), N=0) == -1
    assert call(c, FakeWeights(c, 0), t=0) == -1
    assert call(c, FakeWeights(c, 256), flags=0x8) == -1


def test_workspace_checks():
    c = _cfg()
    need = binding.still_workspace_size(c, 2048, 256, 1)
    assert call(c, FakeWeights(c, 256), ws_bytes=need - 1) == -4
    assert call(c, FakeWeights(c, 256), ws=None) == -4


def test_model_entry_validates_every_layer():
    c = _cfg()
    ws = [FakeWeights(c, 256), FakeWeights(c, 128)]
    arr = (binding.still_layer_weights * 2)(*[w.struct for w in ws])
    ptrs = (ctypes.c_void_p * 2)(FAKE, FAKE)
    r = binding.lib().still_compact_model(ctypes.byref(c), 2, arr, ptrs, ptrs, FAKE, 2048, 1e6, 256, 1,
                                          ptrs, ptrs, None, FAKE, 1 << 40, None)
    assert r == -2
    assert "layer 1" in binding.still_last_error()


def _beta_call(c, w_beta, beta, opts=None, ws_bytes=1 << 40):
    w = FakeWeights(c, 256)
    arr = (binding.still_layer_weights * 1)(w.struct)
    ptrs = (ctypes.c_void_p * 1)(FAKE)
    return binding.lib().still_compact_model_beta(
        ctypes.byref(c), 1, arr, ptrs, ptrs, FAKE, 2048, 1e6, 256, 1, ptrs, ptrs, None,
        w_beta, ctypes.byref(opts) if opts is not None else None, beta, FAKE, ws_bytes, None)


def test_beta_entry_validation():
    c = _cfg()
    ok = (ctypes.c_void_p * 1)(FAKE)
    assert _beta_call(c, ok, None) == -1                               # no beta outputs
    assert _beta_call(c, None, ok) == -1                               # beta without w_beta
    assert _beta_call(c, (ctypes.c_void_p * 1)(None), ok) == -1
    assert _beta_call(c, ok, (ctypes.c_void_p * 1)(FAKE + 2)) == -1    # misaligned float32 output
    assert _beta_call(c, ok, ok, binding.still_beta_opts(float("nan"), 0.0, 0.0)) == -1
    assert _beta_call(c, ok, ok, binding.still_beta_opts(2.0, 1.0, -6.9), ws_bytes=16) == -4


def _acfg(**kw):
    base = dict(n_kv_heads=8, group=4, head_dim=128, n_queries=1, t=655, n_suffix=40, causal=0, scale=0.0,
                mode=configs.MODE_BF16, rope_theta=0.0)
    base.update(kw)
    return binding.still_attend_config(*[base[f] for f, _ in binding.still_attend_config._fields_])


def _attend(c, q=FAKE, ck=FAKE, cv=FAKE, beta=FAKE, k=FAKE, v=FAKE, out=FAKE, ws=FAKE, ws_bytes=1 << 40, qpos=None):
    return binding.lib().still_attend(ctypes.byref(c), q, qpos, ck, cv, beta, k, v, out, ws, ws_bytes, None)


def test_attend_workspace_size():
    n = binding.still_attend_workspace_size(_acfg())
    assert n > 0
    assert binding.still_attend_workspace_size(_acfg(t=4 * 655)) > n
    assert binding.still_attend_workspace_size(_acfg(n_queries=9)) == 0    # 36 query rows per KV head


@pytest.mark.parametrize("kw,status", [
    (dict(mode=5), -3),
    (dict(head_dim=96), -5),
    (dict(group=0), -2),
    (dict(n_queries=9), -5),
    (dict(t=0, n_suffix=0), -2),
    (dict(t=-1), -2),
    (dict(causal=2), -1),
    (dict(causal=1, n_queries=8, group=2, n_suffix=7), -2),
    (dict(scale=float("inf")), -1),
    (dict(rope_theta=-1.0), -1),
])
def test_attend_bad_config(kw, status):
    assert _attend(_acfg(**kw)) == status
    assert binding.still_last_error()


def test_attend_pointer_and_workspace_checks():
    c = _acfg()
    assert _attend(c, q=None) == -1
    assert _attend(c, out=FAKE + 8) == -1
    assert _attend(c, ck=None) == -1                      # t > 0 needs the compact part
    assert _attend(c, k=None) == -1                       # n_suffix > 0 needs the suffix
    assert _attend(c, beta=FAKE + 2) == -1
    need = binding.still_attend_workspace_size(c)
    assert _attend(c, ws_bytes=need - 1) == -4
    assert _attend(c, ws=None) == -4
    r = _acfg(rope_theta=1e6)
    assert _attend(r) == -1                                # rotation needs the positions
    assert _attend(r, qpos=FAKE + 4) == -1                 # fp64 positions, 8-byte aligned
    assert _attend(r, qpos=FAKE, ws_bytes=16) == -4
    # NULL beta (no bias) and NULL suffix pointers with n_suffix = 0 pass validation
    c0 = _acfg(n_suffix=0)
    assert _attend(c0, beta=None, k=None, v=None, ws_bytes=16) == -4


@pytest.mark.parametrize("dc", [128, 256, 384, 512, 1024, 2048])
def test_refine_kernel_wk_rows_stay_inside_the_head(dc):
    """Host model of the W_K fragment rows the fp16 refinement kernel loads
    (refine.hpp: column tiles of 128 pairs, 32 pairs per wave, both RoPE
    members dc/2 apart; a wave with no pairs left in a tile loads the head's
    first 32 pairs).  Every row read must lie inside the cross head's dc rows,
    so no load reaches past the last head of the tiled W_K."""
    PT, hh = 128, dc // 2
    nct = (hh + PT - 1) // PT
    rows = set()
    for ct in range(nct):
        for w in range(4):
            pbase = PT * ct + 32 * w if PT * ct + 32 * w < hh else 0
            for m in range(2):
                row0 = pbase + m * hh
                rows.update(range(row0, row0 + 32))
    assert min(rows) >= 0 and max(rows) < dc
    assert rows == set(range(dc))   # and every row of the head is used


def test_attend_scratch_rejects_oversized_configuration():
    """A configuration whose split partials exceed the static scratch array is
    rejected with STILL_E_WORKSPACE before anything is enqueued (no device
    access: every pointer is fake)."""
    acfg = binding.still_attend_config(4096, 8, 256, 4, 64, 64, 0, 0.0, configs.MODE_BF16, 0.0)
    assert binding.still_attend_workspace_size(acfg) > binding.STILL_ATTEND_SCRATCH_BYTES
    st = binding.still_attend_scratch(acfg, FAKE, None, FAKE, FAKE, None, FAKE, FAKE, FAKE, None)
    assert st == -4
    assert "scratch" in binding.still_last_error()


def test_attend_scratch_size_matches_header():
    m = re.search(r"STILL_ATTEND_SCRATCH_BYTES\s*=\s*(\d+)\s*<<\s*(\d+)", open(HEADER).read())
    assert m and int(m.group(1)) << int(m.group(2)) == binding.STILL_ATTEND_SCRATCH_BYTES


def test_backward_rejects_bf16_mode_and_sizes_fp32_only():
    c16 = _cfg()
    assert binding.still_backward_workspace_size(c16, 2048, 256) == 0
    c32 = _cfg(mode=1)
    assert binding.still_backward_workspace_size(c32, 2048, 256) > 0
    w = FakeWeights(c16, 256)
    g = FakeWeights(c16, 256)
    st = binding.lib().still_compact_layer_backward(ctypes.byref(c16), ctypes.byref(w.struct), FAKE, FAKE, FAKE, 2048,
                                                    1e6, 256, 1, FAKE, FAKE, ctypes.byref(g.struct), None, None,
                                                    FAKE, 1 << 40, None)
    assert st == -5 and "FP32" in binding.still_last_error()
