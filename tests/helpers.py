"""Shared test plumbing: move synthetic inputs to the GPU, run the library
through the C ABI, run the oracle on the same inputs, compare."""
from __future__ import annotations

import sys
import time

import numpy as np

from paper_2606_07878_amd import configs, synth

BF16_TOL = 2e-2    # max relative error per (layer, KV head, C_k|C_v) slice, bf16 I/O
FP32_TOL = 1e-4    # same, fp32 validation mode


def log(msg: str):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)
    sys.stdout.flush()


def dev_tensor(arr: np.ndarray, mode: int, device="cuda"):
    """uint16 bf16 bits -> bf16 tensor (bf16 mode) or float32 tensor of the same values."""
    import torch
    if arr.dtype == np.uint16:
        t = torch.from_numpy(arr.view(np.int16).copy()).view(torch.bfloat16)
        if mode == configs.MODE_FP32:
            t = t.float()
    else:
        t = torch.from_numpy(np.ascontiguousarray(arr))
        t = t.float() if (mode == configs.MODE_FP32 and t.dtype == torch.float64) else t
    return t.to(device)


def weights_to_device(wts: dict, mode: int, device="cuda") -> dict:
    return {k: dev_tensor(v, mode, device) for k, v in wts.items()}


def run_gpu(cfg, cache: dict, wts: dict, rope_theta: float, t: int, mode: int = configs.MODE_BF16,
            rerotate: bool = True, device="cuda"):
    """Compact one layer on the GPU through still_compact_layer; float64 numpy outputs."""
    import torch
    from paper_2606_07878_amd import binding
    K = dev_tensor(cache["K"], mode, device)
    V = dev_tensor(cache["V"], mode, device)
    pos = torch.from_numpy(cache["positions"]).to(device)
    W = weights_to_device(wts, mode, device)
    Ck, Cv, p = binding.compact_layer(cfg, W, K, V, pos, rope_theta, t, rerotate=rerotate, mode=mode)
    torch.cuda.synchronize()
    return (Ck.double().cpu().numpy(), Cv.double().cpu().numpy(), p.cpu().numpy())


def run_oracle(cfg, cache: dict, wts: dict, rope_theta: float, t: int, rerotate: bool = True, heads=None):
    from oracle import compactor
    c64 = synth.as_f64(cache)
    w64 = synth.as_f64(wts)
    return compactor.compact_layer(c64["K"], c64["V"], c64["positions"], rope_theta, w64, cfg, t,
                                   rerotate=rerotate, heads=heads)


def slice_errors(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """max|y - y_ref| / max|y_ref| per leading-axis slice (one KV head)."""
    g = got.reshape(got.shape[0], -1)
    r = ref.reshape(ref.shape[0], -1)
    return np.abs(g - r).max(axis=1) / np.maximum(np.abs(r).max(axis=1), 1e-30)


def assert_parity(got, ref, tol: float, what: str = ""):
    Ck, Cv, p = got
    Rk, Rv, rp = ref
    ek, ev = slice_errors(Ck, Rk), slice_errors(Cv, Rv)
    log(f"{what} max slice rel err: C_k {ek.max():.3e}  C_v {ev.max():.3e}  (tol {tol:g})")
    assert np.all(np.isfinite(Ck)) and np.all(np.isfinite(Cv)), "non-finite output"
    np.testing.assert_allclose(p, rp, rtol=1e-12, atol=1e-9)
    assert ek.max() <= tol, f"C_k slice error {ek.max():.3e} > {tol}"
    assert ev.max() <= tol, f"C_v slice error {ev.max():.3e} > {tol}"
    return ek.max(), ev.max()
