"""ctypes binding of libstill.so (include/still.h).

Argument marshalling only: torch tensors supply device pointers and the
current HIP stream; every step of the compaction runs in the library's HIP
kernels.  There is no fallback: if the library is missing or fails to load,
every entry point raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence

from . import configs

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libstill.so")

STILL_OK = 0
STATUS = {0: "STILL_OK", -1: "STILL_E_INVAL", -2: "STILL_E_SHAPE", -3: "STILL_E_DTYPE",
          -4: "STILL_E_WORKSPACE", -5: "STILL_E_UNSUPPORTED", -6: "STILL_E_HIP"}
STILL_F_REROTATE = 1


class StillError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{STATUS.get(status, status)}: {detail}")
        self.status = status


class still_config(ctypes.Structure):
    _fields_ = [("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("latent_dim", ctypes.c_int32), ("n_blocks", ctypes.c_int32),
                ("cross_every_block", ctypes.c_int32), ("n_cross_heads", ctypes.c_int32),
                ("cross_head_dim", ctypes.c_int32), ("n_self_heads", ctypes.c_int32),
                ("self_head_dim", ctypes.c_int32), ("ffn_kind", ctypes.c_int32),
                ("ffn_hidden", ctypes.c_int32), ("final_norm", ctypes.c_int32),
                ("logit_scale_cross", ctypes.c_float), ("logit_scale_self", ctypes.c_float),
                ("compactor_rope_base", ctypes.c_double), ("rms_eps", ctypes.c_float),
                ("l2_eps", ctypes.c_float), ("mode", ctypes.c_int32)]


_BLOCK_FIELDS = ["ca_wq", "ca_bq", "ca_wk", "ca_bk", "ca_wv", "ca_wo",
                 "sa_wq", "sa_bq", "sa_wk", "sa_bk", "sa_wv", "sa_wo",
                 "ffn_wg", "ffn_wu", "ffn_wd"]


class still_block_weights(ctypes.Structure):
    _fields_ = [(f, ctypes.c_void_p) for f in _BLOCK_FIELDS]


class still_layer_weights(ctypes.Structure):
    _fields_ = [("latents", ctypes.c_void_p), ("t_bank", ctypes.c_int32),
                ("blocks", ctypes.POINTER(still_block_weights)),
                ("w_key", ctypes.c_void_p), ("w_val", ctypes.c_void_p)]


class still_beta_opts(ctypes.Structure):
    _fields_ = [("beta_max", ctypes.c_float), ("mass_alpha", ctypes.c_float), ("log_x", ctypes.c_float)]


class still_attend_config(ctypes.Structure):
    _fields_ = [("n_kv_heads", ctypes.c_int32), ("group", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("n_queries", ctypes.c_int32), ("t", ctypes.c_int32), ("n_suffix", ctypes.c_int32),
                ("causal", ctypes.c_int32), ("scale", ctypes.c_float), ("mode", ctypes.c_int32),
                ("rope_theta", ctypes.c_double)]


_lib = None


def lib():
    """Load libstill.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                               "`python -m paper_2606_07878_amd.build` (no CPU fallback exists)")
        L = ctypes.CDLL(_LIB_PATH)
        L.still_workspace_size.argtypes = [ctypes.POINTER(still_config), ctypes.c_int64, ctypes.c_int32,
                                           ctypes.c_int32]
        L.still_workspace_size.restype = ctypes.c_size_t
        common = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_double, ctypes.c_int32, ctypes.c_uint32]
        L.still_compact_layer.argtypes = [ctypes.POINTER(still_config), ctypes.POINTER(still_layer_weights),
                                          ctypes.c_void_p, ctypes.c_void_p, *common,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
        L.still_compact_layer.restype = ctypes.c_int32
        L.still_compact_model.argtypes = [ctypes.POINTER(still_config), ctypes.c_int32,
                                          ctypes.POINTER(still_layer_weights),
                                          ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(ctypes.c_void_p),
                                          *common,
                                          ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(ctypes.c_void_p),
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
        L.still_compact_model.restype = ctypes.c_int32
        L.still_compact_model_beta.argtypes = [*L.still_compact_model.argtypes[:13],
                                               ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(still_beta_opts),
                                               ctypes.POINTER(ctypes.c_void_p),
                                               ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
        L.still_compact_model_beta.restype = ctypes.c_int32
        L.still_attend_workspace_size.argtypes = [ctypes.POINTER(still_attend_config)]
        L.still_attend_workspace_size.restype = ctypes.c_size_t
        L.still_attend.argtypes = [ctypes.POINTER(still_attend_config), *[ctypes.c_void_p] * 9, ctypes.c_size_t,
                                   ctypes.c_void_p]
        L.still_attend.restype = ctypes.c_int32
        L.still_backward_workspace_size.argtypes = [ctypes.POINTER(still_config), ctypes.c_int64, ctypes.c_int32]
        L.still_backward_workspace_size.restype = ctypes.c_size_t
        L.still_compact_layer_backward.argtypes = [ctypes.POINTER(still_config),
                                                   ctypes.POINTER(still_layer_weights), ctypes.c_void_p,
                                                   ctypes.c_void_p, *common, ctypes.c_void_p, ctypes.c_void_p,
                                                   ctypes.POINTER(still_layer_weights), ctypes.c_void_p,
                                                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                                   ctypes.c_void_p]
        L.still_compact_layer_backward.restype = ctypes.c_int32
        L.still_attend_scratch.argtypes = [ctypes.POINTER(still_attend_config), *[ctypes.c_void_p] * 9]
        L.still_attend_scratch.restype = ctypes.c_int32
        L.still_status_string.argtypes = [ctypes.c_int32]
        L.still_status_string.restype = ctypes.c_char_p
        L.still_last_error.argtypes = []
        L.still_last_error.restype = ctypes.c_char_p
        L.still_version.argtypes = []
        L.still_version.restype = ctypes.c_char_p
        L.still_timing_enable.argtypes = [ctypes.c_int32]
        L.still_timing_enable.restype = ctypes.c_int32
        L.still_timing_reset.argtypes = []
        L.still_timing_reset.restype = ctypes.c_int32
        L.still_timing_read.argtypes = [ctypes.c_int32, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_int64)]
        L.still_timing_read.restype = ctypes.c_int32
        _lib = L
    return _lib


def make_config(cfg: configs.CompactorConfig, mode: int = configs.MODE_BF16) -> still_config:
    return still_config(cfg.n_kv_heads, cfg.head_dim, cfg.latent_dim, cfg.n_blocks, cfg.cross_every_block,
                        cfg.n_cross_heads, cfg.cross_head_dim, cfg.n_self_heads, cfg.self_head_dim,
                        cfg.ffn_kind, cfg.ffn_hidden, cfg.final_norm, cfg.logit_scale_cross,
                        cfg.logit_scale_self, cfg.compactor_rope_base, cfg.rms_eps, cfg.l2_eps, mode)


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    return x.data_ptr() if hasattr(x, "data_ptr") else int(x)


class LayerWeights:
    """still_layer_weights built from a dict of device tensors keyed like
    ``configs.layer_shapes`` (keeps the tensors alive)."""

    def __init__(self, cfg: configs.CompactorConfig, tensors: Dict[str, object]):
        self.tensors = tensors
        nb = cfg.n_blocks
        self._blocks = (still_block_weights * nb)()
        for b in range(nb):
            for f in _BLOCK_FIELDS:
                setattr(self._blocks[b], f, _ptr(tensors.get(f"b{b}.{f}")))
        lat = tensors["latents"]
        self.struct = still_layer_weights(_ptr(lat), int(lat.shape[1]), self._blocks,
                                          _ptr(tensors["w_key"]), _ptr(tensors["w_val"]))


def _check(status: int):
    if status != STILL_OK:
        raise StillError(status, lib().still_last_error().decode())


def still_workspace_size(cfg: still_config, N: int, t: int, n_layers: int = 1) -> int:
    return int(lib().still_workspace_size(ctypes.byref(cfg), N, t, n_layers))


def still_compact_layer(cfg: still_config, w: LayerWeights, K, V, positions, N: int, rope_theta: float,
                        t: int, flags: int, C_k, C_v, out_positions, workspace, workspace_bytes: int,
                        stream) -> int:
    """Raw entry point (pointers or tensors); returns the status code."""
    return lib().still_compact_layer(ctypes.byref(cfg), ctypes.byref(w.struct), _ptr(K), _ptr(V),
                                     _ptr(positions), N, rope_theta, t, flags, _ptr(C_k), _ptr(C_v),
                                     _ptr(out_positions), _ptr(workspace), workspace_bytes, _ptr(stream))


def still_compact_model(cfg: still_config, ws: Sequence[LayerWeights], K: Sequence, V: Sequence, positions,
                        N: int, rope_theta: float, t: int, flags: int, C_k: Sequence, C_v: Sequence,
                        out_positions, workspace, workspace_bytes: int, stream) -> int:
    L = len(ws)
    wa = (still_layer_weights * L)(*[w.struct for w in ws])
    arr = lambda xs: (ctypes.c_void_p * L)(*[_ptr(x) for x in xs])  # noqa: E731
    return lib().still_compact_model(ctypes.byref(cfg), L, wa, arr(K), arr(V), _ptr(positions), N,
                                     rope_theta, t, flags, arr(C_k), arr(C_v), _ptr(out_positions),
                                     _ptr(workspace), workspace_bytes, _ptr(stream))


def still_compact_model_beta(cfg: still_config, ws: Sequence[LayerWeights], K: Sequence, V: Sequence, positions,
                             N: int, rope_theta: float, t: int, flags: int, C_k: Sequence, C_v: Sequence,
                             out_positions, w_beta: Sequence, beta_opts: Optional[still_beta_opts],
                             beta: Sequence, workspace, workspace_bytes: int, stream) -> int:
    L = len(ws)
    wa = (still_layer_weights * L)(*[w.struct for w in ws])
    arr = lambda xs: (ctypes.c_void_p * L)(*[_ptr(x) for x in xs])  # noqa: E731
    return lib().still_compact_model_beta(ctypes.byref(cfg), L, wa, arr(K), arr(V), _ptr(positions), N,
                                          rope_theta, t, flags, arr(C_k), arr(C_v), _ptr(out_positions),
                                          arr(w_beta), ctypes.byref(beta_opts) if beta_opts is not None else None,
                                          arr(beta), _ptr(workspace), workspace_bytes, _ptr(stream))


def still_attend_workspace_size(cfg: still_attend_config) -> int:
    return int(lib().still_attend_workspace_size(ctypes.byref(cfg)))


def still_attend(cfg: still_attend_config, q, q_positions, C_k, C_v, beta, K, V, out, workspace,
                 workspace_bytes: int, stream) -> int:
    """Raw entry point (pointers or tensors); returns the status code."""
    return lib().still_attend(ctypes.byref(cfg), _ptr(q), _ptr(q_positions), _ptr(C_k), _ptr(C_v), _ptr(beta),
                              _ptr(K), _ptr(V), _ptr(out), _ptr(workspace), workspace_bytes, _ptr(stream))


def still_attend_scratch(cfg: still_attend_config, q, q_positions, C_k, C_v, beta, K, V, out, stream) -> int:
    """Raw entry point of the allocation-free attention (no workspace argument);
    returns the status code."""
    return lib().still_attend_scratch(ctypes.byref(cfg), _ptr(q), _ptr(q_positions), _ptr(C_k), _ptr(C_v),
                                      _ptr(beta), _ptr(K), _ptr(V), _ptr(out), _ptr(stream))


STILL_ATTEND_SCRATCH_BYTES = 68 << 20


def still_status_string(status: int) -> str:
    return lib().still_status_string(status).decode()


def still_last_error() -> str:
    return lib().still_last_error().decode()


def still_version() -> str:
    return lib().still_version().decode()


# kernel classes of the timing facility (still.h)
KERNEL_CLASSES = {"cross_attn": 0, "kproj": 1, "qproj": 2, "refine": 3, "latent": 4, "other": 5, "attend": 6,
                  "stage": 7}


def still_timing_enable(class_mask: int) -> None:
    """Record hipEvent pairs around launches of the classes in class_mask (0 = off)."""
    _check(lib().still_timing_enable(int(class_mask)))


def still_timing_reset() -> None:
    _check(lib().still_timing_reset())


def still_timing_read(kernel_class: int):
    """(total ms, launches) of one kernel class since the last reset."""
    ms = ctypes.c_double()
    n = ctypes.c_int64()
    _check(lib().still_timing_read(kernel_class, ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


# ----------------------------------------------------------------------------
# torch conveniences (allocation of outputs / workspace on the caller's device)
# ----------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def compact_model(cfg: configs.CompactorConfig, weights: List[Dict[str, object]], K: List, V: List, positions,
                  rope_theta: float, t: int, rerotate: bool = True, mode: int = configs.MODE_BF16,
                  workspace=None, outputs=None):
    """Compact L layers on the current stream; returns ([C_k], [C_v], out_positions)."""
    torch = _torch()
    dev = K[0].device
    ccfg = make_config(cfg, mode)
    N = int(K[0].shape[1])
    L = len(K)
    need = still_workspace_size(ccfg, N, t, L)
    if need == 0:
        raise StillError(-5, "configuration rejected by still_workspace_size")
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    dt = K[0].dtype
    if outputs is None:
        Ck = [torch.empty(cfg.n_kv_heads, t, cfg.head_dim, dtype=dt, device=dev) for _ in range(L)]
        Cv = [torch.empty(cfg.n_kv_heads, t, cfg.head_dim, dtype=dt, device=dev) for _ in range(L)]
    else:
        Ck, Cv = outputs
    outp = torch.empty(t, dtype=torch.float64, device=dev)
    lw = [w if isinstance(w, LayerWeights) else LayerWeights(cfg, w) for w in weights]
    stream = torch.cuda.current_stream(dev).cuda_stream
    _check(still_compact_model(ccfg, lw, K, V, positions, N, rope_theta, t,
                               STILL_F_REROTATE if rerotate else 0, Ck, Cv, outp, workspace,
                               workspace.numel(), stream))
    return Ck, Cv, outp


def compact_layer(cfg: configs.CompactorConfig, weights: Dict[str, object], K, V, positions, rope_theta: float,
                  t: int, rerotate: bool = True, mode: int = configs.MODE_BF16, workspace=None):
    """Compact one layer through still_compact_layer; returns (C_k, C_v, out_positions)."""
    torch = _torch()
    dev = K.device
    ccfg = make_config(cfg, mode)
    N = int(K.shape[1])
    need = still_workspace_size(ccfg, N, t, 1)
    if need == 0:
        raise StillError(-5, "configuration rejected by still_workspace_size")
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    Ck = torch.empty(cfg.n_kv_heads, t, cfg.head_dim, dtype=K.dtype, device=dev)
    Cv = torch.empty_like(Ck)
    outp = torch.empty(t, dtype=torch.float64, device=dev)
    lw = weights if isinstance(weights, LayerWeights) else LayerWeights(cfg, weights)
    stream = torch.cuda.current_stream(dev).cuda_stream
    _check(still_compact_layer(ccfg, lw, K, V, positions, N, rope_theta, t,
                               STILL_F_REROTATE if rerotate else 0, Ck, Cv, outp, workspace,
                               workspace.numel(), stream))
    return Ck, Cv, outp


def still_backward_workspace_size(cfg: still_config, N: int, t: int) -> int:
    return int(lib().still_backward_workspace_size(ctypes.byref(cfg), N, t))


def still_compact_layer_backward(cfg: still_config, w: LayerWeights, K, V, positions, N: int, rope_theta: float,
                                 t: int, flags: int, dC_k, dC_v, grad: LayerWeights, C_k, C_v, workspace,
                                 workspace_bytes: int, stream) -> int:
    """Raw entry point (pointers or tensors); returns the status code."""
    return lib().still_compact_layer_backward(ctypes.byref(cfg), ctypes.byref(w.struct), _ptr(K), _ptr(V),
                                              _ptr(positions), N, rope_theta, t, flags, _ptr(dC_k), _ptr(dC_v),
                                              ctypes.byref(grad.struct), _ptr(C_k), _ptr(C_v), _ptr(workspace),
                                              workspace_bytes, _ptr(stream))


def compact_layer_backward(cfg: configs.CompactorConfig, weights: Dict[str, object], K, V, positions,
                           rope_theta: float, t: int, dC_k, dC_v, rerotate: bool = True, workspace=None):
    """Gradients of <dC_k, C_k> + <dC_v, C_v> w.r.t. every compactor tensor
    (fp32 mode) through still_compact_layer_backward; returns (grads dict
    keyed like ``weights``, C_k, C_v) as float32 tensors on K's device."""
    torch = _torch()
    dev = K.device
    ccfg = make_config(cfg, configs.MODE_FP32)
    N = int(K.shape[1])
    need = still_backward_workspace_size(ccfg, N, t)
    if need == 0:
        raise StillError(-5, "configuration rejected by still_backward_workspace_size")
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    grads = {k: torch.empty(tuple(v.shape), dtype=torch.float32, device=dev) for k, v in weights.items()}
    Ck = torch.empty(cfg.n_kv_heads, t, cfg.head_dim, dtype=torch.float32, device=dev)
    Cv = torch.empty_like(Ck)
    lw = weights if isinstance(weights, LayerWeights) else LayerWeights(cfg, weights)
    gw = LayerWeights(cfg, grads)
    stream = torch.cuda.current_stream(dev).cuda_stream
    _check(still_compact_layer_backward(ccfg, lw, K, V, positions, N, rope_theta, t,
                                        STILL_F_REROTATE if rerotate else 0, dC_k, dC_v, gw, Ck, Cv, workspace,
                                        workspace.numel(), stream))
    return grads, Ck, Cv


def compact_subrange(cfg: configs.CompactorConfig, weights: Dict[str, object], K, V, positions, rope_theta: float,
                     t: int, start: int, end: int, rerotate: bool = True, mode: int = configs.MODE_BF16):
    """Compact only the cache entries [start, end) of one layer (to t) and
    splice the preserved prefix and suffix back around them: returns
    (K', V', positions') with N - (end - start) + t entries.  The compaction
    runs through still_compact_layer; slicing and concatenation are copies."""
    torch = _torch()
    N = int(K.shape[1])
    if not (0 <= start < end <= N):
        raise StillError(-1, f"subrange [{start}, {end}) outside [0, {N})")
    Ck, Cv, pq = compact_layer(cfg, weights, K[:, start:end].contiguous(), V[:, start:end].contiguous(),
                               positions[start:end].contiguous(), rope_theta, t, rerotate=rerotate, mode=mode)
    return (torch.cat([K[:, :start], Ck, K[:, end:]], dim=1), torch.cat([V[:, :start], Cv, V[:, end:]], dim=1),
            torch.cat([positions[:start], pq, positions[end:]]))


def compact_chunks(cfg: configs.CompactorConfig, weights: Dict[str, object], K, V, positions, rope_theta: float,
                   t: int, chunk: int, rerotate: bool = True, mode: int = configs.MODE_BF16):
    """Independent chunk compaction: consecutive chunks of `chunk` entries (the
    last may be shorter) are each compacted to t by still_compact_layer and
    the compact chunks concatenated in order."""
    torch = _torch()
    N = int(K.shape[1])
    if chunk < 1:
        raise StillError(-1, "chunk must be >= 1")
    lw = weights if isinstance(weights, LayerWeights) else LayerWeights(cfg, weights)
    need = still_workspace_size(make_config(cfg, mode), min(chunk, N), t, 1)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=K.device)   # shared by the chunks (one stream)
    outs = [compact_layer(cfg, lw, K[:, a:a + chunk].contiguous(), V[:, a:a + chunk].contiguous(),
                          positions[a:a + chunk].contiguous(), rope_theta, t, rerotate=rerotate, mode=mode,
                          workspace=ws)
            for a in range(0, N, chunk)]
    return (torch.cat([o[0] for o in outs], dim=1), torch.cat([o[1] for o in outs], dim=1),
            torch.cat([o[2] for o in outs]))


def compact_model_beta(cfg: configs.CompactorConfig, weights: List[Dict[str, object]], K: List, V: List,
                       positions, rope_theta: float, t: int, w_beta: List, beta_max: float = 0.0,
                       mass_alpha: float = 0.0, log_x: float = 0.0, rerotate: bool = True,
                       mode: int = configs.MODE_BF16, workspace=None):
    """compact_model plus the bias head: returns ([C_k], [C_v], out_positions, [beta [H, t] float32])."""
    torch = _torch()
    dev = K[0].device
    ccfg = make_config(cfg, mode)
    N = int(K[0].shape[1])
    L = len(K)
    need = still_workspace_size(ccfg, N, t, L)
    if need == 0:
        raise StillError(-5, "configuration rejected by still_workspace_size")
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    dt = K[0].dtype
    Ck = [torch.empty(cfg.n_kv_heads, t, cfg.head_dim, dtype=dt, device=dev) for _ in range(L)]
    Cv = [torch.empty(cfg.n_kv_heads, t, cfg.head_dim, dtype=dt, device=dev) for _ in range(L)]
    betas = [torch.empty(cfg.n_kv_heads, t, dtype=torch.float32, device=dev) for _ in range(L)]
    outp = torch.empty(t, dtype=torch.float64, device=dev)
    lw = [w if isinstance(w, LayerWeights) else LayerWeights(cfg, w) for w in weights]
    stream = torch.cuda.current_stream(dev).cuda_stream
    _check(still_compact_model_beta(ccfg, lw, K, V, positions, N, rope_theta, t,
                                    STILL_F_REROTATE if rerotate else 0, Ck, Cv, outp, w_beta,
                                    still_beta_opts(beta_max, mass_alpha, log_x), betas, workspace,
                                    workspace.numel(), stream))
    return Ck, Cv, outp, betas


def attend(q, C_k, C_v, beta, K, V, group: int = 1, causal: bool = False, scale: float = 0.0, workspace=None,
           out=None, q_positions=None, rope_theta: float = 0.0):
    """Attention of q [H*group, n_q, d] over [C_k; K] with bias [beta; 0]
    through still_attend on the current stream; returns out like q.  C_k/C_v
    [H, t, d] and K/V [H, S, d] may be None for t = 0 / S = 0; beta [H, t]
    float32 or None.  ``out`` (like q) and ``workspace`` may be given, so that
    the call allocates nothing (graph capture).  With ``q_positions`` (float64
    [n_q] device tensor of logical positions) and ``rope_theta`` the kernel
    rotates q there first."""
    torch = _torch()
    Hq, nq, d = (int(x) for x in q.shape)
    H = Hq // group
    t = int(C_k.shape[1]) if C_k is not None else 0
    S = int(K.shape[1]) if K is not None else 0
    mode = configs.MODE_FP32 if q.dtype == torch.float32 else configs.MODE_BF16
    acfg = still_attend_config(H, group, d, nq, t, S, int(causal), float(scale), mode,
                               float(rope_theta) if q_positions is not None else 0.0)
    need = still_attend_workspace_size(acfg)
    if need == 0:
        _check(lib().still_attend(ctypes.byref(acfg), *[None] * 9, 0, None))   # raises with the reason
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    if out is None:
        out = torch.empty_like(q)
    stream = torch.cuda.current_stream(q.device).cuda_stream
    _check(still_attend(acfg, q, q_positions, C_k, C_v, beta, K, V, out, workspace, workspace.numel(), stream))
    return out
