"""Compactor and workload configurations (shapes only, no arithmetic).

A compactor is the per-layer Perceiver of Section 2.1 / Appendix A: latent
bank Z in R^{H x t x d_l}, B pre-norm blocks of cross-attention (n_c heads of
width d_l each, the "expanded" convention of Appendix A, cross-attention
paragraph), latent self-attention (n_s heads) and a feed-forward sublayer,
then two output heads W_key, W_val.

The five registered workloads are synthetic stand-ins for the paper's Qwen3
(d=128, 8 KV heads, 36 layers) and Gemma-3 (d=256, 42 layers) caches at
8k-128k context and 8x-200x compression.  Only shapes and distributions are
taken from the paper; no dataset is used.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

FFN_NONE = 0
FFN_SWIGLU = 1
FFN_GELU = 2

MODE_BF16 = 0
MODE_FP32 = 1


@dataclasses.dataclass(frozen=True)
class CompactorConfig:
    """Hyper-parameters of one layer's compactor (mirrors ``still_config``)."""

    n_kv_heads: int          # H
    head_dim: int            # d, base-model KV head width
    latent_dim: int          # D = d_l
    n_blocks: int = 1        # B
    cross_every_block: int = 1   # 1: cross-attention in every block; 0: block 0 only
    n_cross_heads: int = 1   # n_c
    cross_head_dim: int = 0  # 0 -> latent_dim (expanded-head convention)
    n_self_heads: int = 1    # n_s (0 disables latent self-attention)
    self_head_dim: int = 0   # 0 -> latent_dim
    ffn_kind: int = FFN_SWIGLU
    ffn_hidden: int = 0
    final_norm: int = 0
    logit_scale_cross: float = 0.0   # 0 -> cross head width (the d_l scale)
    logit_scale_self: float = 0.0    # 0 -> self head width
    compactor_rope_base: float = 10.0
    rms_eps: float = 1e-6
    l2_eps: float = 1e-12

    @property
    def dc(self) -> int:
        return self.cross_head_dim or self.latent_dim

    @property
    def ds(self) -> int:
        return self.self_head_dim or self.latent_dim

    @property
    def scale_cross(self) -> float:
        return self.logit_scale_cross or float(self.dc)

    @property
    def scale_self(self) -> float:
        return self.logit_scale_self or float(self.ds)

    def has_cross(self, block: int) -> bool:
        return self.n_cross_heads > 0 and (self.cross_every_block or block == 0)


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic compaction workload."""

    name: str
    cfg: CompactorConfig
    n_layers: int
    n_tokens: int            # N, cache tokens entering the (first) compaction call
    t: int                   # compact length
    rope_theta: float        # base-model RoPE base
    seed: int
    outlier_channels: int = 0    # channels per head scaled x10 in the position-free key frame
    outlier_scale: float = 10.0
    rounds: int = 0          # iterative re-compaction rounds after the first call
    fresh_tokens: int = 0    # tokens appended before each round
    query_group: int = 4     # base-model query heads per KV head (consumer attention)

    @property
    def ratio(self) -> float:
        return self.n_tokens / self.t


def _qwen8b_compactor(H=8, d=128) -> CompactorConfig:
    return CompactorConfig(n_kv_heads=H, head_dim=d, latent_dim=1024, n_blocks=1,
                           n_cross_heads=8, n_self_heads=8, ffn_kind=FFN_SWIGLU,
                           ffn_hidden=4096)


WORKLOADS = {
    1: Workload(
        name="single-layer H2 d64 N2048 t256 D128",
        cfg=CompactorConfig(n_kv_heads=2, head_dim=64, latent_dim=128, n_blocks=1,
                            n_cross_heads=2, n_self_heads=2, ffn_kind=FFN_SWIGLU,
                            ffn_hidden=512),
        n_layers=1, n_tokens=2048, t=256, rope_theta=1e6, seed=0),
    2: Workload(
        name="qwen8b-shaped 36L H8 d128 N8192 t1024 (8x)",
        cfg=_qwen8b_compactor(), n_layers=36, n_tokens=8192, t=1024,
        rope_theta=1e6, seed=1, outlier_channels=4),
    3: Workload(
        name="qwen8b-shaped 36L H8 d128 N32768 t1024 (32x)",
        cfg=_qwen8b_compactor(), n_layers=36, n_tokens=32768, t=1024,
        rope_theta=1e6, seed=2, outlier_channels=4),
    4: Workload(
        name="qwen8b-shaped 36L H8 d128 N131072 t655 (200x)",
        cfg=_qwen8b_compactor(), n_layers=36, n_tokens=131072, t=655,
        rope_theta=1e6, seed=3, outlier_channels=4),
    5: Workload(
        name="gemma-shaped 42L H8 d256 N65536 t1024 + 8x(1024+8192)",
        cfg=CompactorConfig(n_kv_heads=8, head_dim=256, latent_dim=2048, n_blocks=1,
                            n_cross_heads=8, n_self_heads=8, ffn_kind=FFN_SWIGLU,
                            ffn_hidden=8192),
        n_layers=42, n_tokens=65536, t=1024, rope_theta=1e4, seed=4,
        rounds=8, fresh_tokens=8192, query_group=2),
}


def get_workload(i: int) -> Workload:
    return WORKLOADS[i]


def shrink(w: Workload, n_tokens: Optional[int] = None, t: Optional[int] = None,
           n_layers: Optional[int] = None, **cfg_changes) -> Workload:
    """Same workload with smaller sizes (for quick parity cases)."""
    cfg = dataclasses.replace(w.cfg, **cfg_changes) if cfg_changes else w.cfg
    return dataclasses.replace(w, cfg=cfg,
                               n_tokens=n_tokens if n_tokens is not None else w.n_tokens,
                               t=t if t is not None else w.t,
                               n_layers=n_layers if n_layers is not None else w.n_layers)


# Weight tensors of one block, in a fixed enumeration order.  Storage follows the
# torch.nn.Linear convention: a projection x -> x W (W in R^{in x out} in the
# paper's notation) is stored as the row-major [out][in] matrix W^T.
BLOCK_TENSORS = ("ca_wq", "ca_bq", "ca_wk", "ca_bk", "ca_wv", "ca_wo",
                 "sa_wq", "sa_bq", "sa_wk", "sa_bk", "sa_wv", "sa_wo",
                 "ffn_wg", "ffn_wu", "ffn_wd")


def block_shapes(cfg: CompactorConfig, block: int) -> dict:
    """Shapes of one block's tensors ([out][in] for matrices); absent tensors omitted."""
    D, d = cfg.latent_dim, cfg.head_dim
    s = {}
    if cfg.has_cross(block):
        E = cfg.n_cross_heads * cfg.dc
        s.update(ca_wq=(E, D), ca_bq=(E,), ca_wk=(E, 2 * d), ca_bk=(E,),
                 ca_wv=(E, 2 * d), ca_wo=(D, E))
    if cfg.n_self_heads > 0:
        E = cfg.n_self_heads * cfg.ds
        s.update(sa_wq=(E, D), sa_bq=(E,), sa_wk=(E, D), sa_bk=(E,),
                 sa_wv=(E, D), sa_wo=(D, E))
    if cfg.ffn_kind == FFN_SWIGLU:
        F = cfg.ffn_hidden
        s.update(ffn_wg=(F, D), ffn_wu=(F, D), ffn_wd=(D, F))
    elif cfg.ffn_kind == FFN_GELU:
        F = cfg.ffn_hidden
        s.update(ffn_wu=(F, D), ffn_wd=(D, F))
    return s


def layer_shapes(cfg: CompactorConfig, t: int) -> dict:
    """All tensors of one layer's compactor: latents, per-block tensors, heads."""
    D, d = cfg.latent_dim, cfg.head_dim
    out = {"latents": (cfg.n_kv_heads, t, D)}
    for b in range(cfg.n_blocks):
        for k, v in block_shapes(cfg, b).items():
            out[f"b{b}.{k}"] = v
    out["w_key"] = (d, D)
    out["w_val"] = (d, D)
    return out
