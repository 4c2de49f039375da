"""Workload shapes and the seeded synthetic input generator.

This module holds only configuration data and random draws.  It contains none
of the method's arithmetic: no normalisation, attention, RoPE, projection or
integration.  Both the HIP path (through the Python binding) and the float64
oracle consume the arrays it produces, so parity compares kernels against the
definition on identical inputs.

Draw discipline
---------------
* numpy PCG64, one child stream per (role, index, tick, env) key, derived with
  ``SeedSequence(entropy=seed, spawn_key=key)``.  A draw therefore does not
  depend on the batch size, the layer count or the order in which arrays are
  requested: env 0 of a 32-env workload sees exactly the frames, states and
  noise of env 0 of a 1-env workload with the same seed.
* Values are drawn in float32 and, for bf16 workloads, rounded to the nearest
  bf16 (ties to even) before either side sees them, so both sides start from
  the same representable numbers.
* Weights are N(0, 0.02^2); cache K/V, frame embeddings, states and initial
  action noise are N(0, 1) (the flow starts from Gaussian noise at tau = 1,
  Section 3.2).

The paper evaluates on LIBERO and Kinetix with Pi0 / Pi0.5 checkpoints; none of
those are available, so these seeded draws at the action expert's shapes (chunk
of 50 actions, 10 flow steps, three 256-token camera views per frame, Section 4
and Appendix C) stand in for them.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

DTYPE_F32 = "f32"
DTYPE_BF16 = "bf16"


@dataclass(frozen=True)
class ReflexConfig:
    """Shape of one workload.  Field names follow the C struct in reflex.h."""

    name: str
    # action expert
    n_layers: int
    width: int
    mlp_dim: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    state_dim: int
    action_dim: int
    action_horizon: int
    cond_hidden: int
    # three-region cache
    static_len: int
    frame_tokens: int
    window_frames: int
    frame_dim: int  # 0 = frames arrive as pre-RoPE per-layer K/V
    batch: int
    # numerics
    dtype: str
    num_steps: int
    rms_eps: float = 1e-6
    rope_theta: float = 10000.0
    temb_min_period: float = 4e-3
    temb_max_period: float = 4.0
    embed_scale: float = 1.0
    mod_mode: str = "full"  # "full" (scale/shift/gate) or "scale_only" (Eq. 2)
    # GPU cache layout only: 1 = one spare ring slot for pipelined frame writes
    spare_slot: int = 0
    # GPU numerics ablation only: "fp32" (the method), "bf16", "bf16_fp32_stats"
    norm_precision: str = "fp32"
    # GPU kernel choice only: "auto", or force "rows16" / "pair" (bf16 attention)
    attn_kernel: str = "auto"
    # workload driver
    ticks: int = 1
    tau_schedule: Optional[Tuple[float, ...]] = None
    seed: int = 0

    # ---- derived sizes -------------------------------------------------
    @property
    def dyn_tokens(self) -> int:
        return 1 + self.action_horizon

    @property
    def n_sites(self) -> int:
        return 2 * self.n_layers + 1

    @property
    def cond_dim(self) -> int:
        return self.width + self.state_dim

    @property
    def qkv_dim(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def cache_rows(self) -> int:
        return self.static_len + (self.window_frames + self.spare_slot) * self.frame_tokens

    @property
    def bf16(self) -> bool:
        return self.dtype == DTYPE_BF16

    def taus(self, num_steps: Optional[int] = None) -> np.ndarray:
        """The tau grid tau_0 = 1 > ... > tau_K = 0 as float32 values."""
        k = self.num_steps if num_steps is None else num_steps
        if self.tau_schedule is not None and num_steps is None:
            return np.asarray(self.tau_schedule, dtype=np.float32)
        return (1.0 - np.arange(k + 1, dtype=np.float64) / k).astype(np.float32)

    def replace(self, **kw) -> "ReflexConfig":
        return dataclasses.replace(self, **kw)


# The five workloads.  Sizes are those of a pi0-style action expert (width 1024,
# MLP 4096, 8 query heads sharing one 256-wide K/V head, 18 layers, chunk of 50
# actions) plus one tiny float32 check.
CONFIGS: Dict[str, ReflexConfig] = {
    "tiny_fp32": ReflexConfig(
        name="tiny_fp32", n_layers=2, width=256, mlp_dim=1024, n_q_heads=4,
        n_kv_heads=1, head_dim=64, state_dim=8, action_dim=8,
        action_horizon=16, cond_hidden=256, static_len=64, frame_tokens=32,
        window_frames=2, frame_dim=256, batch=1, dtype=DTYPE_F32,
        num_steps=4, ticks=5),
    "pi0_chunk_bf16": ReflexConfig(
        name="pi0_chunk_bf16", n_layers=18, width=1024, mlp_dim=4096,
        n_q_heads=8, n_kv_heads=1, head_dim=256, state_dim=32, action_dim=32,
        action_horizon=50, cond_hidden=1024, static_len=48, frame_tokens=768,
        window_frames=1, frame_dim=0, batch=1, dtype=DTYPE_BF16,
        num_steps=10, ticks=1),
    "pi0_stream_bf16": ReflexConfig(
        name="pi0_stream_bf16", n_layers=18, width=1024, mlp_dim=4096,
        n_q_heads=8, n_kv_heads=1, head_dim=256, state_dim=32, action_dim=32,
        action_horizon=50, cond_hidden=1024, static_len=48, frame_tokens=768,
        window_frames=2, frame_dim=2048, batch=1, dtype=DTYPE_BF16,
        num_steps=10, ticks=500),
    "pi0_batch32_bf16": ReflexConfig(
        name="pi0_batch32_bf16", n_layers=18, width=1024, mlp_dim=4096,
        n_q_heads=8, n_kv_heads=1, head_dim=256, state_dim=32, action_dim=32,
        action_horizon=50, cond_hidden=1024, static_len=48, frame_tokens=768,
        window_frames=2, frame_dim=2048, batch=32, dtype=DTYPE_BF16,
        num_steps=10, ticks=200),
    "pi0_long_bf16": ReflexConfig(
        name="pi0_long_bf16", n_layers=18, width=1024, mlp_dim=4096,
        n_q_heads=8, n_kv_heads=1, head_dim=256, state_dim=32, action_dim=32,
        action_horizon=50, cond_hidden=1024, static_len=256, frame_tokens=768,
        window_frames=8, frame_dim=0, batch=8, dtype=DTYPE_BF16,
        num_steps=10, ticks=8, embed_scale=64.0,
        tau_schedule=(1.0, 0.999, 0.99, 0.9, 0.7, 0.5, 0.3, 0.1, 0.01, 0.001,
                      0.0)),
}


# ---------------------------------------------------------------------------
# bf16 rounding (input quantisation, not part of the method)
# ---------------------------------------------------------------------------
def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); float32 out."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).copy()
    u += np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    u &= np.uint32(0xFFFF0000)
    return u.view(np.float32)


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 values that are exactly bf16 -> their uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return (u >> np.uint32(16)).astype(np.uint16)


# ---------------------------------------------------------------------------
# seeded draws
# ---------------------------------------------------------------------------
_ROLE = {
    "w_qkv": 1, "w_o": 2, "w_gu": 3, "w_down": 4, "w_state": 5, "w_ain": 6,
    "w_aout": 7, "w_mod1": 8, "w_mod2": 9, "w_kv": 10, "static_k": 11,
    "static_v": 12, "frame": 13, "state": 14, "noise": 15,
}


def _rng(cfg: ReflexConfig, role: str, *key: int) -> np.random.Generator:
    ss = np.random.SeedSequence(entropy=cfg.seed,
                                spawn_key=(_ROLE[role],) + tuple(int(k) for k in key))
    return np.random.Generator(np.random.PCG64(ss))


def _normal(cfg: ReflexConfig, shape, std: float, role: str, *key: int) -> np.ndarray:
    x = _rng(cfg, role, *key).standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return round_bf16(x) if cfg.bf16 else x


WEIGHT_STD = 0.02


def weight_shapes(cfg: ReflexConfig) -> Dict[str, Tuple[int, ...]]:
    """Shapes of every weight tensor; rows are output features (y = x W^T)."""
    L, D = cfg.n_layers, cfg.width
    s = {
        "w_qkv": (L, cfg.qkv_dim, D),
        "w_o": (L, D, cfg.n_q_heads * cfg.head_dim),
        "w_gu": (L, 2 * cfg.mlp_dim, D),
        "w_down": (L, D, cfg.mlp_dim),
        "w_state": (D, cfg.state_dim),
        "w_ain": (D, cfg.action_dim),
        "w_aout": (cfg.action_dim, D),
        "w_mod1": (cfg.n_sites, cfg.cond_hidden, cfg.cond_dim),
        "w_mod2": (cfg.n_sites, 3 * D, cfg.cond_hidden),
    }
    if cfg.frame_dim > 0:
        s["w_kv"] = (L, 2 * cfg.n_kv_heads * cfg.head_dim, cfg.frame_dim)
    return s


def make_weights(cfg: ReflexConfig) -> Dict[str, np.ndarray]:
    """All weights, float32 (bf16-representable for bf16 workloads).

    Stacked tensors are drawn one leading index at a time so a draw does not
    depend on the number of layers or sites.
    """
    out = {}
    for name, shape in weight_shapes(cfg).items():
        if len(shape) == 3:
            arr = np.empty(shape, dtype=np.float32)
            for i in range(shape[0]):
                arr[i] = _normal(cfg, shape[1:], WEIGHT_STD, name, i)
        else:
            arr = _normal(cfg, shape, WEIGHT_STD, name, 0)
        out[name] = arr
    return out


def make_static_kv(cfg: ReflexConfig) -> Tuple[np.ndarray, np.ndarray]:
    """Pre-RoPE static-prefix K and V, each [B, L, static_len, Hkv*head_dim]."""
    shp = (cfg.n_layers, cfg.static_len, cfg.n_kv_heads * cfg.head_dim)
    k = np.stack([_normal(cfg, shp, 1.0, "static_k", b) for b in range(cfg.batch)])
    v = np.stack([_normal(cfg, shp, 1.0, "static_v", b) for b in range(cfg.batch)])
    return k, v


def frame_shape(cfg: ReflexConfig) -> Tuple[int, ...]:
    """Per-env frame shape: embeddings [F, frame_dim] or raw K/V [L, 2, F, Hkv*dh]."""
    if cfg.frame_dim > 0:
        return (cfg.frame_tokens, cfg.frame_dim)
    return (cfg.n_layers, 2, cfg.frame_tokens, cfg.n_kv_heads * cfg.head_dim)


def make_frame_env(cfg: ReflexConfig, tick: int, env: int) -> np.ndarray:
    return _normal(cfg, frame_shape(cfg), 1.0, "frame", tick, env)


def make_frame(cfg: ReflexConfig, tick: int, envs: Optional[Sequence[int]] = None) -> np.ndarray:
    envs = range(cfg.batch) if envs is None else envs
    return np.stack([make_frame_env(cfg, tick, b) for b in envs])


def make_state(cfg: ReflexConfig, tick: int, envs: Optional[Sequence[int]] = None) -> np.ndarray:
    """Proprioceptive state [B, state_dim], float32 (bf16-representable if bf16)."""
    envs = range(cfg.batch) if envs is None else envs
    return np.stack([_normal(cfg, (cfg.state_dim,), 1.0, "state", tick, b) for b in envs])


def make_noise(cfg: ReflexConfig, tick: int, envs: Optional[Sequence[int]] = None) -> np.ndarray:
    """Initial action noise x_0 ~ N(0, I), [B, action_horizon, action_dim], float32.

    The noise is kept in float32 for every workload: the action state is an
    fp32 tensor on both sides.
    """
    envs = range(cfg.batch) if envs is None else envs
    out = []
    for b in envs:
        x = _rng(cfg, "noise", tick, b).standard_normal(
            size=(cfg.action_horizon, cfg.action_dim), dtype=np.float32)
        out.append(x)
    return np.stack(out)

