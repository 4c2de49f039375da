"""Float64 CPU oracle for the Reflex action-expert denoise path.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library; both sides only consume the same seeded inputs.

What it computes
----------------
The paper's method (Reflex, "Real-Time Vision-Language-Action Control through
Streaming Inference") reaches exactly the full-batch result (Appendix A,
Proposition A.1), so the oracle is the full-batch definition written out
plainly: at every Euler step and every layer it rebuilds the whole context K/V
from its sources (static prefix, every frame in the FIFO window), concatenates
[K_pin; K_slide; K_dyn] in chronological order and runs one masked softmax over
it (Eq. 1, Section 3.1).  Nothing is cached across steps.  A separate
partitioned evaluator (per-region partial softmax, merged by log-sum-exp, ring
slots in physical order, cache built once) exists only to check the paper's
equivalence claim against the full-batch path.

Model readings where the paper is silent (all in float64):

* AdaRMSNorm (Eq. 2, Section 3.2; Appendix B.3): RMS(x) = sqrt(mean(x^2) + eps)
  with eps inside the root; the conditioning MLP is Linear -> SiLU -> Linear
  on c = [sinusoidal timestep embedding ; robot state].  Its output is widened
  to (scale, shift, gate): y = x/RMS(x) * (1 + scale) + shift, and the branch
  output is added to the residual stream as h += gate * f(y).  With
  ``mod_mode == "scale_only"`` shift = 0 and gate = 1, which is Eq. 2 exactly.
* Sinusoidal timestep embedding: width D, half sine / half cosine of
  2*pi*tau/period_i with periods geometric between 4e-3 and 4.0.
* RoPE: rotate-half pairing (i, i + d/2), base 10000, on q and k only, with
  absolute positions; angles formed in float64.  Positions: static prefix
  0..Ls-1, frame f token j at Ls + f*F + j, dynamic token i at
  Ls + frames_written*F + i.
* Dynamic-region mask: every dynamic row sees every cached row; the state token
  sees only itself among the dynamic tokens; action tokens see the state token
  and all action tokens.
* MLP: gated GELU (tanh form) on the gate half times the up half.
* Flow integration: x ~ N(0, I) at tau = 1 (Section 3.2), explicit Euler on
  the tau grid tau_0 = 1 > ... > tau_K = 0: x_{k+1} = x_k + (tau_{k+1} - tau_k) v_k.
* Sliding window: FIFO of the last W frames (Section 3.1; Appendix C).

Weights use the "rows are output features" convention: y = x @ W.T.

Parity status: each function below names what pins it.  The whole chunk is
also pinned end to end at micro and tiny shapes by re-derivations that share
nothing with this module (scalar loops, torch library routines) and rebuild
the cached context from the raw sources with hand-enumerated positions
(tests/test_oracle_pins.py); the paper prints no worked numerical example.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

F64 = np.float64


# ---------------------------------------------------------------------------
# elementwise pieces
# ---------------------------------------------------------------------------
def rms(x: np.ndarray, eps: float) -> np.ndarray:
    """RMS(x) = sqrt(mean_i x_i^2 + eps) over the last axis (Eq. 2).

    Pinned by: zero-modulation AdaRMSNorm vs torch.nn.functional.rms_norm and
    the constant-vector closed form.
    """
    x = np.asarray(x, dtype=F64)
    return np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def ada_rms_norm(x, scale, shift, eps: float) -> np.ndarray:
    """x / RMS(x) * (1 + scale) + shift (Eq. 2 with the shift extension).

    Pinned by: scale_only equals the Appendix B.3 forward; zero modulation
    equals plain RMSNorm; constant input closed form.
    """
    x = np.asarray(x, dtype=F64)
    return x / rms(x, eps) * (1.0 + scale) + shift


def silu(u) -> np.ndarray:
    """SiLU(u) = u * sigmoid(u) (Appendix B.3 conditioning MLP). Pinned vs torch."""
    u = np.asarray(u, dtype=F64)
    return u / (1.0 + np.exp(-u))


def gelu_tanh(u) -> np.ndarray:
    """GELU, tanh approximation (Hendrycks & Gimpel). Pinned vs torch."""
    u = np.asarray(u, dtype=F64)
    return 0.5 * u * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (u + 0.044715 * u ** 3)))


def timestep_embedding(tau: float, dim: int, min_period: float, max_period: float) -> np.ndarray:
    """Sinusoidal embedding of the flow time tau (c = [t_k, s_t], Section 3.2).

    Half sine, half cosine of 2*pi*tau/period_i, period_i geometric from
    min_period to max_period.  Pinned by closed-form values in the tests.
    """
    half = dim // 2
    frac = np.linspace(0.0, 1.0, half, dtype=F64)
    period = min_period * (max_period / min_period) ** frac
    arg = 2.0 * math.pi * float(tau) / period
    return np.concatenate([np.sin(arg), np.cos(arg)])


def rope_angles(pos: np.ndarray, dim: int, theta: float) -> np.ndarray:
    """Angles pos * theta^(-2i/dim), i < dim/2, in float64: shape [n, dim/2]."""
    i = np.arange(dim // 2, dtype=F64)
    inv = theta ** (-2.0 * i / dim)
    return np.asarray(pos, dtype=F64)[:, None] * inv[None, :]


def rope(z: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half RoPE at absolute positions.

    z: [n, ..., dim], pos: [n].  Pair (i, i + dim/2) is rotated by the angle
    pos * theta^(-2i/dim).  Pinned by the complex-number form, norm
    preservation, rope(z, 0) = z and relative-position invariance.
    """
    z = np.asarray(z, dtype=F64)
    dim = z.shape[-1]
    half = dim // 2
    ang = rope_angles(pos, dim, theta)
    shape = (z.shape[0],) + (1,) * (z.ndim - 2) + (half,)
    c = np.cos(ang).reshape(shape)
    s = np.sin(ang).reshape(shape)
    a, b = z[..., :half], z[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


# ---------------------------------------------------------------------------
# conditioning
# ---------------------------------------------------------------------------
@dataclass
class Modulation:
    scale: np.ndarray
    shift: np.ndarray
    gate: np.ndarray


def condition_vector(cfg, tau: float, state: np.ndarray) -> np.ndarray:
    """c = [sinusoidal(tau) ; s] (Section 3.2)."""
    temb = timestep_embedding(tau, cfg.width, cfg.temb_min_period, cfg.temb_max_period)
    return np.concatenate([temb, np.asarray(state, dtype=F64)])


def modulation(w1: np.ndarray, w2: np.ndarray, c: np.ndarray, width: int, mode: str) -> Modulation:
    """Linear -> SiLU -> Linear on c, split into (scale, shift, gate).

    Follows the conditioning MLP of Appendix B.3 (gamma = 1 + MLP(c), Eq. 2),
    widened to three width-D outputs.  Pinned vs torch.nn.Sequential.
    """
    m = np.asarray(w2, F64) @ silu(np.asarray(w1, F64) @ c)
    scale, shift, gate = m[:width], m[width:2 * width], m[2 * width:3 * width]
    if mode == "scale_only":
        shift = np.zeros_like(shift)
        gate = np.ones_like(gate)
    return Modulation(scale, shift, gate)


# ---------------------------------------------------------------------------
# sliding window / ring bookkeeping (Section 3.1 FIFO, Section 3.4 ring buffer,
# Appendix B.1-B.2)
# ---------------------------------------------------------------------------
@dataclass(frozen=True)
class RingStep:
    frame_index: int      # f, the index of the frame being written
    slot: int             # physical slot f mod W
    pos0: int             # absolute RoPE position of the frame's first token
    n_valid: int          # frames visible after the write, min(f+1, W)
    evicted: int          # tokens evicted by this write (F once the ring is full)
    dyn_pos0: int         # absolute position of dynamic token 0 after the write


def ring_step(frames_written: int, window: int, frame_tokens: int, static_len: int) -> RingStep:
    """Bookkeeping of one FIFO write.  Pinned by the hand-enumerated trace."""
    f = int(frames_written)
    return RingStep(
        frame_index=f,
        slot=f % window,
        pos0=static_len + f * frame_tokens,
        n_valid=min(f + 1, window),
        evicted=frame_tokens if f >= window else 0,
        dyn_pos0=static_len + (f + 1) * frame_tokens,
    )


def window_frames(frames_written: int, window: int) -> List[int]:
    """Frame indices in the FIFO window, oldest first."""
    return list(range(max(0, frames_written - window), frames_written))


def dyn_pos0(cfg, frames_written: int) -> int:
    return cfg.static_len + frames_written * cfg.frame_tokens


# ---------------------------------------------------------------------------
# context K/V from sources (no cache)
# ---------------------------------------------------------------------------
def static_kv(cfg, static_k: np.ndarray, static_v: np.ndarray, layer: int, env: int):
    """Pinned prefix K (RoPE at 0..Ls-1) and V for one env and layer: [Ls, Hkv, dh].

    Pinned by positions read back from its output and by the raw-source
    brute force of the whole chunk.
    """
    Hkv, dh = cfg.n_kv_heads, cfg.head_dim
    k = np.asarray(static_k[env, layer], F64).reshape(-1, Hkv, dh)
    v = np.asarray(static_v[env, layer], F64).reshape(-1, Hkv, dh)
    pos = np.arange(cfg.static_len)
    return rope(k, pos, cfg.rope_theta), v


def frame_kv(cfg, weights, frame_env: np.ndarray, frame_index: int, layer: int):
    """K/V of one frame at one layer: [F, Hkv, dh] each.

    Embedding path (frame_dim > 0): K = E W_k^T, V = E W_v^T with the layer's
    frame projection, RoPE on K at the frame's absolute positions.  Direct path
    (frame_dim == 0): the frame carries pre-RoPE K/V per layer.  Pinned by
    positions read back from its output against the hand-enumerated ring trace
    and by the raw-source brute force of the whole chunk.
    """
    Hkv, dh, F = cfg.n_kv_heads, cfg.head_dim, cfg.frame_tokens
    pos = cfg.static_len + frame_index * F + np.arange(F)
    if cfg.frame_dim > 0:
        E = np.asarray(frame_env, F64)
        w = np.asarray(weights["w_kv"][layer], F64)
        k = (E @ w[:Hkv * dh].T).reshape(F, Hkv, dh)
        v = (E @ w[Hkv * dh:].T).reshape(F, Hkv, dh)
    else:
        raw = np.asarray(frame_env[layer], F64)
        k = raw[0].reshape(F, Hkv, dh)
        v = raw[1].reshape(F, Hkv, dh)
    return rope(k, pos, cfg.rope_theta), v


def context_kv(cfg, weights, static_k, static_v, frames: Dict[int, np.ndarray],
               frames_written: int, layer: int, env: int):
    """[K_pin; K_slide] and [V_pin; V_slide] in chronological order, rebuilt."""
    ks, vs = static_kv(cfg, static_k, static_v, layer, env)
    K, V = [ks], [vs]
    for f in window_frames(frames_written, cfg.window_frames):
        k, v = frame_kv(cfg, weights, frames[f][env], f, layer)
        K.append(k)
        V.append(v)
    return np.concatenate(K, axis=0), np.concatenate(V, axis=0)


# ---------------------------------------------------------------------------
# attention (Eq. 1)
# ---------------------------------------------------------------------------
def dyn_allowed(n_ctx: int, T: int) -> np.ndarray:
    """Visibility of [context ; dynamic] keys for the T dynamic query rows."""
    allowed = np.ones((T, n_ctx + T), dtype=bool)
    allowed[0, n_ctx + 1:] = False  # state token: itself only among dynamic keys
    return allowed


def masked_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, allowed: np.ndarray) -> np.ndarray:
    """softmax(q K^T / sqrt(d)) V over the allowed keys, per query head.

    q: [T, Hq, dh]; K, V: [N, Hkv, dh]; query head j reads K/V head
    j // (Hq / Hkv).  Returns [T, Hq, dh].  Pinned vs
    torch.nn.functional.scaled_dot_product_attention and a scalar loop.
    """
    T, Hq, dh = q.shape
    Hkv = K.shape[1]
    group = Hq // Hkv
    out = np.empty((T, Hq, dh), dtype=F64)
    for j in range(Hq):
        kv = j // group
        s = (q[:, j, :] @ K[:, kv, :].T) / math.sqrt(dh)
        s = np.where(allowed, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, j, :] = p @ V[:, kv, :]
    return out


def partitioned_attention(q: np.ndarray, regions: Sequence[Tuple[np.ndarray, np.ndarray, np.ndarray]]) -> np.ndarray:
    """Eq. 1 evaluated region by region and merged with log-sum-exp.

    regions: (K_r, V_r, allowed_r) with allowed_r [T, n_r].  Used only to check
    the equivalence of Proposition A.1 against ``masked_attention``.
    """
    T, Hq, dh = q.shape
    out = np.empty((T, Hq, dh), dtype=F64)
    for j in range(Hq):
        ms, ls, os_ = [], [], []
        for K, V, allowed in regions:
            Hkv = K.shape[1]
            kv = j // (Hq // Hkv)
            s = (q[:, j, :] @ K[:, kv, :].T) / math.sqrt(dh)
            s = np.where(allowed, s, -np.inf)
            m = s.max(axis=1)
            m_safe = np.where(np.isfinite(m), m, 0.0)
            p = np.exp(s - m_safe[:, None])
            ms.append(m)
            ls.append(p.sum(axis=1))
            os_.append(p @ V[:, kv, :])
        m_all = np.max(np.stack(ms), axis=0)
        num = np.zeros((T, dh))
        den = np.zeros(T)
        for m, l, o in zip(ms, ls, os_):
            w = np.where(np.isfinite(m), np.exp(np.where(np.isfinite(m), m, 0.0) - m_all), 0.0)
            num += w[:, None] * o
            den += w * l
        out[:, j, :] = num / den[:, None]
    return out


# ---------------------------------------------------------------------------
# action expert
# ---------------------------------------------------------------------------
AttnFn = Callable[[int, np.ndarray, np.ndarray, np.ndarray], np.ndarray]


def velocity(cfg, weights, state: np.ndarray, x: np.ndarray, tau: float,
             dyn_positions: np.ndarray, attend: AttnFn,
             diag: Optional[dict] = None) -> np.ndarray:
    """One forward of the action expert for one env: v_theta(x, tau) [H, d_a].

    ``attend(layer, q, k_dyn, v_dyn)`` returns the attention output [T, Hq, dh]
    for the dynamic queries given this step's dynamic K/V; the full-batch and
    the partitioned evaluators plug in here.
    """
    L, D, Fm = cfg.n_layers, cfg.width, cfg.mlp_dim
    Hq, Hkv, dh = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    eps = cfg.rms_eps
    c = condition_vector(cfg, tau, state)
    mods = [modulation(weights["w_mod1"][s], weights["w_mod2"][s], c, D, cfg.mod_mode)
            for s in range(2 * L + 1)]

    w_state = np.asarray(weights["w_state"], F64)
    w_ain = np.asarray(weights["w_ain"], F64)
    h = np.concatenate([(w_state @ np.asarray(state, F64))[None, :],
                        np.asarray(x, F64) @ w_ain.T], axis=0) * cfg.embed_scale
    T = h.shape[0]
    for l in range(L):
        m1, m2 = mods[2 * l], mods[2 * l + 1]
        y = ada_rms_norm(h, m1.scale, m1.shift, eps)
        qkv = y @ np.asarray(weights["w_qkv"][l], F64).T
        q = qkv[:, :Hq * dh].reshape(T, Hq, dh)
        k = qkv[:, Hq * dh:(Hq + Hkv) * dh].reshape(T, Hkv, dh)
        v = qkv[:, (Hq + Hkv) * dh:].reshape(T, Hkv, dh)
        q = rope(q, dyn_positions, cfg.rope_theta)
        k = rope(k, dyn_positions, cfg.rope_theta)
        o = attend(l, q, k, v)
        if diag is not None:
            diag.setdefault("attn", []).append(o.copy())
        h = h + m1.gate * (o.reshape(T, Hq * dh) @ np.asarray(weights["w_o"][l], F64).T)
        y2 = ada_rms_norm(h, m2.scale, m2.shift, eps)
        u = y2 @ np.asarray(weights["w_gu"][l], F64).T
        z = gelu_tanh(u[:, :Fm]) * u[:, Fm:]
        h = h + m2.gate * (z @ np.asarray(weights["w_down"][l], F64).T)
    mf = mods[2 * L]
    yf = ada_rms_norm(h[1:], mf.scale, mf.shift, eps)
    return yf @ np.asarray(weights["w_aout"], F64).T


def euler_integrate(vel: Callable[[np.ndarray, float], np.ndarray], x0: np.ndarray,
                    taus: Sequence[float], record: Optional[list] = None) -> np.ndarray:
    """x_{k+1} = x_k + (tau_{k+1} - tau_k) v(x_k, tau_k), k = 0..K-1.

    Noise at tau = 1 is carried to actions at tau = 0 (Section 2.1, Section 3.2).
    Pinned by closed forms (constant field, linear field).
    """
    x = np.asarray(x0, F64).copy()
    taus = [float(t) for t in taus]
    for k in range(len(taus) - 1):
        v = vel(x, taus[k])
        if record is not None:
            record.append(np.asarray(v, F64).copy())
        x = x + (taus[k + 1] - taus[k]) * v
    return x


def full_batch_attend(cfg, weights, static_k, static_v, frames, frames_written, env) -> AttnFn:
    """Eq. 1 as one softmax over the rebuilt, concatenated context (no cache)."""
    def attend(layer, q, k, v):
        Kc, Vc = context_kv(cfg, weights, static_k, static_v, frames, frames_written, layer, env)
        K = np.concatenate([Kc, k], axis=0)
        V = np.concatenate([Vc, v], axis=0)
        return masked_attention(q, K, V, dyn_allowed(Kc.shape[0], q.shape[0]))
    return attend


def denoise_chunk(cfg, weights, static_k, static_v, frames: Dict[int, np.ndarray],
                  frames_written: int, state: np.ndarray, noise: np.ndarray,
                  taus: Sequence[float], envs: Optional[Sequence[int]] = None,
                  diag: Optional[dict] = None) -> np.ndarray:
    """Full-batch denoise of one action chunk per env: returns x_K [B', H, d_a].

    frames maps a frame index to its per-env array ([B, ...]); only the
    frames in the window of ``frames_written`` are read.  state [B, d_s] and
    noise [B, H, d_a] are indexed by env.  ``envs`` selects a subset of envs
    (rows of state/noise/frames are still indexed by the true env id).
    With ``diag`` a dict, the per-step velocities are recorded under "v".
    """
    envs = range(np.asarray(state).shape[0]) if envs is None else envs
    T = cfg.action_horizon + 1
    pos = dyn_pos0(cfg, frames_written) + np.arange(T)
    out = []
    for b in envs:
        attend = full_batch_attend(cfg, weights, static_k, static_v, frames, frames_written, b)
        s_b = np.asarray(state[b], F64)
        vel = lambda x, tau: velocity(cfg, weights, s_b, x, tau, pos, attend)  # noqa: E731
        rec = [] if diag is not None else None
        out.append(euler_integrate(vel, noise[b], taus, record=rec))
        if diag is not None:
            diag.setdefault("v", []).append(rec)
    return np.stack(out)


# ---------------------------------------------------------------------------
# partitioned evaluation (for the Proposition A.1 check only)
# ---------------------------------------------------------------------------
class PartitionedCache:
    """A simulated three-region cache: static rows once, ring slots in physical
    order, FIFO overwrite of slot f mod W.  Built once, read at every step."""

    def __init__(self, cfg, weights, static_k, static_v, env: int):
        self.cfg, self.weights, self.env = cfg, weights, env
        self.static = [static_kv(cfg, static_k, static_v, l, env) for l in range(cfg.n_layers)]
        self.slots: List[Optional[Tuple[int, list]]] = [None] * cfg.window_frames
        self.frames_written = 0

    def write(self, frame_env: np.ndarray) -> RingStep:
        cfg = self.cfg
        st = ring_step(self.frames_written, cfg.window_frames, cfg.frame_tokens, cfg.static_len)
        kv = [frame_kv(cfg, self.weights, frame_env, st.frame_index, l) for l in range(cfg.n_layers)]
        self.slots[st.slot] = (st.frame_index, kv)
        self.frames_written += 1
        return st

    def attend(self, layer, q, k, v, naive_dyn: Optional[Tuple[np.ndarray, np.ndarray]] = None):
        T = q.shape[0]
        regions = [(self.static[layer][0], self.static[layer][1],
                    np.ones((T, self.cfg.static_len), dtype=bool))]
        for slot in self.slots:
            if slot is None:
                continue
            kf, vf = slot[1][layer]
            regions.append((kf, vf, np.ones((T, kf.shape[0]), dtype=bool)))
        kd, vd = (k, v) if naive_dyn is None else naive_dyn
        regions.append((kd, vd, dyn_allowed(0, T)))
        return partitioned_attention(q, regions)


def denoise_chunk_partitioned(cfg, weights, cache: PartitionedCache, state_env: np.ndarray,
                              noise_env: np.ndarray, taus: Sequence[float],
                              naive_cache: bool = False, diag: Optional[dict] = None) -> np.ndarray:
    """One env's chunk through the simulated partitioned cache.

    With ``naive_cache`` the dynamic K/V of the first Euler step are reused at
    every later step (a cache whose key leaves out the timestep is filled at
    the first step and hit afterwards), the negative control of Section 4.6.
    """
    T = cfg.action_horizon + 1
    pos = dyn_pos0(cfg, cache.frames_written) + np.arange(T)
    stale: Dict[int, Tuple[np.ndarray, np.ndarray]] = {}
    step = {"k": 0}

    def attend(layer, q, k, v):
        use = stale.get(layer) if (naive_cache and step["k"] > 0) else None
        if naive_cache and step["k"] == 0:
            stale[layer] = (k, v)
        return cache.attend(layer, q, k, v, naive_dyn=use)

    s_b = np.asarray(state_env, F64)

    def vel(x, tau):
        out = velocity(cfg, weights, s_b, x, tau, pos, attend, diag=diag)
        step["k"] += 1
        return out

    return euler_integrate(vel, noise_env, taus)
