"""Python binding of libreflex.so (ctypes).

Argument marshalling only: device memory and the stream come from PyTorch,
every step of the denoise path runs in the library's HIP kernels.  There is no
fallback: if the shared library is missing or a call fails, an exception is
raised.
"""
from __future__ import annotations

import collections
import ctypes
import os
import re
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .workloads import ReflexConfig

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libreflex.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "reflex.h")

REFLEX_OK = 0
REFLEX_EINVAL = -1
REFLEX_EDTYPE = -2
REFLEX_EHIP = -3
REFLEX_ESTATE = -4
REFLEX_ENONFINITE = -5
REFLEX_ESCRATCH = -6
DTYPE_F32 = 0
DTYPE_BF16 = 1
MOD_FULL = 0
MOD_SCALE_ONLY = 1
MAX_STEPS = 64
MODE_REFLEX = 0
MODE_STANDARD = 1
MODE_NAIVE = 2
MODE_UNFUSED = 3
MODES = {"reflex": MODE_REFLEX, "standard": MODE_STANDARD, "naive": MODE_NAIVE, "unfused": MODE_UNFUSED}
NORM_PRECISIONS = {"fp32": 0, "bf16": 1, "bf16_fp32_stats": 2}
ATTN_KERNELS = {"auto": 0, "rows16": 1, "pair": 2, "rows16p": 3}

c_i32, c_i64, c_f32, c_f64, c_vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double, ctypes.c_void_p


class ConfigC(ctypes.Structure):
    _fields_ = [
        ("n_layers", c_i32), ("width", c_i32), ("mlp_dim", c_i32), ("n_q_heads", c_i32),
        ("n_kv_heads", c_i32), ("head_dim", c_i32), ("state_dim", c_i32), ("action_dim", c_i32),
        ("action_horizon", c_i32), ("cond_hidden", c_i32), ("static_len", c_i32),
        ("frame_tokens", c_i32), ("window_frames", c_i32), ("frame_dim", c_i32), ("batch", c_i32),
        ("dtype", c_i32), ("mod_mode", c_i32), ("max_steps", c_i32), ("rms_eps", c_f32),
        ("embed_scale", c_f32), ("rope_theta", c_f64), ("temb_min_period", c_f64),
        ("temb_max_period", c_f64), ("spare_slot", c_i32), ("norm_precision", c_i32),
        ("attn_kernel", c_i32),
    ]


class WeightsC(ctypes.Structure):
    _fields_ = [
        ("w_qkv", c_vp), ("w_o", c_vp), ("w_gu", c_vp), ("w_down", c_vp), ("w_state", c_vp),
        ("w_ain", c_vp), ("w_aout", c_vp), ("w_mod1", c_vp), ("w_mod2", c_vp), ("w_kv", c_vp),
        ("dtype", c_i32),
    ]


class RingStepC(ctypes.Structure):
    _fields_ = [
        ("frame_index", c_i64), ("slot", c_i32), ("n_valid", c_i32), ("pos0", c_i64),
        ("dyn_pos0", c_i64), ("evicted", c_i32), ("reserved", c_i32),
    ]


class SourcesC(ctypes.Structure):
    _fields_ = [
        ("static_k", c_vp), ("static_v", c_vp), ("frames", ctypes.POINTER(c_vp)), ("n_frames", c_i32),
        ("reserved", c_i32),
    ]


class ReflexError(RuntimeError):
    def __init__(self, status: int, what: str, text: str):
        super().__init__(f"{what} failed with status {status}: {text}")
        self.status = status


_LIB = None


def load_library() -> ctypes.CDLL:
    """Load libreflex.so (built in-tree by build.py); raise if it is absent."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} not found: build it with __graft_entry__.build() "
                          "(hipcc --offload-arch=gfx950)")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    sig = {
        "reflex_query_sizes": (c_i32, [P(ConfigC), P(ctypes.c_size_t), P(ctypes.c_size_t)]),
        "reflex_cache_init": (c_i32, [P(ConfigC), P(WeightsC), c_vp, c_vp, c_vp, c_vp, c_vp, P(c_vp)]),
        "reflex_cache_write_frame": (c_i32, [c_vp, c_vp, P(c_i64), P(c_i32)]),
        "reflex_denoise_chunk": (c_i32, [c_vp, c_vp, c_vp, c_i32, c_vp, c_vp]),
        "reflex_denoise_chunk_baseline": (c_i32, [c_vp, c_i32, P(SourcesC), c_vp, c_vp, c_i32, c_vp, c_vp]),
        "reflex_pipeline_write_frame": (c_i32, [c_vp, c_vp, c_vp, P(c_i64), P(c_i32)]),
        "reflex_pipeline_denoise_chunk": (c_i32, [c_vp, c_vp, c_vp, c_i32, c_vp, c_vp, c_i64, P(c_i64)]),
        "reflex_denoise_chunk_static": (c_i32, [c_vp, c_vp, c_vp, c_i32, c_vp, c_vp]),
        "reflex_check_status": (c_i32, [c_vp]),
        "reflex_destroy": (c_i32, [c_vp]),
        "reflex_strerror": (ctypes.c_char_p, [c_i32]),
        "reflex_ring_plan": (c_i32, [c_i64, c_i32, c_i32, c_i32, P(RingStepC)]),
        "reflex_frames_written": (c_i64, [c_vp]),
        "reflex_profile_enable": (c_i32, [c_vp, c_i32]),
        "reflex_profile_read": (c_i32, [c_vp, P(ctypes.c_char_p), P(c_f64), P(c_i32), P(c_i32)]),
        "reflex_profile_graph": (c_i32, [c_vp, c_vp, c_vp, c_i32, c_vp, c_vp, ctypes.c_uint32, c_i32, P(c_f64),
                                         P(c_i32)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _LIB = lib
    return lib


def header_functions() -> Sequence[str]:
    """Names of the functions declared in include/reflex.h."""
    with open(HEADER_PATH) as fh:
        text = fh.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z0-9_]+\s*\*?\s*(reflex_[a-z_]+)\s*\(", text, re.M)))


def strerror(status: int) -> str:
    return load_library().reflex_strerror(status).decode()


def _check(status: int, what: str) -> None:
    if status != REFLEX_OK:
        raise ReflexError(status, what, strerror(status))


def config_to_c(cfg: ReflexConfig, max_steps: Optional[int] = None) -> ConfigC:
    ms = max_steps if max_steps is not None else max(cfg.num_steps, 1)
    return ConfigC(
        n_layers=cfg.n_layers, width=cfg.width, mlp_dim=cfg.mlp_dim, n_q_heads=cfg.n_q_heads,
        n_kv_heads=cfg.n_kv_heads, head_dim=cfg.head_dim, state_dim=cfg.state_dim,
        action_dim=cfg.action_dim, action_horizon=cfg.action_horizon, cond_hidden=cfg.cond_hidden,
        static_len=cfg.static_len, frame_tokens=cfg.frame_tokens, window_frames=cfg.window_frames,
        frame_dim=cfg.frame_dim, batch=cfg.batch, dtype=DTYPE_BF16 if cfg.bf16 else DTYPE_F32,
        mod_mode=MOD_SCALE_ONLY if cfg.mod_mode == "scale_only" else MOD_FULL, max_steps=ms,
        rms_eps=cfg.rms_eps, embed_scale=cfg.embed_scale, rope_theta=cfg.rope_theta,
        temb_min_period=cfg.temb_min_period, temb_max_period=cfg.temb_max_period, spare_slot=cfg.spare_slot,
        norm_precision=NORM_PRECISIONS[cfg.norm_precision], attn_kernel=ATTN_KERNELS[cfg.attn_kernel])


def query_sizes(cfg: ReflexConfig, max_steps: Optional[int] = None) -> Tuple[int, int]:
    lib = load_library()
    c = config_to_c(cfg, max_steps)
    cb, wb = ctypes.c_size_t(0), ctypes.c_size_t(0)
    _check(lib.reflex_query_sizes(ctypes.byref(c), ctypes.byref(cb), ctypes.byref(wb)), "reflex_query_sizes")
    return cb.value, wb.value


def query_sizes_status(c: ConfigC) -> int:
    lib = load_library()
    cb, wb = ctypes.c_size_t(0), ctypes.c_size_t(0)
    return lib.reflex_query_sizes(ctypes.byref(c), ctypes.byref(cb), ctypes.byref(wb))


def ring_plan(frames_written: int, window: int, frame_tokens: int, static_len: int) -> Dict[str, int]:
    lib = load_library()
    out = RingStepC()
    _check(lib.reflex_ring_plan(frames_written, window, frame_tokens, static_len, ctypes.byref(out)),
           "reflex_ring_plan")
    return {k: getattr(out, k) for k, _ in RingStepC._fields_ if k != "reserved"}


class ReflexEngine:
    """One library context: caller-owned device buffers + the host context.

    weights: numpy float32 arrays (bf16-representable for bf16 workloads) or
    torch tensors already on the device with the config's dtype.
    """

    WEIGHT_ORDER = ("w_qkv", "w_o", "w_gu", "w_down", "w_state", "w_ain", "w_aout", "w_mod1", "w_mod2", "w_kv")

    def __init__(self, cfg: ReflexConfig, weights, static_k, static_v, device: str = "cuda:0",
                 max_steps: Optional[int] = None, weight_dtype_override=None):
        import torch

        self.torch = torch
        self.cfg = cfg
        self.device = torch.device(device)
        self.lib = load_library()
        self.dtype = torch.bfloat16 if cfg.bf16 else torch.float32
        self.max_steps = max_steps if max_steps is not None else max(cfg.num_steps, 1)
        self.stream = torch.cuda.Stream(device=self.device)
        self.writer = None  # second stream of the asynchronous pipeline, made on first use
        self.last_n_frames = None
        self.ctx = c_vp(None)
        self._bufs = {}
        # the weights and the static K/V may still be in production on the
        # caller's stream: the library reads them on the engine stream
        self.stream.wait_stream(torch.cuda.current_stream(self.device))
        with torch.cuda.stream(self.stream):
            self.w = {}
            for name in self.WEIGHT_ORDER:
                if name not in weights:
                    continue
                self.w[name] = self._dev(weights[name], weight_dtype_override)
            sk = self._dev(static_k)
            sv = self._dev(static_v)
            # kept for the Standard strategy, which encodes them again at every step
            self._static = (sk, sv)
            self._window = collections.deque(maxlen=cfg.window_frames)
            self.cache_bytes, self.ws_bytes = query_sizes(cfg, self.max_steps)
            self.cache = torch.empty(self.cache_bytes, dtype=torch.uint8, device=self.device)
            self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)
            wc = WeightsC(**{n: (self.w[n].data_ptr() if n in self.w else None) for n in self.WEIGHT_ORDER})
            probe = self.w["w_o"].dtype  # dtype probe of the output projection
            wc.dtype = DTYPE_BF16 if probe == torch.bfloat16 else (DTYPE_F32 if probe == torch.float32 else 99)
            cc = config_to_c(cfg, self.max_steps)
            st = self.lib.reflex_cache_init(ctypes.byref(cc), ctypes.byref(wc), self.cache.data_ptr(),
                                            self.ws.data_ptr(), sk.data_ptr() if sk.numel() else None,
                                            sv.data_ptr() if sv.numel() else None,
                                            self.stream.cuda_stream, ctypes.byref(self.ctx))
            _check(st, "reflex_cache_init")
        self.stream.synchronize()

    # -- helpers -------------------------------------------------------------
    def _dev(self, a, dtype=None):
        torch = self.torch
        dt = dtype if dtype is not None else self.dtype
        if isinstance(a, torch.Tensor):
            return a.to(device=self.device, dtype=dt).contiguous()
        return torch.from_numpy(np.ascontiguousarray(a)).to(device=self.device).to(dt).contiguous()

    def _f32(self, a):
        torch = self.torch
        if isinstance(a, torch.Tensor):
            return a.to(device=self.device, dtype=torch.float32).contiguous()
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(self.device)

    # -- API -----------------------------------------------------------------
    def current(self):
        """Context manager making the engine's stream the caller's current
        stream.

        Every call orders the engine's stream after the caller's current stream
        and the caller's stream after the engine's work.  With a caller stream
        of its own, the second ordering leaves a wait for the engine's event in
        another hardware queue for as long as that work runs, and the chunk's
        kernels then run with longer gaps between them: a batch-1 chunk took
        9.78 ms against 8.73 ms with the orderings on the engine's own stream
        (32 envs 28.8 against 28.4 ms, the long context 18.5 against 17.8 ms).
        Inside this context both orderings stay on the one stream."""
        return self.torch.cuda.stream(self.stream)

    def _enter(self):
        """Order the engine stream after the caller's current stream."""
        caller = self.torch.cuda.current_stream(self.device)
        self.stream.wait_stream(caller)
        return caller

    def write_frame(self, frame) -> Tuple[int, int]:
        """Write one frame for all envs; returns (frame_index, evicted_tokens).

        Device work runs on the engine's stream; the caller's current stream
        is ordered after it, so later work there sees the written cache."""
        caller = self._enter()
        with self.torch.cuda.stream(self.stream):
            f = self._dev(frame)
            fi, ev = c_i64(0), c_i32(0)
            _check(self.lib.reflex_cache_write_frame(self.ctx, f.data_ptr(), ctypes.byref(fi), ctypes.byref(ev)),
                   "reflex_cache_write_frame")
            self._window.append(f)  # the window's frames, for the Standard strategy
        caller.wait_stream(self.stream)
        return fi.value, ev.value

    def pipeline_write(self, frame) -> Tuple[int, int]:
        """Write one frame on the engine's writer stream (asynchronous
        pipeline, needs ``cfg.spare_slot = 1``); returns (frame_index,
        evicted_tokens).  The write overlaps chunks on the engine stream; the
        library orders the two streams on the device.  The caller's stream is
        not made to wait for the write."""
        torch = self.torch
        if self.writer is None:
            self.writer = torch.cuda.Stream(device=self.device)
        self.writer.wait_stream(torch.cuda.current_stream(self.device))
        with torch.cuda.stream(self.writer):
            f = self._dev(frame)
            f.record_stream(self.writer)  # not reused before the writer has read it
            fi, ev = c_i64(0), c_i32(0)
            _check(self.lib.reflex_pipeline_write_frame(self.ctx, f.data_ptr(), self.writer.cuda_stream,
                                                        ctypes.byref(fi), ctypes.byref(ev)),
                   "reflex_pipeline_write_frame")
            self._window.append(f)
        return fi.value, ev.value

    def _staged(self, key, a):
        """Device fp32 view of an input; numpy inputs are copied into a
        persistent buffer so repeated calls keep the same device pointers (and
        so replay the same captured graph)."""
        torch = self.torch
        if isinstance(a, torch.Tensor) and a.device == self.device and a.dtype == torch.float32 \
                and a.is_contiguous():
            return a
        src = a if isinstance(a, torch.Tensor) else torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
        buf = self._bufs.get(key)
        if buf is None or tuple(buf.shape) != tuple(src.shape):
            buf = torch.empty(tuple(src.shape), dtype=torch.float32, device=self.device)
            self._bufs[key] = buf
        buf.copy_(src.to(torch.float32), non_blocking=False)
        return buf

    def denoise(self, state, noise, num_steps: Optional[int] = None, taus: Optional[Sequence[float]] = None,
                out=None, mode: str = "reflex", n_frames: Optional[int] = None, static_scratch: bool = False):
        """Denoise one chunk per env; returns the fp32 action tensor (device).

        Without ``out`` the result lands in a buffer owned by the engine that
        the next call overwrites.  The caller's current stream is ordered
        after the denoise, so reading the result there is safe.

        ``mode`` selects the cache strategy: "reflex" (the method), or the
        comparison baselines "standard" (the static prefix and the window's
        frames, as last passed to ``write_frame``, are encoded again before
        every step) and "naive" (the first step's dynamic K/V are reused).

        ``n_frames`` (pipelined ring, ``cfg.spare_slot = 1``) selects the
        window: the first n_frames frames, or -1 for the newest frame whose
        write has completed; the value used is left in ``last_n_frames``.

        ``static_scratch`` runs the chunk through the allocation-free entry
        point (the library's static device array holds the transient buffers,
        no graph).  ``taus`` may be a device tensor: the library copies it to
        the host on the engine stream."""
        torch = self.torch
        if mode not in MODES:
            raise ValueError(f"unknown mode {mode!r}")
        if n_frames is not None and mode != "reflex":
            raise ValueError("a pipelined window is only available to the method")
        k = num_steps if num_steps is not None else self.cfg.num_steps
        if taus is None and self.cfg.tau_schedule is not None and k == self.cfg.num_steps:
            taus = self.cfg.taus()  # the workload's own schedule
        caller = self._enter()
        with torch.cuda.stream(self.stream):
            s = self._staged("state", state)
            n = self._staged("noise", noise)
            if out is None:
                out = self._bufs.get("out")
                if out is None or tuple(out.shape) != tuple(n.shape):
                    out = torch.empty(tuple(n.shape), dtype=torch.float32, device=self.device)
                    self._bufs["out"] = out
            tau_arr = None
            if isinstance(taus, torch.Tensor) and taus.is_cuda:
                if taus.dtype != torch.float32 or taus.numel() != k + 1 or not taus.is_contiguous():
                    raise ValueError("a device tau schedule is a contiguous fp32 tensor of num_steps + 1 values")
                self._keep_taus = taus
                tau_arr = taus.data_ptr()
            elif taus is not None:
                tau_np = np.ascontiguousarray(np.asarray(taus, dtype=np.float32))
                if tau_np.shape[0] != k + 1:
                    raise ValueError("tau schedule needs num_steps + 1 entries")
                self._keep_taus = tau_np
                tau_arr = tau_np.ctypes.data
            if static_scratch:
                if mode != "reflex" or n_frames is not None:
                    raise ValueError("the allocation-free entry point computes the method over all frames")
                _check(self.lib.reflex_denoise_chunk_static(self.ctx, s.data_ptr(), n.data_ptr(), k, tau_arr,
                                                            out.data_ptr()), "reflex_denoise_chunk_static")
            elif n_frames is not None:
                used = c_i64(0)
                _check(self.lib.reflex_pipeline_denoise_chunk(self.ctx, s.data_ptr(), n.data_ptr(), k, tau_arr,
                                                              out.data_ptr(), n_frames, ctypes.byref(used)),
                       "reflex_pipeline_denoise_chunk")
                self.last_n_frames = used.value
            elif mode == "reflex":
                _check(self.lib.reflex_denoise_chunk(self.ctx, s.data_ptr(), n.data_ptr(), k, tau_arr,
                                                     out.data_ptr()), "reflex_denoise_chunk")
            else:
                src = self._sources() if mode == "standard" else None
                _check(self.lib.reflex_denoise_chunk_baseline(self.ctx, MODES[mode], src, s.data_ptr(),
                                                              n.data_ptr(), k, tau_arr, out.data_ptr()),
                       "reflex_denoise_chunk_baseline")
            self._keep_io = (s, n, out)
        caller.wait_stream(self.stream)
        return out

    def _sources(self):
        sk, sv = self._static
        frames = list(self._window)[-min(self.frames_written(), self.cfg.window_frames):] \
            if self.frames_written() else []
        arr = (c_vp * max(len(frames), 1))(*[f.data_ptr() for f in frames])
        src = SourcesC(static_k=sk.data_ptr() if sk.numel() else None,
                       static_v=sv.data_ptr() if sv.numel() else None,
                       frames=ctypes.cast(arr, ctypes.POINTER(c_vp)), n_frames=len(frames))
        self._keep_src = (arr, src)
        return ctypes.byref(src)

    def check_status(self) -> int:
        """reflex_check_status: waits for the engine stream; REFLEX_ENONFINITE
        when a chunk since the last check produced a non-finite action, else 0."""
        st = int(self.lib.reflex_check_status(self.ctx))
        if st not in (REFLEX_OK, REFLEX_ENONFINITE):
            _check(st, "reflex_check_status")
        return st

    def synchronize(self):
        if self.writer is not None:
            self.writer.synchronize()
        self.stream.synchronize()

    def frames_written(self) -> int:
        return int(self.lib.reflex_frames_written(self.ctx))

    def tick_state(self) -> Tuple[int, int, int]:
        """Device tick state (frames_written, n_valid, dyn_pos0), the first three
        of the four int64 at the start of the workspace."""
        self.synchronize()
        t = self.ws[:24].view(self.torch.int64).cpu().tolist()
        return int(t[0]), int(t[1]), int(t[2])

    def hole_row(self) -> int:
        """Fourth tick-state value: the logical cached row from which the
        physical rows skip the spare slot."""
        self.synchronize()
        return int(self.ws[24:32].view(self.torch.int64).cpu().item())

    def cache_views(self):
        """(K [B, L, R, dh], V^T [B, L, dh, R]) views of the cache, config dtype."""
        c = self.cfg
        R = c.cache_rows
        n = c.batch * c.n_layers * R * c.head_dim
        half = self.cache_bytes // 2
        esz = 2 if c.bf16 else 4
        k = self.cache[: n * esz].view(self.dtype).view(c.batch, c.n_layers, R, c.head_dim)
        v = self.cache[half: half + n * esz].view(self.dtype).view(c.batch, c.n_layers, c.head_dim, R)
        return k, v

    def _profiled(self, call) -> Dict[str, Tuple[float, int]]:
        _check(self.lib.reflex_profile_enable(self.ctx, 1), "reflex_profile_enable")
        try:
            call()
            self.synchronize()
            n = 32
            names = (ctypes.c_char_p * n)()
            ms = (c_f64 * n)()
            cnt = (c_i32 * n)()
            nc = c_i32(n)
            _check(self.lib.reflex_profile_read(self.ctx, names, ms, cnt, ctypes.byref(nc)), "reflex_profile_read")
            return {names[i].decode(): (ms[i], cnt[i]) for i in range(nc.value)}
        finally:
            self.lib.reflex_profile_enable(self.ctx, 0)

    def profile(self, state, noise, num_steps: Optional[int] = None,
                mode: str = "reflex") -> Dict[str, Tuple[float, int]]:
        """Run one denoise eagerly with per-launch events; {class: (ms, launches)}."""
        return self._profiled(lambda: self.denoise(state, noise, num_steps, mode=mode))

    def class_names(self) -> List[str]:
        """The library's kernel classes, in the bit order of class masks."""
        n = 32
        names = (ctypes.c_char_p * n)()
        ms = (c_f64 * n)()
        cnt = (c_i32 * n)()
        nc = c_i32(n)
        _check(self.lib.reflex_profile_read(self.ctx, names, ms, cnt, ctypes.byref(nc)), "reflex_profile_read")
        return [names[i].decode() for i in range(nc.value)]

    def profile_graph(self, state, noise, classes: Sequence[str], reps: int = 5,
                      num_steps: Optional[int] = None) -> Tuple[float, int]:
        """Device time of the given kernel classes inside the chunk's graph:
        one full denoise first, then a captured graph of the same chunk in
        which each launch of those classes is bracketed by wall-clock stamps
        (reflex_profile_graph), replayed reps times.  Returns (ms per chunk
        summed over those classes' launches, launches per chunk)."""
        names = self.class_names()
        unknown = [c for c in classes if c not in names]
        if unknown:
            raise ValueError(f"unknown kernel classes {unknown}")
        mask = 0
        for c in classes:
            mask |= 1 << names.index(c)
        k = num_steps if num_steps is not None else self.cfg.num_steps
        out = self.denoise(state, noise, k)
        s, n, _ = self._keep_io
        taus = self._keep_taus if (self.cfg.tau_schedule is not None and k == self.cfg.num_steps) else None
        tau_arr = taus.ctypes.data if isinstance(taus, np.ndarray) else None
        ms = c_f64(0.0)
        cnt = c_i32(0)
        _check(self.lib.reflex_profile_graph(self.ctx, s.data_ptr(), n.data_ptr(), k, tau_arr, out.data_ptr(),
                                             mask, reps, ctypes.byref(ms), ctypes.byref(cnt)),
               "reflex_profile_graph")
        return ms.value, cnt.value

    def profile_write(self, frame) -> Dict[str, Tuple[float, int]]:
        """Write one frame eagerly with per-launch events; {class: (ms, launches)}."""
        return self._profiled(lambda: self.write_frame(frame))

    def close(self):
        if self.ctx:
            self.synchronize()
            self.lib.reflex_destroy(self.ctx)
            self.ctx = c_vp(None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
