"""Future-conditional overlap scheduling (Section 3.3, Algorithm 1) around the
denoise engine.

A control loop executes one action per control period from a queue holding
the current chunk.  While the last K actions of the chunk run, the next chunk
is already being computed, so it is ready when the queue runs dry:

* K = ceil(mean inference latency / control period), re-estimated at every
  chunk from measured latencies (exponential moving average);
* the next inference is launched after C - K actions of the current chunk;
* it is conditioned on the predicted state at the hand-over, not on the
  sensor state at launch time: the policy computes actions for t + Delta, and
  with a low-level controller that tracks its commands the robot will be
  near the last commanded action, s_hat(t + Delta) ~ a_cmd(t) (the
  propagator returns the last action left in the queue).

Two comparison schedules run through the same loop:

* "sync": the next inference starts only when the queue is empty (K = 0), so
  every chunk stalls the robot for the inference latency;
* "async_naive": the overlap launch of Algorithm 1 without the future-state
  prediction: the chunk is conditioned on the sensor state at launch time.

Observation frames reach the engine's ring through the pipelined writer at
their capture time; a chunk reads the newest frame whose write has completed.
Reported: stall rate (control periods with no action to execute), reaction
latency (capture of the newest frame a chunk saw to the execution of that
chunk's first action), inference latency, the chosen K, and the state
alignment error at each hand-over (|conditioning state - robot state|).

The loop is written against small clock / policy interfaces so the same code
runs in real time on the GPU and on a simulated clock in host-only tests.
"""
from __future__ import annotations

import math
import time
from collections import deque
from dataclasses import dataclass, field
from typing import Callable, Deque, Dict, List, Optional

import numpy as np

STRATEGIES = ("reflex", "async_naive", "sync")


class FirstOrderRobot:
    """A robot whose controller tracks the commanded action with a first-order
    lag: s <- s + alpha * (a_cmd - s) each control period; without a command
    (a stall) it keeps moving toward the last one."""

    def __init__(self, state: np.ndarray, alpha: float = 0.5):
        self.s = np.asarray(state, dtype=np.float64).copy()
        self.alpha = float(alpha)
        self.cmd = self.s.copy()

    def step(self, action: Optional[np.ndarray]) -> None:
        if action is not None:
            self.cmd = np.asarray(action, dtype=np.float64)
        self.s = self.s + self.alpha * (self.cmd - self.s)


def predict_future_state(s_now: np.ndarray, queue: Deque[np.ndarray], k: int) -> np.ndarray:
    """Propagator of Algorithm 1 with the first-order approximation
    s_hat(t + Delta) ~ a_cmd: the last of the k actions still to be executed
    before the next chunk takes over (the sensor state if none is left)."""
    if k <= 0 or not queue:
        return np.asarray(s_now, dtype=np.float64).copy()
    return np.asarray(queue[min(k, len(queue)) - 1], dtype=np.float64).copy()


def overlap_steps(mean_latency_s: float, period_s: float, chunk: int) -> int:
    """K = ceil(mean inference latency / control period), kept below the chunk
    length (at least one action of a chunk runs before the next launch)."""
    k = int(math.ceil(mean_latency_s / period_s - 1e-9)) if mean_latency_s > 0 else 0
    return max(0, min(k, chunk - 1))


class RealClock:
    def now(self) -> float:
        return time.perf_counter()

    def sleep_until(self, t: float) -> None:
        while True:
            d = t - time.perf_counter()
            if d <= 0:
                return
            time.sleep(d - 0.0005 if d > 0.001 else 0)


class SimClock:
    """Simulated time for host-only tests: sleeping advances the clock."""

    def __init__(self):
        self.t = 0.0

    def now(self) -> float:
        return self.t

    def sleep_until(self, t: float) -> None:
        self.t = max(self.t, t)


@dataclass
class Launch:
    t_launch: float
    state: np.ndarray
    newest_frame: int      # index of the newest frame the chunk reads (-1: none)
    handle: object


@dataclass
class RunStats:
    strategy: str
    cycles: int = 0
    stalls: int = 0
    chunks: int = 0
    k_used: List[int] = field(default_factory=list)
    latency_s: List[float] = field(default_factory=list)
    reaction_s: List[float] = field(default_factory=list)
    state_err: List[float] = field(default_factory=list)

    def summary(self) -> Dict[str, object]:
        def pct(a, q):
            return round(float(np.percentile(np.asarray(a) * 1e3, q)), 3) if a else None

        return {
            "strategy": self.strategy,
            "cycles": self.cycles,
            "chunks": self.chunks,
            "stall_rate": round(self.stalls / max(1, self.cycles), 4),
            "k_mean": round(float(np.mean(self.k_used)), 2) if self.k_used else None,
            "inference_ms_mean": round(float(np.mean(self.latency_s)) * 1e3, 3) if self.latency_s else None,
            "reaction_ms_mean": round(float(np.mean(self.reaction_s)) * 1e3, 3) if self.reaction_s else None,
            "reaction_ms_p95": pct(self.reaction_s, 95),
            "state_err_mean": round(float(np.mean(self.state_err)), 5) if self.state_err else None,
        }


class OverlapScheduler:
    """Algorithm 1 control loop.

    policy: object with
      launch(state [ds]) -> handle   start one chunk inference (asynchronous)
      ready(handle) -> bool          inference finished
      result(handle) -> [C, da]      the chunk's actions (host)
      latency(handle) -> float       seconds from launch to completion
      frame_of(handle) -> int        index of the newest frame the chunk reads (-1: none)
      write_frame(index)             hand a captured frame to the pipelined writer
    """

    def __init__(self, policy, chunk: int, period_s: float, strategy: str = "reflex", ema: float = 0.3,
                 clock=None, frame_period_s: Optional[float] = None):
        if strategy not in STRATEGIES:
            raise ValueError(f"unknown strategy {strategy!r}")
        self.policy, self.C, self.period, self.strategy = policy, int(chunk), float(period_s), strategy
        self.ema = float(ema)
        self.clock = clock or RealClock()
        self.frame_period = frame_period_s

    def run(self, robot: FirstOrderRobot, n_cycles: int) -> RunStats:
        st = RunStats(self.strategy)
        clk, pol, C = self.clock, self.policy, self.C
        captured: Dict[int, float] = {}
        t0 = clk.now()
        next_frame_t = t0 if self.frame_period else None
        frame_idx = 0

        def capture(now):
            nonlocal next_frame_t, frame_idx
            while next_frame_t is not None and now >= next_frame_t:
                pol.write_frame(frame_idx)
                captured[frame_idx] = next_frame_t
                frame_idx += 1
                next_frame_t += self.frame_period

        def launch(state):
            t = clk.now()
            h = pol.launch(state)
            return Launch(t, np.asarray(state, dtype=np.float64).copy(), pol.frame_of(h), h)

        # initial inference (not counted): the first chunk, waited for
        capture(clk.now())
        first = launch(robot.s)
        while not pol.ready(first.handle):
            clk.sleep_until(clk.now() + self.period / 20)
        queue: Deque[np.ndarray] = deque(pol.result(first.handle))
        mean_lat = pol.latency(first.handle)
        k = overlap_steps(mean_lat, self.period, C) if self.strategy != "sync" else 0
        st.k_used.append(k)
        done_in_chunk = 0
        pending: Optional[Launch] = None
        # control ticks on the grid t0 + i * period (the camera's grid too)
        t_next = t0 + math.ceil((clk.now() - t0) / self.period - 1e-9) * self.period
        for _ in range(n_cycles):
            clk.sleep_until(t_next)
            now = clk.now()
            capture(now)
            if not queue and pending is not None and pol.ready(pending.handle):
                # hand-over: the awaited chunk replaces the empty queue
                lat = pol.latency(pending.handle)
                st.latency_s.append(lat)
                mean_lat = (1 - self.ema) * mean_lat + self.ema * lat
                queue = deque(pol.result(pending.handle))
                st.state_err.append(float(np.max(np.abs(pending.state - robot.s))))
                if pending.newest_frame >= 0:
                    st.reaction_s.append(now - captured[pending.newest_frame])
                st.chunks += 1
                pending = None
                done_in_chunk = 0
                k = overlap_steps(mean_lat, self.period, C) if self.strategy != "sync" else 0
                st.k_used.append(k)
            st.cycles += 1
            if queue:
                robot.step(queue.popleft())
                done_in_chunk += 1
                if pending is None and self.strategy != "sync" and done_in_chunk == C - k:
                    cond = predict_future_state(robot.s, queue, k) if self.strategy == "reflex" else robot.s
                    pending = launch(cond)
            else:
                st.stalls += 1
                robot.step(None)
                if pending is None:  # sync, or a chunk shorter than the overlap
                    pending = launch(robot.s)
            t_next += self.period
        return st


class SimPolicy:
    """Host-only stand-in for the engine: a fixed inference latency on a
    SimClock; the chunk's actions come from a callable of the state."""

    def __init__(self, clock: SimClock, latency_s: float, chunk_fn: Callable[[np.ndarray], np.ndarray],
                 write_latency_s: float = 0.0):
        self.clock, self.lat, self.fn, self.wlat = clock, float(latency_s), chunk_fn, float(write_latency_s)
        self.frames: Dict[int, float] = {}

    def write_frame(self, index: int) -> None:
        self.frames[index] = self.clock.now() + self.wlat  # completion time

    def launch(self, state):
        done = [i for i, t in self.frames.items() if t <= self.clock.now()]
        return (self.clock.now(), self.fn(np.asarray(state, dtype=np.float64)), max(done) if done else -1)

    def frame_of(self, h) -> int:
        return h[2]

    def ready(self, h) -> bool:
        return self.clock.now() >= h[0] + self.lat - 1e-12

    def result(self, h):
        return list(h[1])

    def latency(self, h) -> float:
        return self.lat


class EnginePolicy:
    """The denoise engine as the policy: chunks on the engine stream over the
    newest completed frame, frames through the pipelined writer.  Needs an
    engine with a spare ring slot; batch 1."""

    def __init__(self, engine, frames, noise_fn: Callable[[int], np.ndarray]):
        import torch

        self.torch, self.eng, self.frames, self.noise_fn = torch, engine, frames, noise_fn
        self.launched = 0
        self.written = 0
        self.base = engine.frames_written()  # frames from before this policy are not indexed

    def write_frame(self, index: int) -> None:
        self.eng.pipeline_write(self.frames[index % len(self.frames)])
        self.written = index + 1

    def frame_of(self, h) -> int:
        return max(-1, h["n"] - 1 - self.base)

    def launch(self, state):
        torch = self.torch
        # a host array: the engine copies it into one persistent device buffer,
        # so every chunk replays the same captured graph (a new device tensor
        # per launch would be a new pointer, and a new capture)
        st = np.ascontiguousarray(np.asarray(state, dtype=np.float32)[None])
        noise = self.noise_fn(self.launched)
        self.launched += 1
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(self.eng.stream)
        out = self.eng.denoise(st, noise, n_frames=-1 if self.eng.frames_written() else None)
        b.record(self.eng.stream)
        return {"out": out.clone(), "a": a, "b": b, "n": self.eng.last_n_frames}

    def ready(self, h) -> bool:
        return h["b"].query()

    def result(self, h):
        return list(h["out"][0].double().cpu().numpy())

    def latency(self, h) -> float:
        return h["a"].elapsed_time(h["b"]) / 1e3
