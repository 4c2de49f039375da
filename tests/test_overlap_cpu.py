"""Host-only checks of the Algorithm 1 overlap scheduler on a simulated clock
with a fixed-latency stand-in policy: the overlap K, the future-state
propagator, and the stall counts and reaction latencies that follow in closed
form from the schedule."""
import math
from collections import deque

import numpy as np
import pytest

from paper_2607_14695_amd import overlap as OV

P = 0.02  # control period (50 Hz)


def _ramp_policy(clock, latency, chunk, da=4, write_latency=0.0):
    """Each chunk moves the command linearly away from the conditioning state."""
    def fn(state):
        steps = np.arange(1, chunk + 1)[:, None] * 0.01
        return [state[:da] + s for s in steps]
    return OV.SimPolicy(clock, latency, fn, write_latency_s=write_latency)


def _run(strategy, latency, chunk=10, cycles=200, alpha=0.5, frame_period=None, write_latency=0.0):
    clk = OV.SimClock()
    pol = _ramp_policy(clk, latency, chunk, write_latency=write_latency)
    sch = OV.OverlapScheduler(pol, chunk, P, strategy=strategy, clock=clk, frame_period_s=frame_period)
    robot = OV.FirstOrderRobot(np.zeros(4), alpha=alpha)
    return sch.run(robot, cycles)


def test_overlap_steps_is_ceil_of_latency_over_period():
    assert OV.overlap_steps(0.0, P, 50) == 0
    assert OV.overlap_steps(0.011, P, 50) == 1
    assert OV.overlap_steps(0.020, P, 50) == 1
    assert OV.overlap_steps(0.0201, P, 50) == 2
    assert OV.overlap_steps(0.050, P, 50) == 3
    assert OV.overlap_steps(5.0, P, 50) == 49  # at least one action per chunk before the launch


def test_propagator_returns_last_command_before_handover():
    q = deque([np.full(2, i, dtype=float) for i in range(5)])
    s = np.array([9.0, 9.0])
    np.testing.assert_array_equal(OV.predict_future_state(s, q, 3), [2.0, 2.0])
    np.testing.assert_array_equal(OV.predict_future_state(s, q, 9), [4.0, 4.0])
    np.testing.assert_array_equal(OV.predict_future_state(s, q, 0), s)
    np.testing.assert_array_equal(OV.predict_future_state(s, deque(), 2), s)


@pytest.mark.parametrize("lat_periods", [0.5, 1.0, 2.5, 4.0])
def test_sync_stalls_for_the_inference_latency(lat_periods):
    chunk, cycles = 10, 400
    st = _run("sync", lat_periods * P, chunk=chunk, cycles=cycles)
    stalls_per_chunk = math.ceil(lat_periods - 1e-9)
    per = chunk + stalls_per_chunk
    assert st.stalls == (cycles // per) * stalls_per_chunk + max(0, cycles % per - chunk)
    assert all(k == 0 for k in st.k_used)


@pytest.mark.parametrize("strategy", ["reflex", "async_naive"])
@pytest.mark.parametrize("lat_periods", [0.5, 1.0, 2.5, 4.0])
def test_overlap_never_stalls_when_latency_is_steady(strategy, lat_periods):
    st = _run(strategy, lat_periods * P, chunk=10, cycles=400)
    assert st.stalls == 0
    assert set(st.k_used) == {math.ceil(lat_periods - 1e-9)}
    assert st.chunks == 400 // 10 - 1  # hand-overs after the initial chunk


def test_future_state_prediction_reduces_handover_error():
    """With a first-order robot that lags its commands, conditioning on the
    last command (reflex) lands closer to the robot's state at the hand-over
    than conditioning on the sensor state at launch (async_naive)."""
    good = _run("reflex", 2.5 * P, chunk=10, cycles=400, alpha=0.9)
    naive = _run("async_naive", 2.5 * P, chunk=10, cycles=400, alpha=0.9)
    assert good.summary()["state_err_mean"] < 0.5 * naive.summary()["state_err_mean"]


def test_reaction_latency_closed_forms():
    """Frames captured every control period, written instantly: an overlapped
    chunk launched at tick j reads the frame of tick j and starts at tick
    j + K + 1; a sync chunk launched at tick j starts at tick j + ceil(L / P)."""
    lat = 2.5 * P
    r = _run("reflex", lat, chunk=10, cycles=300, frame_period=P).reaction_s
    s = _run("sync", lat, chunk=10, cycles=300, frame_period=P).reaction_s
    np.testing.assert_allclose(r, (3 + 1) * P, atol=1e-9)
    np.testing.assert_allclose(s, 3 * P, atol=1e-9)


def test_reaction_latency_counts_write_time():
    """A frame whose write has not completed at launch is not read: the
    chunk reads the one before it, one frame period older."""
    lat = 1.5 * P
    r = _run("reflex", lat, chunk=10, cycles=300, frame_period=P, write_latency=0.5 * P).reaction_s
    np.testing.assert_allclose(r, (2 + 1) * P + P, atol=1e-9)


def test_k_adapts_to_a_latency_change():
    """Inference slows from 1.5 to 3.5 periods after the fifth launch: the
    first slow chunk arrives one period late (one stall), then K follows the
    measured latency and the stalls stop."""
    clk = OV.SimClock()
    pol = _ramp_policy(clk, 1.5 * P, 10)
    n = {"launch": 0}
    base_launch = pol.launch

    def launch(state):
        n["launch"] += 1
        pol.lat = 1.5 * P if n["launch"] <= 5 else 3.5 * P
        return base_launch(state)

    pol.launch = launch
    sch = OV.OverlapScheduler(pol, 10, P, strategy="reflex", clock=clk, ema=1.0)
    st = sch.run(OV.FirstOrderRobot(np.zeros(4)), 200)
    assert st.k_used[:5] == [2] * 5
    assert st.k_used[-1] == 4
    assert st.stalls == 1


def test_unknown_strategy_rejected():
    with pytest.raises(ValueError):
        OV.OverlapScheduler(None, 10, P, strategy="eager")


class _SlowOncePolicy(OV.SimPolicy):
    """A fixed inference latency, except that launch number `slow_index` is
    held up by `extra_s` more (a host stall inside one tick)."""

    def __init__(self, clock, latency_s, chunk_fn, slow_index, extra_s):
        super().__init__(clock, latency_s, chunk_fn)
        self.n, self.slow, self.extra = 0, slow_index, extra_s

    def launch(self, state):
        t, acts, fr = super().launch(state)
        lat = self.lat + (self.extra if self.n == self.slow else 0.0)
        self.n += 1
        return (t, acts, fr, lat)

    def ready(self, h):
        return self.clock.now() >= h[0] + h[3] - 1e-12

    def latency(self, h):
        return h[3]


@pytest.mark.parametrize("extra_periods", [0.5, 1.5, 3.5])
def test_forced_overrun_is_counted_as_stalls(extra_periods):
    """One chunk held up by a host stall: the overlapped schedule launched it
    with K actions left, the queue runs dry K + 1 periods after the launch and
    every further period until the chunk lands is a stall; the latency average
    then raises K, so the steady chunks after it do not stall."""
    chunk, lat = 10, 2.5 * P
    clk = OV.SimClock()
    fn = lambda s: [s[:4] + 0.01 * i for i in range(1, chunk + 1)]  # noqa: E731
    pol = _SlowOncePolicy(clk, lat, fn, slow_index=4, extra_s=extra_periods * P)
    sch = OV.OverlapScheduler(pol, chunk, P, strategy="reflex", clock=clk)
    st = sch.run(OV.FirstOrderRobot(np.zeros(4)), 300)
    k = math.ceil(lat / P - 1e-9)
    expect = max(0, math.ceil((lat + extra_periods * P) / P - 1e-9) - k - 1)
    assert st.stalls == expect, (st.stalls, expect)
    assert max(st.latency_s) == pytest.approx(lat + extra_periods * P)


def test_release_grid_counts_a_slow_tick_as_one_miss():
    """The benchmark's 20 ms release grid on a fake clock: a tick that takes
    2.5 periods is one missed deadline, and the next tick is released at the
    next grid point after it (no queue of late ticks)."""
    import bench

    t = {"now": 0.0}
    durations = iter([0.005, 0.005, 0.050, 0.005, 0.005])

    def tick():
        t["now"] += next(durations)

    def sleep(dt):
        t["now"] += dt

    def now():
        t["now"] += 1e-6  # a spin iteration costs a microsecond
        return t["now"]

    lat = bench.release_grid(tick, 5, 0.020, now=now, sleep=sleep)
    misses = [x > 0.020 for x in lat]
    assert misses == [False, False, True, False, False]
    assert lat[2] == pytest.approx(0.050, abs=1e-3)
    # the slow tick, released at 40 ms, ended at 90 ms: the next one waits for the 100 ms grid point
    assert lat[3] == pytest.approx(0.005, abs=1e-3)
