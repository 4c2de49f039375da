#!/usr/bin/env python3
"""Benchmark of the Reflex denoise hot path on one MI355X.

A "step" is one control tick of the pi0-scale single-chunk workload: write one
observation frame into the ring (768 tokens x 18 layers of K/V, RoPE at the
absolute position) and denoise one 50 x 32 action chunk with 10 Euler steps of
the 18-layer width-1024 action expert over 48 static + 768 window + 51 dynamic
tokens, batch 1, bf16 operands with fp32 statistics and accumulation.  Inputs
are resident in HBM before the timed region.

Prints one JSON line.  Besides the headline (chunks/s at batch 1), it reports
the denoise-step latency, a batch-32 tick (frames through the per-layer K/V
projection), per-kernel-class device times from the library's event profile,
the roofline of the dominant kernel and the float64 CPU oracle timed on this
host's cores as a reference baseline.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2607_14695_amd.profiling import load_traffic  # noqa: E402

METRIC = "denoise-step latency (us) + action chunks/s at batch 1/32; attn HBM GB/s"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0


def _device_inputs(cfg, torch, seed=0):
    """Synthetic weights / cache / inputs drawn on the device (values do not
    affect timing; parity is covered by the tests with the seeded generator)."""
    from paper_2607_14695_amd import workloads as WL

    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    dt = torch.bfloat16 if cfg.bf16 else torch.float32
    w = {}
    for name, shape in WL.weight_shapes(cfg).items():
        w[name] = (torch.randn(shape, generator=g, device="cuda") * WL.WEIGHT_STD).to(dt)
    shp = (cfg.batch, cfg.n_layers, cfg.static_len, cfg.head_dim)
    sk = torch.randn(shp, generator=g, device="cuda").to(dt)
    sv = torch.randn(shp, generator=g, device="cuda").to(dt)
    frames = [torch.randn((cfg.batch,) + WL.frame_shape(cfg), generator=g, device="cuda").to(dt) for _ in range(3)]
    state = torch.randn((cfg.batch, cfg.state_dim), generator=g, device="cuda")
    noise = torch.randn((cfg.batch, cfg.action_horizon, cfg.action_dim), generator=g, device="cuda")
    return w, sk, sv, frames, state, noise


def _class_bytes_flops(cfg):
    """Algorithmic HBM bytes and flops of ONE launch of each kernel class.

    GEMMs: weight bytes + activation bytes in + one copy of the output (fp32
    for the split-K residual projections, the operand type otherwise).
    Attention (with its split merge, one unit per layer): the visible cached K
    and V rows + q and the dynamic k, v in + o out, all in the operand type.
    Residual/norm: h and the projection in, h and y out, the modulation rows.
    Final kernel: h, the projection and the action head in, actions in and out;
    at every step but the last it also embeds the new actions for the next
    step (the embedding weights, state, h and y out, the modulation rows), so
    its figures are the average over a chunk's K launches.  Token embedding +
    first norm (once per chunk): the embedding weights, state, x in, h and y
    out.  Modulation (three launches per chunk): the conditioning weights."""
    B, T = cfg.batch, cfg.action_horizon + 1
    M = B * T
    D, Fm, Hq, dh = cfg.width, cfg.mlp_dim, cfg.n_q_heads, cfg.head_dim
    eb = 2 if cfg.bf16 else 4
    nqkv = (Hq + 2) * dh
    Lc = cfg.static_len + cfg.window_frames * cfg.frame_tokens
    out = {
        "gemm_qkv": (nqkv * D * eb + M * D * eb + M * nqkv * eb, 2.0 * M * nqkv * D),
        "gemm_o": (D * Hq * dh * eb + M * Hq * dh * eb + M * D * 4, 2.0 * M * D * Hq * dh),
        "gemm_gate_up": (2 * Fm * D * eb + M * D * eb + M * Fm * eb, 2.0 * M * 2 * Fm * D),
        "gemm_down": (D * Fm * eb + M * Fm * eb + M * D * 4, 2.0 * M * D * Fm),
    }
    vis = Lc * T + (1 + (T - 1) * T)  # visible keys summed over the dynamic rows of one env
    out["attention"] = (B * (2 * Lc * dh * eb + T * Hq * dh * eb + 2 * T * dh * eb + T * Hq * dh * eb),
                        B * 4.0 * Hq * dh * vis)
    out["resid_norm"] = (_norm_bytes(cfg), 0.0)
    da, ds = cfg.action_dim, cfg.state_dim
    K = cfg.num_steps
    nxt = (K - 1) / K  # share of the final launches that embed the next step
    out["final_euler"] = (M * D * 4 * 2 + da * D * eb + 2 * B * (T - 1) * da * 4 + B * 6 * D * 4
                          + nxt * (D * (ds + da) * eb + B * ds * 4 + M * D * (4 + eb) + B * 3 * D * 4),
                          2.0 * B * (T - 1) * da * D + nxt * 2.0 * B * (ds + (T - 1) * da) * D)
    out["embed_norm"] = (D * (ds + da) * eb + B * ds * 4 + B * (T - 1) * da * 4 + M * D * (4 + eb) + B * 3 * D * 4,
                         2.0 * B * (ds + (T - 1) * da) * D)
    S = 2 * cfg.n_layers + 1
    ch, C = cfg.cond_hidden, D + ds
    out["modulation"] = ((S * ch * C + S * 3 * D * ch) * eb / 3.0,
                         2.0 * cfg.num_steps * B * S * (ch * C + 3 * D * ch) / 3.0)
    return out


def _roofline(kernel, bound, nbytes, flops, seconds, traffic=None):
    """Roofline object of one kernel class from its algorithmic bytes/flops per
    launch and its average launch duration."""
    if bound == "mfma":
        achieved, peak, unit = flops / seconds / 1e12, BF16_PEAK_TFLOPS, "TFLOP/s"
    else:
        achieved, peak, unit = nbytes / seconds / 1e9, HBM_PEAK_GBS, "GB/s"
    return {"kernel": kernel, "bound": bound, "achieved": round(achieved, 1), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "traffic": traffic, "avg_us": round(seconds * 1e6, 3)}


def _graph_profile(eng, state, noise, reps=3):
    """{class: (ms per chunk, launches per chunk)}, each kernel class timed
    inside the chunk's captured graph: its launches bracketed by wall-clock
    stamp kernels, each bracket less the cost of a launch boundary measured at
    the same point (reflex_profile_graph), so every kernel runs in the chunk's
    own order and cache state.  Launch counts from one eager profiled chunk.
    "attention_unit" is the attention kernel and its split merge (one unit
    per layer)."""
    eager = eng.profile(state, noise)
    out = {}
    for cls, (_, n) in eager.items():
        if n and cls not in ("frame_proj", "ring_write"):
            # at least 30 stamped launches per class: a class launched once
            # per chunk has one boundary calibration per replay
            out[cls] = eng.profile_graph(state, noise, [cls], reps=max(reps, -(-30 // n)))
    if out.get("attn_merge", (0, 0))[1]:
        ms, _ = eng.profile_graph(state, noise, ["attention", "attn_merge"], reps=reps)
        out["attention_unit"] = (ms, out["attention"][1])
    return out


def _class_times(prof):
    """{class: (total ms, launches)} with the attention merge folded into the
    attention (one attention unit per layer: the kernel and its merge)."""
    out = {k: v for k, v in prof.items() if v[1] and k not in ("attn_merge", "attention_unit")}
    if "attention_unit" in prof:
        out["attention"] = prof["attention_unit"]
    elif "attention" in out and prof.get("attn_merge", (0, 0))[1]:
        out["attention"] = (out["attention"][0] + prof["attn_merge"][0], out["attention"][1])
    return out


def _avg_us(prof):
    """Average device microseconds per launch of every timed class."""
    return {k: round(v[0] / v[1] * 1e3, 3) for k, v in prof.items() if v[1] and k != "attention_unit"}


def _norm_bytes(cfg):
    """Algorithmic bytes of one residual + AdaRMSNorm launch: read h and the
    projection output, write h (fp32) and y (operand type), plus the gate,
    scale and shift rows of every env."""
    M = cfg.batch * (cfg.action_horizon + 1)
    eb = 2 if cfg.bf16 else 4
    return M * cfg.width * (4 + 4 + 4 + eb) + cfg.batch * 3 * cfg.width * 4


def _ring_bytes(cfg, prof_w):
    """(bytes, flops) of the ring writer's launches for one frame of all envs.
    Direct path: pre-RoPE K/V in, RoPE'd K and V^T out.  Embedding path: the
    frame projection GEMM, whose epilogue writes RoPE'd K and V^T into the
    cache (frame + per-layer Wk/Wv in, bf16 K/V out)."""
    eb = 2 if cfg.bf16 else 4
    kv = cfg.batch * cfg.n_layers * 2 * cfg.frame_tokens * cfg.head_dim  # K and V elements
    if cfg.frame_dim == 0:
        return {"ring_write": (2 * kv * eb, 0.0)}
    n = cfg.n_layers * 2 * cfg.head_dim
    m = cfg.batch * cfg.frame_tokens
    return {"frame_proj": (m * cfg.frame_dim * eb + n * cfg.frame_dim * eb + m * n * eb, 2.0 * m * n * cfg.frame_dim)}


def release_grid(tick, ticks, period_s, now=time.perf_counter, sleep=time.sleep):
    """Latencies (s) of `ticks` calls of tick() released on a grid of period_s:
    a tick's latency runs from its release to tick()'s return.  A tick that
    would start after its release starts at once, and no queue builds up behind
    a slow tick: the next release is the first grid point not already passed.
    A latency above period_s is a missed deadline."""
    lat = []
    t0 = now()
    k = 0
    for _ in range(ticks):
        release = t0 + k * period_s
        cur = now()
        if cur < release:
            sleep(max(0.0, release - cur - 0.0005))
            while now() < release:
                pass
        tick()
        done = now()
        lat.append(done - release)
        k = int((done - t0) / period_s) + 1
    return lat



def _on(eng, torch):
    """Make the engine's stream the current stream for the measurements that
    follow (ReflexEngine.current: the calls then leave no wait for the
    engine's work pending in another hardware queue while it runs); returns
    the stream that was current."""
    prev = torch.cuda.current_stream()
    torch.cuda.set_stream(eng.stream)
    return prev


def _off(eng, prev, torch):
    eng.synchronize()
    torch.cuda.set_stream(prev)


def _stream_ticks(eng, frames, state, noise, ticks, warmup, torch, period_s=0.020):
    """Tick latency on the 20 ms release grid (release_grid): frame write +
    denoise, synced on the device."""
    import numpy as np

    for i in range(warmup):
        eng.write_frame(frames[i % len(frames)])
        eng.denoise(state, noise)
    eng.synchronize()
    torch.cuda.synchronize()
    it = [0]

    def tick():
        eng.write_frame(frames[it[0] % len(frames)])
        eng.denoise(state, noise)
        eng.synchronize()
        torch.cuda.synchronize()
        it[0] += 1

    a = np.array(release_grid(tick, ticks, period_s)) * 1e3
    return {"period_ms": period_s * 1e3, "ticks": ticks, "p50_ms": round(float(np.percentile(a, 50)), 3),
            "p99_ms": round(float(np.percentile(a, 99)), 3), "mean_ms": round(float(a.mean()), 3),
            "misses": int((a > period_s * 1e3).sum())}


def _time_ticks(eng, frames, state, noise, steps, warmup, torch, denoise_only=False):
    for i in range(warmup):
        if not denoise_only:
            eng.write_frame(frames[i % len(frames)])
        eng.denoise(state, noise)
    eng.synchronize()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        if not denoise_only:
            eng.write_frame(frames[i % len(frames)])
        eng.denoise(state, noise)
    eng.synchronize()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / steps


def _chunk_latencies(eng, state, noise, n, torch, warmup=20):
    """Device time of n back-to-back single chunks, each bracketed by events on
    the engine's stream (ms): mean and percentiles, after `warmup` untimed
    chunks."""
    import numpy as np

    for _ in range(warmup):
        eng.denoise(state, noise)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    for a, b in evs:
        a.record(eng.stream)
        eng.denoise(state, noise)
        b.record(eng.stream)
    eng.synchronize()
    torch.cuda.synchronize()
    ms = np.array([a.elapsed_time(b) for a, b in evs])
    return {"mean": round(float(ms.mean()), 4), "p50": round(float(np.percentile(ms, 50)), 4),
            "p95": round(float(np.percentile(ms, 95)), 4), "p99": round(float(np.percentile(ms, 99)), 4), "n": n}


def _mode_chunks(eng, state, noise, torch, n):
    """Device time per chunk (ms, mean of n back-to-back chunks between two
    events on the engine's stream) under each cache strategy, once the ring is
    full, plus how far the naive strategy's actions land from the method's."""
    out, acts = {}, {}
    for mode in ("reflex", "standard", "naive", "unfused"):
        acts[mode] = eng.denoise(state, noise, mode=mode).clone()  # captures the graph
        eng.denoise(state, noise, mode=mode)
        eng.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(eng.stream)
        for _ in range(n):
            eng.denoise(state, noise, mode=mode)
        b.record(eng.stream)
        eng.synchronize()
        out[f"{mode}_chunk_ms"] = round(a.elapsed_time(b) / n, 4)
    out["standard_over_reflex"] = round(out["standard_chunk_ms"] / out["reflex_chunk_ms"], 3)
    # the fusion ablation: the same chunk with every fusion undone
    out["unfused_over_reflex"] = round(out["unfused_chunk_ms"] / out["reflex_chunk_ms"], 3)
    out["standard_equals_reflex"] = bool(torch.equal(acts["reflex"], acts["standard"]))
    d = (acts["naive"] - acts["reflex"]).double()
    out["naive_vs_reflex_mse"] = float((d * d).mean())
    out["naive_vs_reflex_maxabs"] = float(d.abs().max())
    out["chunks_timed"] = n
    return out


def _pipeline(cfg, w, sk, sv, frames, state, noise, torch, rounds, warmup):
    """Tick time of frame write + chunk on a ring with a spare slot, run both
    ways in alternation so drift between them cancels: "sequential" = write
    then chunk on the engine stream (the chunk reads every frame written);
    "pipelined" = the write on the engine's second stream while the chunk, on
    the engine stream, reads the frames written before this tick's frame
    (asynchronous pipeline, Section 3.3).  Each tick is bracketed by events on
    the engine stream, made current, which waits for the writer stream at the
    end (device time), and by the host clock (tick latency including launch).
    The window a chunk read is checked on every tick; the write and the chunk
    alone are timed the same way."""
    import numpy as np

    from paper_2607_14695_amd.reflex import ReflexEngine

    eng = ReflexEngine(cfg.replace(spare_slot=1), w, sk, sv)
    prev = _on(eng, torch)
    cur = torch.cuda.current_stream()
    for i in range(cfg.window_frames):
        eng.write_frame(frames[i % len(frames)])
    eng.synchronize()
    times = {k: ([], []) for k in ("sequential", "pipelined", "write", "chunk")}
    for r in range(warmup + rounds):
        for kind in ("sequential", "pipelined", "write", "chunk"):
            fr = frames[(r + len(kind)) % len(frames)]
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            t0 = time.perf_counter()
            a.record(cur)
            f_before = eng.frames_written()
            if kind == "sequential":
                eng.write_frame(fr)
                out = eng.denoise(state, noise)
            elif kind == "pipelined":
                eng.pipeline_write(fr)
                out = eng.denoise(state, noise, n_frames=f_before)
                if eng.last_n_frames != f_before:
                    raise RuntimeError(f"pipelined chunk read {eng.last_n_frames} frames, expected {f_before}")
            elif kind == "write":
                eng.write_frame(fr)
                out = None
            else:
                out = eng.denoise(state, noise)
            if eng.writer is not None:
                cur.wait_stream(eng.writer)
            cur.wait_stream(eng.stream)
            b.record(cur)
            b.synchronize()
            host = time.perf_counter() - t0
            if out is not None and not bool(torch.isfinite(out).all()):
                raise RuntimeError(f"non-finite actions in the {kind} pipeline tick")
            if r >= warmup:
                times[kind][0].append(a.elapsed_time(b))
                times[kind][1].append(host * 1e3)
    res = {}
    for kind, (dev, host) in times.items():
        d, h = np.array(dev), np.array(host)
        res[f"{kind}_ms"] = round(float(d.mean()), 4)
        res[f"{kind}_ms_spread"] = [round(float(np.percentile(d, 10)), 4), round(float(np.percentile(d, 90)), 4)]
        res[f"{kind}_host_ms"] = round(float(h.mean()), 4)
    res["pipelined_speedup"] = round(res["sequential_ms"] / res["pipelined_ms"], 4)
    spread = max(res["sequential_ms_spread"][1] - res["sequential_ms_spread"][0],
                 res["pipelined_ms_spread"][1] - res["pipelined_ms_spread"][0])
    # share of the write's time taken off the tick by running it beside the
    # chunk; omitted when the write is shorter than the tick-to-tick spread
    if res["write_ms"] > spread:
        res["write_hidden_fraction"] = round((res["sequential_ms"] - res["pipelined_ms"]) / res["write_ms"], 3)
    else:
        res["write_hidden_fraction"] = None
    res["rounds"] = rounds
    _off(eng, prev, torch)
    eng.close()
    return res


def _scheduler(cfg, w, sk, sv, frames, noise, torch, chunks):
    """Algorithm 1 in real time around the engine at batch 1: 50-action chunks
    at a 20 ms control period, a frame every period through the pipelined
    writer, a first-order robot; stall rate, reaction latency, inference
    latency and hand-over state error for each schedule."""
    import numpy as np

    from paper_2607_14695_amd import overlap as OV
    from paper_2607_14695_amd.reflex import ReflexEngine

    eng = ReflexEngine(cfg.replace(spare_slot=1), w, sk, sv)
    prev = _on(eng, torch)
    out = {}
    for strategy in OV.STRATEGIES:
        pol = OV.EnginePolicy(eng, frames, lambda i: noise)
        sch = OV.OverlapScheduler(pol, cfg.action_horizon, 0.020, strategy=strategy, frame_period_s=0.020)
        st = sch.run(OV.FirstOrderRobot(np.zeros(cfg.state_dim), alpha=0.5), chunks * cfg.action_horizon)
        out[strategy] = st.summary()
    _off(eng, prev, torch)
    eng.close()
    return out


def _event_ms(eng, torch, fn, n):
    """Mean device ms of n back-to-back calls of fn, between two events on the
    engine's stream (after one untimed call)."""
    fn()
    eng.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(eng.stream)
    for _ in range(n):
        fn()
    b.record(eng.stream)
    eng.synchronize()
    return round(a.elapsed_time(b) / n, 4)


def sweep_window(torch, log, windows=(1, 2, 5, 10, 20, 50)):
    """Context-window sweep (Section 4.6, context window size): batch 1,
    768-token frames through the per-layer Wk/Wv, the ring filled with W
    frames; chunk time of the method and of the Standard recompute, the
    attention launch time, and a tick (write + chunk)."""
    from paper_2607_14695_amd import workloads as WL
    from paper_2607_14695_amd.reflex import ReflexEngine

    base = WL.CONFIGS["pi0_stream_bf16"]
    w, sk, sv, frames, state, noise = _device_inputs(base, torch, seed=3)
    rows = []
    for W in windows:
        cfg = base.replace(window_frames=W)
        eng = ReflexEngine(cfg, w, sk, sv)
        prev = _on(eng, torch)
        for i in range(W):
            eng.write_frame(frames[i % len(frames)])
        r = {"window_frames": W, "cached_tokens": cfg.static_len + W * cfg.frame_tokens}
        r["reflex_chunk_ms"] = _event_ms(eng, torch, lambda: eng.denoise(state, noise), 10)
        r["standard_chunk_ms"] = _event_ms(eng, torch, lambda: eng.denoise(state, noise, mode="standard"), 3)
        r["standard_over_reflex"] = round(r["standard_chunk_ms"] / r["reflex_chunk_ms"], 3)
        a_ms, a_n = eng.profile_graph(state, noise, ["attention"])
        m_ms, m_n = eng.profile_graph(state, noise, ["attn_merge"])  # (0, 0) with one key split
        r["attention_us"] = round(a_ms / a_n * 1e3, 3)
        r["attn_merge_us"] = round(m_ms / m_n * 1e3, 3) if m_n else 0.0
        k = [0]

        def tick():
            eng.write_frame(frames[k[0] % len(frames)])
            k[0] += 1
            eng.denoise(state, noise)

        r["tick_ms"] = _event_ms(eng, torch, tick, 10)
        _off(eng, prev, torch)
        eng.close()
        log(f"window {r}")
        rows.append(r)
    return rows


def sweep_chunk(torch, log, horizons=(25, 50, 75, 100)):
    """Action-chunk sweep: 10-step chunk time for H actions at batch 1 and 32
    (2-frame ring of 768-token frames, 48 static tokens)."""
    from paper_2607_14695_amd import workloads as WL
    from paper_2607_14695_amd.reflex import ReflexEngine

    rows = []
    for name in ("pi0_stream_bf16", "pi0_batch32_bf16"):
        base = WL.CONFIGS[name]
        w, sk, sv, frames, state, _ = _device_inputs(base, torch, seed=4)
        for H in horizons:
            cfg = base.replace(action_horizon=H)
            noise = torch.randn((cfg.batch, H, cfg.action_dim), device="cuda")
            eng = ReflexEngine(cfg, w, sk, sv)
            prev = _on(eng, torch)
            for i in range(cfg.window_frames):
                eng.write_frame(frames[i])
            ms = _event_ms(eng, torch, lambda: eng.denoise(state, noise), 5)
            _off(eng, prev, torch)
            r = {"workload": name, "batch": cfg.batch, "action_horizon": H, "dynamic_tokens": H + 1,
                 "chunk_ms": ms, "denoise_step_us": round(ms / cfg.num_steps * 1e3, 1),
                 "actions_per_s": round(cfg.batch * H / (ms / 1e3), 1)}
            eng.close()
            log(f"chunk {r}")
            rows.append(r)
        del w
    return rows


def soak(torch, log, ticks):
    """Stability stress (Section 4.6): the x64-embedding, 8-env, 8-frame workload
    streamed for `ticks` ticks in closed loop (each chunk's last action is the
    next tick's state), with the norm path in fp32 (the method), with a bf16
    residual stream and fp32 statistics, and fully in bf16.  Per variant: ticks
    with a non-finite action, the largest |action|, the chunk time, and the
    deviation from the fp32 trajectory over time (same frames and noise)."""
    from paper_2607_14695_amd import workloads as WL
    from paper_2607_14695_amd.reflex import ReflexEngine

    cfg = WL.CONFIGS["pi0_long_bf16"]
    w, sk, sv, frames, state, noise = _device_inputs(cfg, torch, seed=5)
    modes = ("fp32", "bf16_fp32_stats", "bf16")
    engs = {m: ReflexEngine(cfg.replace(norm_precision=m), w, sk, sv) for m in modes}
    st = {m: state.clone() for m in modes}
    bad = {m: torch.zeros(ticks, device="cuda") for m in modes}
    amax = {m: torch.zeros(ticks, device="cuda") for m in modes}
    dev = {m: torch.zeros(ticks, device="cuda") for m in modes}
    gen = torch.Generator(device="cuda")
    gen.manual_seed(7)
    t0 = time.perf_counter()
    for t in range(ticks):
        nz = torch.randn(noise.shape, generator=gen, device="cuda")
        outs = {}
        for m in modes:
            engs[m].write_frame(frames[t % len(frames)])
            outs[m] = engs[m].denoise(st[m], nz).clone()
        for m in modes:
            o = outs[m]
            fin = torch.isfinite(o)
            bad[m][t] = (~fin).any().float()
            amax[m][t] = torch.where(fin, o.abs(), torch.zeros_like(o)).max()
            dev[m][t] = (torch.nan_to_num(o, nan=1e30, posinf=1e30, neginf=-1e30) - outs["fp32"]).abs().max()
            # closed loop; a non-finite action leaves the state where it was
            nxt = o[:, -1, :cfg.state_dim]
            st[m] = torch.where(torch.isfinite(nxt), nxt, st[m])
        if (t + 1) % 250 == 0:
            torch.cuda.synchronize()
            log(f"soak tick {t + 1}/{ticks}: " + ", ".join(
                f"{m} bad={int(bad[m][:t + 1].sum())} dev={float(dev[m][t]):.3g}" for m in modes))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    out = {"workload": "pi0_long_bf16 (8 envs, 256 static + 8x768 ring, token embeddings x64, tau schedule "
                       "concentrated near 0 and 1), closed loop: state <- last action of the previous chunk",
           "ticks": ticks, "wall_s": round(wall, 1), "variants": {}}
    marks = [t for t in (0, 9, 99, 999, 1999, ticks - 1) if t < ticks]
    for m in modes:
        b = bad[m].cpu()
        first = int(b.nonzero()[0]) if b.any() else None
        out["variants"][m] = {
            "nonfinite_ticks": int(b.sum()), "first_nonfinite_tick": first,
            "max_abs_action": round(float(amax[m].max()), 4),
            "chunk_ms": _event_ms(engs[m], torch, lambda: engs[m].denoise(st[m], noise), 5),
            "dev_from_fp32_at_tick": {str(t + 1): round(float(dev[m][t]), 6) for t in marks},
            "dev_from_fp32_max": round(float(dev[m].max()), 6),
        }
        engs[m].close()
    return out


def _warm_clocks(torch, seconds=0.3):
    """Keep the GPU busy for `seconds` with library GEMMs before a profiled
    region.  After an idle spell the clocks take tens of milliseconds to come
    back up: in a kernel trace the first batch-32 chunk after idle averaged
    42 us per attention launch (46 us in its first step) against 39 us for
    every later chunk, with or without a frame write before it.  The warm-up
    kernels are not the library's and stay out of the profile tables."""
    a = torch.randn(8192, 8192, device="cuda", dtype=torch.bfloat16)
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(8):
            torch.matmul(a, a)
        torch.cuda.synchronize()
    del a


def profile_run(torch, log, name, ticks, stamps=False):
    """A short run of one workload for the profiler: the GPU warmed up, the
    ring filled, then `ticks` ticks of frame write + chunk through the
    captured graphs (the launch configuration of the timed benchmark), each
    tick synchronized.  With `stamps`, then the in-graph class timing the
    benchmark reports (_graph_profile), its per-launch microseconds in the
    returned record, so that a kernel trace of this run holds the very
    dispatches those figures measure."""
    from paper_2607_14695_amd import workloads as WL
    from paper_2607_14695_amd.reflex import ReflexEngine

    cfg = WL.CONFIGS[name]
    w, sk, sv, frames, state, noise = _device_inputs(cfg, torch)
    eng = ReflexEngine(cfg, w, sk, sv)
    _warm_clocks(torch)
    prev = _on(eng, torch)
    for i in range(cfg.window_frames):
        eng.write_frame(frames[i % len(frames)])
    for i in range(ticks):
        eng.write_frame(frames[i % len(frames)])
        out = eng.denoise(state, noise)
        eng.synchronize()
        if not bool(torch.isfinite(out).all()):
            raise RuntimeError(f"non-finite actions in the profiled {name} run")
        log(f"profile run {name}: tick {i + 1}/{ticks}")
    rec = {"metric": "profile_run", "workload": name, "ticks": ticks, "batch": cfg.batch}
    if stamps:
        gp = _graph_profile(eng, state, noise)
        rec["stamp_us"] = {k: round(v[0] / v[1] * 1e3, 3) for k, v in gp.items() if v[1]}
        log(f"profile run {name}: in-graph class timing done")
    _off(eng, prev, torch)
    eng.close()
    return rec


def cpu_baseline(cfg, log):
    """The float64 oracle timed on this host's cores: one full chunk (1 env,
    10 Euler steps, one frame in the window), median of four runs (about 12 s)."""
    import numpy as np

    from oracle import reflex_oracle as O
    from paper_2607_14695_amd import workloads as WL

    cores = len(os.sched_getaffinity(0))
    model = None
    try:
        import subprocess

        for line in subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout.splitlines():
            if line.startswith("Model name:"):
                model = line.split(":", 1)[1].strip()
                break
    except Exception:  # lscpu missing: the model stays unknown
        pass
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=cores)
    except Exception:  # threadpoolctl missing: BLAS uses its default pool
        limiter = None
    rng = np.random.default_rng(0)
    w = {}
    for name, shape in WL.weight_shapes(cfg).items():
        w[name] = rng.standard_normal(size=shape) * WL.WEIGHT_STD
    shp = (1, cfg.n_layers, cfg.static_len, cfg.head_dim)
    sk, sv = rng.standard_normal(size=shp), rng.standard_normal(size=shp)
    frames = {0: rng.standard_normal(size=(1,) + WL.frame_shape(cfg))}
    state = rng.standard_normal(size=(1, cfg.state_dim))
    noise = rng.standard_normal(size=(1, cfg.action_horizon, cfg.action_dim))
    times = []
    for _ in range(4):
        t0 = time.perf_counter()
        O.denoise_chunk(cfg, w, sk, sv, frames, 1, state, noise, cfg.taus())
        times.append(time.perf_counter() - t0)
        log(f"cpu oracle chunk: {times[-1]:.2f} s")
    sec = float(np.median(times))
    if limiter is not None:
        limiter.unregister()
    return {"value": 1.0 / sec, "unit": "chunks/s", "cores": cores, "cpu_model": model, "kind": "oracle",
            "sample": "one full pi0_chunk_bf16 chunk (env 0, 10 Euler steps, 48 static + 768 frame "
                      f"+ 51 dynamic tokens), float64 numpy, median of 4 runs = {sec:.2f} s/chunk"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-b32", action="store_true")
    ap.add_argument("--no-long", action="store_true",
                    help="skip the long-context stress chunk (batch 8, 8-frame ring, 6,400 cached tokens)")
    ap.add_argument("--no-latency", action="store_true",
                    help="skip the per-chunk event-timed latency distribution (for counter-collection runs)")
    ap.add_argument("--no-baselines", action="store_true",
                    help="skip the Standard / Naive-cache strategy timings")
    ap.add_argument("--no-pipeline", action="store_true",
                    help="skip the two-stream (asynchronous pipeline) tick timings")
    ap.add_argument("--no-scheduler", action="store_true",
                    help="skip the real-time Algorithm 1 scheduler run (about 10 s)")
    ap.add_argument("--sweep", choices=("window", "chunk", "all"),
                    help="instead of the benchmark line, print one JSON line of the window and/or chunk sweeps")
    ap.add_argument("--soak", type=int, metavar="TICKS",
                    help="instead of the benchmark line, print one JSON line of the norm-precision soak")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 256 MiB elementwise copy (reference for HBM byte counters)")
    ap.add_argument("--profile-workload", metavar="NAME",
                    help="instead of the benchmark line, run a few ticks of one workload (for rocprofv3)")
    ap.add_argument("--stamps", action="store_true",
                    help="with --profile-workload: also the benchmark's in-graph class timing")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(environments would shard over GPUs with replicated weights and no collective)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2607_14695_amd import workloads as WL
    from paper_2607_14695_amd.reflex import ReflexEngine

    def log(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    if args.soak:
        print(json.dumps({"metric": "soak", "data": "synthetic", "dtype": "bf16", **soak(torch, log, args.soak)}),
              flush=True)
        return

    if args.sweep:
        out = {"metric": "sweeps", "data": "synthetic", "dtype": "bf16"}
        if args.sweep in ("window", "all"):
            out["window"] = sweep_window(torch, log)
        if args.sweep in ("chunk", "all"):
            out["chunk"] = sweep_chunk(torch, log)
        print(json.dumps(out), flush=True)
        return

    if args.calibrate_copy:
        # a plain copy of known size: 256 MiB read + 256 MiB written per launch
        src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst
        log("calibration copy: 3 x 256 MiB")

    if args.profile_workload:
        print(json.dumps(profile_run(torch, log, args.profile_workload, max(1, args.steps), args.stamps)),
              flush=True)
        return

    cfg = WL.CONFIGS["pi0_chunk_bf16"]
    w, sk, sv, frames, state, noise = _device_inputs(cfg, torch)
    eng = ReflexEngine(cfg, w, sk, sv)
    prev = _on(eng, torch)
    log("engine ready (pi0_chunk_bf16)")
    tick_s = _time_ticks(eng, frames, state, noise, args.steps, args.warmup, torch)
    log(f"tick {tick_s * 1e3:.3f} ms")
    chunk_s = _time_ticks(eng, frames, state, noise, args.steps, args.warmup, torch, denoise_only=True)
    log(f"chunk {chunk_s * 1e3:.3f} ms")
    pw = eng.profile_write(frames[0])
    rb = _ring_bytes(cfg, pw)
    rw_ms, rw_n = pw["ring_write"]
    ring_gbs = rb["ring_write"][0] / (rw_ms / rw_n / 1e3) / 1e9
    lat = None
    if not args.no_latency:
        lat = _chunk_latencies(eng, state, noise, max(100, args.steps), torch)
        log(f"chunk latency p50 {lat['p50']:.3f} ms, p99 {lat['p99']:.3f} ms")
    finite = bool(torch.isfinite(eng.denoise(state, noise)).all())
    if not finite:
        raise RuntimeError("non-finite actions from the timed batch-1 configuration")
    prof = _graph_profile(eng, state, noise)
    log("profile: " + ", ".join(f"{k}={v[0]:.3f}ms/{v[1]}" for k, v in prof.items() if v[1]))
    bf = _class_bytes_flops(cfg)
    # the dominant kernel class: the largest share of the chunk's device time,
    # over every class (the attention counted with its split merge)
    ct = _class_times(prof)
    dominant = max((k for k in ct if k in bf), key=lambda k: ct[k][0])
    ms, n = ct[dominant]
    traffic = load_traffic(os.path.join(ROOT, "profiles", f"traffic_{cfg.name}.json"), dominant)
    roofline = _roofline(dominant, "hbm", bf[dominant][0], bf[dominant][1], ms / n / 1e3, traffic)
    roofline["share_of_chunk"] = round(ms / sum(v[0] for v in ct.values()), 4)
    attn_ms, attn_n = ct["attention"]
    attn_gbs = bf["attention"][0] / (attn_ms / attn_n / 1e3) / 1e9
    kernel_avg_us = _avg_us(prof)
    n_ms, n_n = prof["resid_norm"]
    norm_gbs = _norm_bytes(cfg) / (n_ms / n_n / 1e3) / 1e9
    _off(eng, prev, torch)
    eng.close()
    del eng, w

    b32 = None
    if not args.no_b32:
        c32 = WL.CONFIGS["pi0_batch32_bf16"]
        w32, sk32, sv32, fr32, st32, nz32 = _device_inputs(c32, torch, seed=1)
        e32 = ReflexEngine(c32, w32, sk32, sv32)
        prev = _on(e32, torch)
        steps32 = max(3, args.steps // 3)
        t32 = _time_ticks(e32, fr32, st32, nz32, steps32, 2, torch)
        c32s = _time_ticks(e32, fr32, st32, nz32, steps32, 1, torch, denoise_only=True)
        if not bool(torch.isfinite(e32.denoise(st32, nz32)).all()):
            raise RuntimeError("non-finite actions from the timed batch-32 configuration")
        p32 = _graph_profile(e32, st32, nz32)
        pw32 = e32.profile_write(fr32[0])
        rb32 = _ring_bytes(c32, pw32)
        bf32 = _class_bytes_flops(c32)
        ct32 = _class_times(p32)
        a_ms, a_n = ct32["attention"]
        b32 = {
            "workload": "pi0_batch32_bf16 tick: 32 envs, frame write through per-layer Wk/Wv 2048->256 "
                        "(embedding path) + 10-step denoise over 48 static + 2x768 ring + 51 dynamic tokens",
            "chunks_per_s": round(c32.batch / t32, 2),
            "tick_ms": round(t32 * 1e3, 3),
            "chunk_ms": round(c32s * 1e3, 3),
            "denoise_step_us": round(c32s / c32.num_steps * 1e6, 1),
            "attn_hbm_gbs": round(bf32["attention"][0] / (a_ms / a_n / 1e3) / 1e9, 1),
            "attn_mfma_tflops": round(bf32["attention"][1] / (a_ms / a_n / 1e3) / 1e12, 1),
            "kernel_avg_us": _avg_us(p32),
        }
        tf32 = os.path.join(ROOT, "profiles", f"traffic_{c32.name}.json")
        b32["roofline"] = {"attention": _roofline("attention", "hbm", *bf32["attention"], a_ms / a_n / 1e3,
                                                  load_traffic(tf32, "attention"))}
        for k in ("gemm_qkv", "gemm_gate_up", "gemm_o", "gemm_down"):
            ms_k, n_k = p32[k]
            b32[f"{k}_mfma_tflops"] = round(bf32[k][1] / (ms_k / n_k / 1e3) / 1e12, 1)
            b32["roofline"][k] = _roofline(k, "mfma", *bf32[k], ms_k / n_k / 1e3, load_traffic(tf32, k))
        proj_ms = sum(p32[k][0] for k in ("gemm_qkv", "gemm_gate_up", "gemm_o", "gemm_down"))
        b32["projections_us_per_step"] = round(proj_ms / c32.num_steps * 1e3, 1)
        fp_ms, fp_n = pw32["frame_proj"]
        b32["frame_proj_mfma_tflops"] = round(rb32["frame_proj"][1] / (fp_ms / fp_n / 1e3) / 1e12, 1)
        b32["roofline"]["frame_proj"] = _roofline("frame_proj", "mfma", *rb32["frame_proj"], fp_ms / fp_n / 1e3,
                                                  load_traffic(tf32, "frame_proj"))
        b32["write_us"] = {k: round(v[0] / v[1] * 1e3, 3) for k, v in pw32.items() if v[1]}
        n32_ms, n32_n = p32["resid_norm"]
        b32["norm_gbs"] = round(_norm_bytes(c32) / (n32_ms / n32_n / 1e3) / 1e9, 1)
        if not args.no_latency:
            # the batched streaming workload's 200 ticks, released on the 20 ms grid
            b32["stream_ticks"] = _stream_ticks(e32, fr32, st32, nz32, c32.ticks, 3, torch)
            log(f"b32 stream ticks: {b32['stream_ticks']}")
        if not args.no_baselines:
            b32["strategies"] = _mode_chunks(e32, st32, nz32, torch, 3)
            log(f"b32 strategies: {b32['strategies']}")
        _off(e32, prev, torch)
        e32.close()
        if not args.no_pipeline:
            b32["pipeline"] = _pipeline(c32, w32, sk32, sv32, fr32, st32, nz32, torch, 10, 2)
            log(f"b32 pipeline: {b32['pipeline']}")
        log(f"b32 tick {t32 * 1e3:.3f} ms, chunk {c32s * 1e3:.3f} ms")

    long_ctx = None
    if not args.no_long:
        # the stress workload where the attention dominates: 8 envs, 256 static
        # + 8 x 768 ring tokens, x64 embeddings, its own tau schedule
        cl = WL.CONFIGS["pi0_long_bf16"]
        wl, skl, svl, frl, stl, nzl = _device_inputs(cl, torch, seed=3)
        el = ReflexEngine(cl, wl, skl, svl)
        prev = _on(el, torch)
        for f in range(cl.window_frames):
            el.write_frame(frl[f % len(frl)])
        cls_ = _time_ticks(el, frl, stl, nzl, max(3, args.steps // 3), 1, torch, denoise_only=True)
        if not bool(torch.isfinite(el.denoise(stl, nzl)).all()):
            raise RuntimeError("non-finite actions from the timed long-context configuration")
        pl = _graph_profile(el, stl, nzl)
        bfl = _class_bytes_flops(cl)
        al_ms, al_n = _class_times(pl)["attention"]
        long_ctx = {
            "workload": "pi0_long_bf16 chunk: 8 envs, 256 static + 8 x 768 ring + 51 dynamic tokens, x64 "
                        "embeddings, tau schedule near 0 and 1, 10 Euler steps",
            "chunks_per_s": round(cl.batch / cls_, 2),
            "chunk_ms": round(cls_ * 1e3, 3),
            "attn_us": round(al_ms / al_n * 1e3, 2),
            "attn_hbm_gbs": round(bfl["attention"][0] / (al_ms / al_n / 1e3) / 1e9, 1),
            "attn_mfma_tflops": round(bfl["attention"][1] / (al_ms / al_n / 1e3) / 1e12, 1),
            "kernel_avg_us": _avg_us(pl),
        }
        tfl = os.path.join(ROOT, "profiles", f"traffic_{cl.name}.json")
        long_ctx["roofline"] = {"attention": _roofline("attention", "hbm", *bfl["attention"], al_ms / al_n / 1e3,
                                                       load_traffic(tfl, "attention"))}
        for k in ("gemm_qkv", "gemm_gate_up", "gemm_o", "gemm_down"):
            long_ctx["roofline"][k] = _roofline(k, "mfma", *bfl[k], pl[k][0] / pl[k][1] / 1e3, load_traffic(tfl, k))
        _off(el, prev, torch)
        el.close()
        del el, wl
        log(f"long context: {long_ctx}")

    stream = strategies = pipeline = scheduler = None
    if not (args.no_latency and args.no_baselines and args.no_pipeline and args.no_scheduler):
        cs = WL.CONFIGS["pi0_stream_bf16"]
        ws_, sks, svs, frs, sts, nzs = _device_inputs(cs, torch, seed=2)
        es = ReflexEngine(cs, ws_, sks, svs)
        prev = _on(es, torch)
        if not args.no_latency:
            stream = _stream_ticks(es, frs, sts, nzs, cs.ticks, 5, torch)
            stream["workload"] = ("pi0_stream_bf16: 1 env, 768-token frames of width 2048 through the per-layer "
                                  "Wk/Wv projection into a 2-frame ring, 10-step denoise per tick, ticks released "
                                  "every 20 ms")
            log(f"stream ticks: {stream}")
        if not args.no_baselines:
            while es.frames_written() < cs.window_frames:
                es.write_frame(frs[es.frames_written() % len(frs)])
            strategies = _mode_chunks(es, sts, nzs, torch, 20)
            strategies["workload"] = ("pi0_stream_bf16 chunk with a full 2-frame ring: Standard re-encodes the 48 "
                                      "static tokens and both 768-token frames (Wk/Wv projection + RoPE) before "
                                      "every Euler step; Naive reuses the first step's dynamic K/V")
            pst = es.profile(sts, nzs, mode="standard")
            strategies["standard_class_ms"] = {k: round(v[0], 4) for k, v in pst.items() if v[1]}
            log(f"strategies: {strategies}")
        _off(es, prev, torch)
        es.close()
        if not args.no_pipeline:
            pipeline = _pipeline(cs, ws_, sks, svs, frs, sts, nzs, torch, 30, 3)
            pipeline["workload"] = ("pi0_stream_bf16 tick on a ring with one spare slot: 768x2048 frame through the "
                                    "per-layer Wk/Wv projection + 10-step chunk; pipelined = write on a second "
                                    "stream, chunk over the frames before it")
            log(f"pipeline: {pipeline}")
        if not args.no_scheduler:
            scheduler = _scheduler(cs, ws_, sks, svs, frs, nzs, torch, 3)
            scheduler["workload"] = ("pi0_stream_bf16 at batch 1: Algorithm 1 with 50-action chunks at a 20 ms "
                                     "control period, a 768x2048 frame every period through the pipelined writer, "
                                     "first-order robot (alpha 0.5); 150 control periods per schedule (the first chunk, then two hand-overs)")
            log(f"scheduler: {scheduler}")
        del es, ws_

    cpu = None if args.no_cpu_baseline else cpu_baseline(cfg, log)

    result = {
        "metric": METRIC,
        "value": round(cfg.batch / tick_s, 3),
        "unit": "chunks/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(tick_s * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "pi0_chunk_bf16 tick: 18-layer width-1024 action expert (MLP 4096, 8 q heads / 1 kv "
                        "head of 256), one 768-token frame written to a 1-frame ring (direct K/V path) + "
                        "10-step Euler denoise of a 50x32 action chunk over 48 static + 768 frame + 51 "
                        "dynamic tokens",
            "batch": cfg.batch,
            "euler_steps": cfg.num_steps,
            "cached_tokens": cfg.static_len + cfg.window_frames * cfg.frame_tokens,
        },
        "denoise_step_us": round(chunk_s / cfg.num_steps * 1e6, 2),
        "chunk_ms": round(chunk_s * 1e3, 4),
        "chunk_latency_ms": lat,
        "attn_hbm_gbs": round(attn_gbs, 1),
        "norm_gbs": round(norm_gbs, 1),
        "ring_write_gbs": round(ring_gbs, 1),
        "ring_write_us": round(rw_ms / rw_n * 1e3, 3),
        "stream_ticks": stream,
        "strategies": strategies,
        "pipeline": pipeline,
        "scheduler": scheduler,
        "kernel_avg_us": kernel_avg_us,
        "roofline": roofline,
        "b32": b32,
        "long_ctx": long_ctx,
        "cpu_baseline": cpu,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
