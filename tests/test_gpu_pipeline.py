"""GPU checks of the asynchronous pipeline (Section 3.3): frames written on a
second stream while chunks are denoised on the context's stream, over a ring
with one spare slot.

* With the spare slot and synchronous calls, every chunk matches the oracle
  (frame f lands in slot f mod (W+1); the window is read around the spare
  slot), and the tick state holds the documented values.
* Pipelined (writer stream + denoise stream, each chunk one frame behind the
  writer), every chunk equals bit for bit the chunk a synchronously driven
  context computes over the same frames, through several wraps of the ring.
* The "newest completed write" choice returns a legal window and its chunk.
* Misuse is rejected with REFLEX_EINVAL."""
import numpy as np
import pytest
import torch

from oracle import reflex_oracle as O
from paper_2607_14695_amd import reflex as R
from paper_2607_14695_amd import workloads as WL

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-4
BF16_REL, BF16_ABS = 1e-2, 5e-2

RAGGED = WL.CONFIGS["tiny_fp32"].replace(
    name="ragged_fp32", batch=3, static_len=40, frame_tokens=24, window_frames=3, action_horizon=5,
    n_q_heads=3, head_dim=128, width=128, mlp_dim=192, cond_hidden=64, state_dim=8, action_dim=5,
    frame_dim=72, n_layers=2, num_steps=3)

SPARE_CASES = {
    "tiny_fp32": WL.CONFIGS["tiny_fp32"].replace(spare_slot=1),
    "ragged_bf16_dh256_direct": RAGGED.replace(name="sp256", dtype="bf16", head_dim=256, frame_dim=0,
                                               spare_slot=1),
    "ragged_fp32_w1_embed": RAGGED.replace(name="sp1", window_frames=1, spare_slot=1),
}


def _setup(cfg, ticks):
    w = WL.make_weights(cfg)
    sk, sv = WL.make_static_kv(cfg)
    frames = {t: WL.make_frame(cfg, t) for t in range(ticks)}
    return w, sk, sv, frames


def _close(cfg, got, ref):
    if cfg.bf16:
        rel = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
        return rel <= BF16_REL and float(np.max(np.abs(got - ref))) <= BF16_ABS
    return float(np.max(np.abs(got - ref))) <= FP32_TOL


@pytest.mark.parametrize("case", sorted(SPARE_CASES))
def test_spare_slot_layout_matches_oracle(case):
    cfg = SPARE_CASES[case]
    ticks = 2 * (cfg.window_frames + 1) + 1
    w, sk, sv, frames = _setup(cfg, ticks)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    slots = cfg.window_frames + 1
    for t in range(ticks):
        f, ev = eng.write_frame(frames[t])
        st = O.ring_step(t, cfg.window_frames, cfg.frame_tokens, cfg.static_len)
        assert (f, ev) == (st.frame_index, st.evicted)
        assert eng.tick_state() == (t + 1, st.n_valid, st.dyn_pos0)
        assert eng.hole_row() == cfg.static_len + ((t + 1) % slots) * cfg.frame_tokens
        if cfg.frame_dim > 0 and not cfg.bf16:
            # frame t's keys sit in slot t mod (W + 1)
            K, _ = eng.cache_views()
            r0 = cfg.static_len + (t % slots) * cfg.frame_tokens
            kf, _ = O.frame_kv(cfg, w, frames[t][0], t, 0)
            np.testing.assert_allclose(K[0, 0, r0:r0 + cfg.frame_tokens].cpu().numpy(), kf[:, 0],
                                       rtol=1e-4, atol=1e-4)
        if t in (0, cfg.window_frames, ticks - 1):
            print(f"spare {case} after {t + 1} frames", flush=True)
            state, noise = WL.make_state(cfg, t), WL.make_noise(cfg, t)
            got = eng.denoise(state, noise).cpu().numpy()
            ref = O.denoise_chunk(cfg, w, sk, sv, frames, t + 1, state, noise, cfg.taus())
            assert _close(cfg, got, ref), (case, t)
    eng.close()


@pytest.mark.parametrize("case", sorted(SPARE_CASES))
def test_pipelined_chunks_equal_sequential_chunks(case):
    cfg = SPARE_CASES[case]
    ticks = 3 * (cfg.window_frames + 1) + 2
    w, sk, sv, frames = _setup(cfg, ticks)
    # reference: a synchronously driven context, chunk after n frames for every n
    seq = R.ReflexEngine(cfg, w, sk, sv)
    ref = {}
    for n in range(ticks + 1):
        if n > 0:
            seq.write_frame(frames[n - 1])
        ref[n] = seq.denoise(WL.make_state(cfg, n), WL.make_noise(cfg, n)).clone()
    seq.synchronize()
    seq.close()

    eng = R.ReflexEngine(cfg, w, sk, sv)
    outs = {}
    for t in range(ticks):
        eng.pipeline_write(frames[t])  # frame t on the writer stream
        # one frame behind: the window of frames < t, overlapping the write
        out = eng.denoise(WL.make_state(cfg, t), WL.make_noise(cfg, t), n_frames=t)
        assert eng.last_n_frames == t
        outs[t] = out.clone()
    eng.synchronize()
    for t in range(ticks):
        assert torch.equal(outs[t], ref[t]), (case, t, float((outs[t] - ref[t]).abs().max()))
    # a chunk over every frame written so far waits for the newest write
    last = eng.denoise(WL.make_state(cfg, ticks), WL.make_noise(cfg, ticks), n_frames=ticks)
    eng.synchronize()
    assert torch.equal(last, ref[ticks])
    eng.close()


def test_pipeline_newest_completed_window():
    cfg = SPARE_CASES["tiny_fp32"]
    ticks = 6
    w, sk, sv, frames = _setup(cfg, ticks)
    seq = R.ReflexEngine(cfg, w, sk, sv)
    ref = {}
    for n in range(ticks + 1):
        if n > 0:
            seq.write_frame(frames[n - 1])
        ref[n] = seq.denoise(WL.make_state(cfg, 0), WL.make_noise(cfg, 0)).clone()
    seq.synchronize()
    seq.close()
    eng = R.ReflexEngine(cfg, w, sk, sv)
    state, noise = WL.make_state(cfg, 0), WL.make_noise(cfg, 0)
    for t in range(ticks):
        eng.pipeline_write(frames[t])
        out = eng.denoise(state, noise, n_frames=-1).clone()
        n = eng.last_n_frames
        assert n in (t, t + 1), (t, n)
        eng.synchronize()
        assert torch.equal(out, ref[n]), (t, n)
    # once every write has completed, the newest frame is taken
    eng.synchronize()
    eng.denoise(state, noise, n_frames=-1)
    assert eng.last_n_frames == ticks
    eng.close()


def test_pipeline_rejects_misuse():
    cfg = WL.CONFIGS["tiny_fp32"]
    w, sk, sv, frames = _setup(cfg, 3)
    plain = R.ReflexEngine(cfg, w, sk, sv)
    with pytest.raises(R.ReflexError) as ei:
        plain.pipeline_write(frames[0])
    assert ei.value.status == R.REFLEX_EINVAL
    with pytest.raises(R.ReflexError) as ei:
        plain.denoise(WL.make_state(cfg, 0), WL.make_noise(cfg, 0), n_frames=0)
    assert ei.value.status == R.REFLEX_EINVAL
    plain.close()

    eng = R.ReflexEngine(cfg.replace(spare_slot=1), w, sk, sv)
    for t in range(3):
        eng.pipeline_write(frames[t])
    state, noise = WL.make_state(cfg, 0), WL.make_noise(cfg, 0)
    for bad in (0, 1, 4, -2):  # only 2 or 3 frames (or -1) are legal after 3 writes
        with pytest.raises(R.ReflexError) as ei:
            eng.denoise(state, noise, n_frames=bad)
        assert ei.value.status == R.REFLEX_EINVAL, bad
    with pytest.raises(R.ReflexError) as ei:
        eng.denoise(state, noise, mode="standard")
    assert ei.value.status == R.REFLEX_EINVAL
    # the naive strategy and the plain call still work on a spare-slot context
    eng.denoise(state, noise, mode="naive")
    eng.denoise(state, noise)
    eng.synchronize()
    eng.close()


def test_overlap_scheduler_with_engine():
    """Algorithm 1 in real time around the engine (tiny workload, 20 ms
    control period, a frame every period through the pipelined writer): the
    chunks come back with the engine's actions, the overlapped schedules never
    stall, and the synchronous one stalls once per chunk."""
    from paper_2607_14695_amd import overlap as OV

    cfg = SPARE_CASES["tiny_fp32"]
    w, sk, sv, frames = _setup(cfg, 4)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    noise = torch.from_numpy(WL.make_noise(cfg, 0)).cuda()
    chunk = cfg.action_horizon
    for strategy in ("reflex", "async_naive", "sync"):
        pol = OV.EnginePolicy(eng, [frames[t] for t in range(4)], lambda i: noise)
        sch = OV.OverlapScheduler(pol, chunk, 0.02, strategy=strategy, frame_period_s=0.02)
        st = sch.run(OV.FirstOrderRobot(np.zeros(cfg.state_dim)), 3 * chunk)
        s = st.summary()
        print(strategy, s, flush=True)
        assert st.chunks >= 2
        assert s["inference_ms_mean"] < 20.0
        if strategy == "sync":
            assert st.stalls >= st.chunks
        else:
            assert st.stalls == 0 and set(st.k_used) == {1}
    eng.synchronize()
    eng.close()
