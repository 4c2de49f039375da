"""Non-finite detection and FIFO recovery, the device tau schedule, and the
bf16 attention kernels against the oracle on an empty ring and with no cached
rows at all.

A NaN written into frame f reaches every chunk whose window holds frame f:
the chunks after frames f .. f+W-1 are non-finite, and the chunk after frame
f+W, whose write evicted frame f from the FIFO ring (Section 3.1), is finite
again and matches the oracle.  reflex_check_status reports the non-finite
chunks (the NaN/Inf events counted by the stability comparison of
Section 4.6).
"""
import numpy as np
import pytest
import torch

from oracle import reflex_oracle as O
from paper_2607_14695_amd import reflex as R
from paper_2607_14695_amd import workloads as WL

pytestmark = pytest.mark.gpu

BF16_REL, BF16_ABS = 1e-2, 5e-2

RAGGED = WL.CONFIGS["tiny_fp32"].replace(
    name="status", batch=2, static_len=40, frame_tokens=24, window_frames=3, action_horizon=5, n_q_heads=3,
    head_dim=128, width=128, mlp_dim=192, cond_hidden=64, state_dim=8, action_dim=5, frame_dim=72, n_layers=2,
    num_steps=3)


def _setup(cfg, ticks):
    w = WL.make_weights(cfg)
    sk, sv = WL.make_static_kv(cfg)
    frames = {t: WL.make_frame(cfg, t) for t in range(ticks)}
    return w, sk, sv, frames


def _bf16_close(got, ref, tag):
    rel = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    mx = float(np.max(np.abs(got - ref)))
    print(f"{tag}: rel-L2 {rel:.2e} max-abs {mx:.2e}", flush=True)
    assert rel <= BF16_REL and mx <= BF16_ABS, (tag, rel, mx)


@pytest.mark.parametrize("dtype,frame_dim", [("bf16", 72), ("bf16", 0), ("f32", 72)])
def test_nan_frame_poisons_its_window_then_is_evicted(dtype, frame_dim):
    cfg = RAGGED.replace(name=f"nan_{dtype}_{frame_dim}", dtype=dtype, frame_dim=frame_dim)
    W = cfg.window_frames
    f_bad = 2
    ticks = f_bad + W + 2
    w, sk, sv, frames = _setup(cfg, ticks)
    bad = frames[f_bad].copy()
    if frame_dim > 0:
        bad[1, 5, 7] = np.nan  # env 1, token 5 of the embedding
    else:
        bad[1, 0, 1, 5, 7] = np.nan  # env 1, layer 0, a value row
    frames[f_bad] = bad
    eng = R.ReflexEngine(cfg, w, sk, sv)
    assert eng.check_status() == R.REFLEX_OK
    for t in range(ticks):
        eng.write_frame(frames[t])
        state, noise = WL.make_state(cfg, t), WL.make_noise(cfg, t)
        got = eng.denoise(state, noise).cpu().numpy()
        st = eng.check_status()
        poisoned = f_bad <= t <= f_bad + W - 1
        print(f"{cfg.name} tick {t}: env1 finite {np.isfinite(got[1]).all()} status {st}", flush=True)
        # env 0 never sees the NaN: envs have their own rings
        assert np.isfinite(got[0]).all(), t
        if poisoned:
            assert not np.isfinite(got[1]).all(), t
            assert st == R.REFLEX_ENONFINITE, (t, st)
        else:
            assert np.isfinite(got[1]).all(), t
            assert st == R.REFLEX_OK, (t, st)
            if t > f_bad:
                ref = O.denoise_chunk(cfg, w, sk, sv, frames, t + 1, state, noise, cfg.taus())
                if dtype == "f32":
                    assert float(np.max(np.abs(got - ref))) <= 1e-4, t
                else:
                    _bf16_close(got, ref, f"{cfg.name} tick {t} after eviction")
    eng.close()


def test_device_tau_schedule_equals_host_schedule():
    cfg = RAGGED.replace(name="device_taus", dtype="bf16", num_steps=4)
    w, sk, sv, frames = _setup(cfg, 2)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    for t in range(2):
        eng.write_frame(frames[t])
    state, noise = WL.make_state(cfg, 1), WL.make_noise(cfg, 1)
    taus = np.array([1.0, 0.8, 0.45, 0.1, 0.0], dtype=np.float32)
    host = eng.denoise(state, noise, taus=taus).clone()
    dev_taus = torch.from_numpy(taus).cuda()
    dev = eng.denoise(state, noise, taus=dev_taus).clone()
    eng.synchronize()
    assert torch.equal(host, dev)
    ref = O.denoise_chunk(cfg, w, sk, sv, frames, 2, state, noise, taus)
    _bf16_close(dev.cpu().numpy(), ref, "device tau schedule")
    eng.close()


@pytest.mark.parametrize("attn", ["rows16", "rows16p", "pair"])
@pytest.mark.parametrize("static_len", [40, 0])
def test_bf16_empty_ring_against_oracle(attn, static_len):
    """No frame written: the cached rows are the static prefix alone, or none
    at all (no prefix either), for each bf16 attention kernel."""
    cfg = RAGGED.replace(name=f"empty_{attn}_{static_len}", dtype="bf16", static_len=static_len,
                         attn_kernel=attn)
    w, sk, sv, frames = _setup(cfg, 1)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    state, noise = WL.make_state(cfg, 0), WL.make_noise(cfg, 0)
    got = eng.denoise(state, noise).cpu().numpy()
    eng.synchronize()
    ref = O.denoise_chunk(cfg, w, sk, sv, frames, 0, state, noise, cfg.taus())
    _bf16_close(got, ref, f"empty ring, static_len {static_len}, {attn}")
    # one frame later the same engine matches again
    eng.write_frame(frames[0])
    got = eng.denoise(state, noise).cpu().numpy()
    eng.synchronize()
    ref = O.denoise_chunk(cfg, w, sk, sv, frames, 1, state, noise, cfg.taus())
    _bf16_close(got, ref, f"one frame, static_len {static_len}, {attn}")
    eng.close()
