"""GPU parity of the two comparison strategies of Section 4 (Baselines, and
the partitioned-attention ablation of Section 4.6), called through the C ABI
entry point reflex_denoise_chunk_baseline.

* Standard (full history recomputation at every step) re-encodes the static
  prefix and every window frame before each Euler step.  The re-encoded rows
  are the same bytes, so the actions must equal the method's bit for bit, and
  the cache and the device tick state must come out unchanged.
* Naive Cache (the dynamic K/V of the first step reused at every later step)
  must match the oracle's naive evaluator to the usual tolerance, and differ
  from the method by far more than that tolerance."""
import ctypes

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

STANDARD_CASES = {
    "tiny_fp32": WL.CONFIGS["tiny_fp32"],
    "ragged_bf16_dh128_direct": RAGGED.replace(name="rb128", dtype="bf16", head_dim=128, frame_dim=0),
    "ragged_bf16_dh256_embed": RAGGED.replace(name="rb256", dtype="bf16", head_dim=256, frame_dim=48),
    "no_static_fp32": RAGGED.replace(name="ns", static_len=0, frame_dim=0, window_frames=2),
}


def _setup(cfg, ticks):
    w = WL.make_weights(cfg)
    sk, sv = WL.make_static_kv(cfg)
    frames = {t: WL.make_frame(cfg, t) for t in range(ticks)}
    return w, sk, sv, frames


@pytest.mark.parametrize("case", sorted(STANDARD_CASES))
def test_standard_equals_reflex_bitwise(case):
    cfg = STANDARD_CASES[case]
    w, sk, sv, frames = _setup(cfg, 7)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    for t in [-1] + list(range(7)):
        if t >= 0:
            eng.write_frame(frames[t])
        if t not in (-1, 0, 2, 6):
            continue
        print(f"standard {case} after {t + 1} frames", flush=True)
        state, noise = WL.make_state(cfg, t + 1), WL.make_noise(cfg, t + 1)
        eng.synchronize()
        cache0 = eng.cache.clone()
        tick0 = eng.tick_state()
        a = eng.denoise(state, noise).clone()
        b = eng.denoise(state, noise, mode="standard").clone()
        eng.synchronize()
        assert torch.equal(a, b), (case, t, float((a - b).abs().max()))
        assert torch.equal(cache0, eng.cache), (case, t)
        assert eng.tick_state() == tick0
        assert eng.frames_written() == t + 1
        # replaying the captured Standard graph gives the same result again
        c = eng.denoise(state, noise, mode="standard").clone()
        eng.synchronize()
        assert torch.equal(a, c)
    eng.close()


def _strong_attention(w):
    """Attention projections and the action head scaled by 8 (exact in bf16),
    so that stale dynamic K/V move the actions by order one."""
    w2 = dict(w)
    for name in ("w_qkv", "w_o", "w_aout"):
        w2[name] = w[name] * 8.0
    return w2


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_naive_matches_oracle_and_differs_from_reflex(dtype):
    cfg = RAGGED.replace(name=f"naive_{dtype}", dtype=dtype, head_dim=64 if dtype == "f32" else 256)
    w, sk, sv, frames = _setup(cfg, 4)
    w = _strong_attention(w)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    caches = [O.PartitionedCache(cfg, w, sk, sv, env=b) for b in range(cfg.batch)]
    for t in range(4):
        eng.write_frame(frames[t])
        for b in range(cfg.batch):
            caches[b].write(frames[t][b])
    state, noise = WL.make_state(cfg, 4), WL.make_noise(cfg, 4)
    naive = eng.denoise(state, noise, mode="naive").cpu().numpy()
    good = eng.denoise(state, noise).cpu().numpy()
    eng.synchronize()
    ref = np.stack([O.denoise_chunk_partitioned(cfg, w, caches[b], state[b], noise[b], cfg.taus(), naive_cache=True)
                    for b in range(cfg.batch)])
    err = float(np.max(np.abs(naive - ref)))
    rel = float(np.linalg.norm(naive - ref) / np.linalg.norm(ref))
    gap = float(np.max(np.abs(naive - good)))
    print(f"naive {dtype}: vs oracle max-abs {err:.2e} rel-L2 {rel:.2e}; vs method {gap:.3f}", flush=True)
    if dtype == "f32":
        assert err <= FP32_TOL
        assert gap > 1000 * FP32_TOL
    else:
        assert rel <= BF16_REL and err <= BF16_ABS
        assert gap > 2 * BF16_ABS
    eng.close()


def test_naive_single_step_equals_reflex():
    """With one Euler step there is no later step to reuse stale K/V, so the
    naive strategy reduces to the method exactly."""
    cfg = WL.CONFIGS["tiny_fp32"]
    w, sk, sv, frames = _setup(cfg, 2)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    eng.write_frame(frames[0])
    eng.write_frame(frames[1])
    state, noise = WL.make_state(cfg, 0), WL.make_noise(cfg, 0)
    a = eng.denoise(state, noise, num_steps=1).clone()
    b = eng.denoise(state, noise, num_steps=1, mode="naive").clone()
    eng.synchronize()
    assert torch.equal(a, b)
    eng.close()


def test_baseline_rejects_bad_arguments():
    cfg = WL.CONFIGS["tiny_fp32"]
    w, sk, sv, frames = _setup(cfg, 1)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    eng.write_frame(frames[0])
    s = torch.from_numpy(WL.make_state(cfg, 0)).cuda()
    n = torch.from_numpy(WL.make_noise(cfg, 0)).cuda()
    out = torch.empty_like(n)
    lib = eng.lib
    # unknown mode
    st = lib.reflex_denoise_chunk_baseline(eng.ctx, 7, None, s.data_ptr(), n.data_ptr(), cfg.num_steps, None,
                                           out.data_ptr())
    assert st == R.REFLEX_EINVAL
    # Standard without sources, and with a window of the wrong length
    st = lib.reflex_denoise_chunk_baseline(eng.ctx, R.MODE_STANDARD, None, s.data_ptr(), n.data_ptr(),
                                           cfg.num_steps, None, out.data_ptr())
    assert st == R.REFLEX_EINVAL
    sk_d, sv_d = eng._static
    src = R.SourcesC(static_k=sk_d.data_ptr(), static_v=sv_d.data_ptr(), frames=None, n_frames=0)
    st = lib.reflex_denoise_chunk_baseline(eng.ctx, R.MODE_STANDARD, src, s.data_ptr(), n.data_ptr(),
                                           cfg.num_steps, None, out.data_ptr())
    assert st == R.REFLEX_EINVAL
    # a NULL frame pointer in the window
    arr = (R.c_vp * 1)(None)
    src = R.SourcesC(static_k=sk_d.data_ptr(), static_v=sv_d.data_ptr(),
                     frames=ctypes.cast(arr, ctypes.POINTER(R.c_vp)), n_frames=1)
    st = lib.reflex_denoise_chunk_baseline(eng.ctx, R.MODE_STANDARD, src, s.data_ptr(), n.data_ptr(),
                                           cfg.num_steps, None, out.data_ptr())
    assert st == R.REFLEX_EINVAL
    eng.close()


@pytest.mark.parametrize("case", ["tiny_fp32", "ragged_bf16_dh256_embed", "ragged_bf16_dh128_direct"])
def test_unfused_schedule_matches_oracle(case):
    """The fusion ablation's unfused schedule computes the same chunk: within
    the parity bar of the oracle, and close to the fused result."""
    cfg = STANDARD_CASES[case]
    w, sk, sv, frames = _setup(cfg, 3)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    for t in range(3):
        eng.write_frame(frames[t])
    state, noise = WL.make_state(cfg, 3), WL.make_noise(cfg, 3)
    fused = eng.denoise(state, noise).cpu().numpy()
    unfused = eng.denoise(state, noise, mode="unfused").cpu().numpy()
    again = eng.denoise(state, noise, mode="unfused").cpu().numpy()  # graph replay
    eng.close()
    ref = O.denoise_chunk(cfg, w, sk, sv, frames, 3, state, noise, cfg.taus())
    assert np.array_equal(unfused, again)
    if cfg.bf16:
        rel = float(np.linalg.norm(unfused - ref) / np.linalg.norm(ref))
        assert rel <= BF16_REL and float(np.max(np.abs(unfused - ref))) <= BF16_ABS, rel
    else:
        assert float(np.max(np.abs(unfused - ref))) <= FP32_TOL
        assert float(np.max(np.abs(unfused - fused))) <= 1e-5
