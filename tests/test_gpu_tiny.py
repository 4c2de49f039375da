"""GPU parity of the HIP path against the float64 oracle on small shapes the
oracle finishes in seconds: the tiny fp32 workload (max-abs 1e-4 on the action
chunk) and ragged variants that leave partial key tiles, partial query blocks,
several envs and an empty ring.  Integer bookkeeping is compared bit-exactly."""
import numpy as np
import pytest
import torch

from oracle import reflex_oracle as O
from paper_2607_14695_amd import reflex as R
from paper_2607_14695_amd import workloads as WL

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-4


def _setup(cfg, ticks):
    w = WL.make_weights(cfg)
    sk, sv = WL.make_static_kv(cfg)
    frames = {t: WL.make_frame(cfg, t) for t in range(ticks)}
    return w, sk, sv, frames


@pytest.fixture(scope="module")
def tiny():
    cfg = WL.CONFIGS["tiny_fp32"]
    return (cfg,) + _setup(cfg, cfg.ticks)


RAGGED = WL.CONFIGS["tiny_fp32"].replace(
    name="ragged_fp32", batch=3, static_len=40, frame_tokens=24, window_frames=3, action_horizon=5,
    n_q_heads=3, head_dim=128, width=128, mlp_dim=192, cond_hidden=64, state_dim=8, action_dim=5,
    frame_dim=72, n_layers=2, num_steps=3)


def test_tiny_static_prefix_and_tick_state(tiny):
    cfg, w, sk, sv, frames = tiny
    eng = R.ReflexEngine(cfg, w, sk, sv)
    assert eng.tick_state() == (0, 0, cfg.static_len)
    K, Vt = eng.cache_views()
    K, Vt = K.cpu().numpy(), Vt.cpu().numpy()
    for l in range(cfg.n_layers):
        ks, vs = O.static_kv(cfg, sk, sv, l, 0)
        np.testing.assert_allclose(K[0, l, :cfg.static_len], ks[:, 0], rtol=1e-5, atol=1e-5)
        np.testing.assert_allclose(Vt[0, l, :, :cfg.static_len], vs[:, 0].T, rtol=0, atol=0)
    eng.close()


def test_tiny_ring_writes_match_oracle_and_trace(tiny):
    cfg, w, sk, sv, frames = tiny
    eng = R.ReflexEngine(cfg, w, sk, sv)
    for t in range(cfg.ticks):
        f, ev = eng.write_frame(frames[t])
        st = O.ring_step(t, cfg.window_frames, cfg.frame_tokens, cfg.static_len)
        assert (f, ev) == (st.frame_index, st.evicted)
        assert eng.tick_state() == (t + 1, st.n_valid, st.dyn_pos0)
        assert eng.frames_written() == t + 1
        K, Vt = eng.cache_views()
        K, Vt = K.cpu().numpy(), Vt.cpu().numpy()
        r0 = cfg.static_len + st.slot * cfg.frame_tokens
        for l in range(cfg.n_layers):
            kf, vf = O.frame_kv(cfg, w, frames[t][0], t, l)
            np.testing.assert_allclose(K[0, l, r0:r0 + cfg.frame_tokens], kf[:, 0], rtol=1e-4, atol=1e-4)
            np.testing.assert_allclose(Vt[0, l, :, r0:r0 + cfg.frame_tokens], vf[:, 0].T, rtol=1e-4, atol=1e-4)
    eng.close()


def test_tiny_denoise_every_tick(tiny):
    cfg, w, sk, sv, frames = tiny
    eng = R.ReflexEngine(cfg, w, sk, sv)
    for t in range(cfg.ticks):
        eng.write_frame(frames[t])
        state, noise = WL.make_state(cfg, t), WL.make_noise(cfg, t)
        got = eng.denoise(state, noise)
        eng.synchronize()
        ref = O.denoise_chunk(cfg, w, sk, sv, frames, t + 1, state, noise, cfg.taus())
        err = np.max(np.abs(got.cpu().numpy() - ref))
        assert err <= FP32_TOL, (t, err)
    eng.close()


def test_tiny_empty_ring(tiny):
    cfg, w, sk, sv, frames = tiny
    eng = R.ReflexEngine(cfg, w, sk, sv)
    state, noise = WL.make_state(cfg, 0), WL.make_noise(cfg, 0)
    got = eng.denoise(state, noise)
    eng.synchronize()
    ref = O.denoise_chunk(cfg, w, sk, sv, frames, 0, state, noise, cfg.taus())
    assert np.max(np.abs(got.cpu().numpy() - ref)) <= FP32_TOL
    eng.close()


def test_tiny_cache_bytes_unchanged_by_denoise(tiny):
    """Timestep invariance (Section 3.1): the denoise only reads the cache."""
    cfg, w, sk, sv, frames = tiny
    eng = R.ReflexEngine(cfg, w, sk, sv)
    for t in range(3):
        eng.write_frame(frames[t])
    eng.synchronize()
    before = eng.cache.clone()
    for k in range(3):
        eng.denoise(WL.make_state(cfg, k), WL.make_noise(cfg, k))
        eng.synchronize()
        assert torch.equal(before, eng.cache)
    eng.close()


def test_tiny_per_step_velocity(tiny):
    """Each Euler step on its own: v_k = (x_{k+1} - x_k) / dt from a 1-step call
    started at the oracle's x_k (a check that x_K alone could hide)."""
    cfg, w, sk, sv, frames = tiny
    eng = R.ReflexEngine(cfg, w, sk, sv)
    for t in range(2):
        eng.write_frame(frames[t])
    state, noise = WL.make_state(cfg, 1), WL.make_noise(cfg, 1)
    taus = cfg.taus()
    diag = {}
    O.denoise_chunk(cfg, w, sk, sv, frames, 2, state, noise, taus, diag=diag)
    x = noise[0].astype(np.float64)
    for k in range(cfg.num_steps):
        xk32 = x.astype(np.float32)
        got = eng.denoise(state, xk32[None], num_steps=1, taus=[taus[k], taus[k + 1]])
        eng.synchronize()
        dt = float(taus[k + 1]) - float(taus[k])
        v_gpu = (got.cpu().numpy()[0].astype(np.float64) - xk32) / dt
        v_ref = diag["v"][0][k]
        assert np.max(np.abs(v_gpu - v_ref)) <= 1e-3, k
        x = x + dt * v_ref
    eng.close()


def test_tiny_graph_replay_is_deterministic(tiny):
    cfg, w, sk, sv, frames = tiny
    eng = R.ReflexEngine(cfg, w, sk, sv)
    eng.write_frame(frames[0])
    state = torch.from_numpy(WL.make_state(cfg, 0)).cuda()
    noise = torch.from_numpy(WL.make_noise(cfg, 0)).cuda()
    outs = []
    for _ in range(4):
        outs.append(eng.denoise(state, noise).clone())
        eng.synchronize()
        torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o, outs[0])
    eng.close()


def test_tiny_engine_stream_current(tiny):
    """Calls made with the engine's own stream current (ReflexEngine.current)
    return the same actions, bit for bit, as calls from the default stream, and
    the oracle's within the fp32 bound; frame writes inside the context reach
    the chunks outside it."""
    cfg, w, sk, sv, frames = tiny
    eng = R.ReflexEngine(cfg, w, sk, sv)
    default = torch.cuda.current_stream()
    eng.write_frame(frames[0])
    state, noise = WL.make_state(cfg, 1), WL.make_noise(cfg, 1)
    ref_gpu = eng.denoise(state, noise).cpu().numpy().copy()
    with eng.current():
        assert torch.cuda.current_stream() == eng.stream
        got = eng.denoise(state, noise).clone()
        eng.write_frame(frames[1])
        got2 = eng.denoise(state, noise).clone()
    assert torch.cuda.current_stream() == default
    eng.synchronize()
    assert np.array_equal(got.cpu().numpy(), ref_gpu)
    after = eng.denoise(state, noise).cpu().numpy()
    assert np.array_equal(after, got2.cpu().numpy())
    ref = O.denoise_chunk(cfg, w, sk, sv, frames, 2, state, noise, cfg.taus())
    assert np.max(np.abs(after - ref)) <= FP32_TOL
    eng.close()


def test_tiny_scale_only_and_custom_schedule():
    cfg = WL.CONFIGS["tiny_fp32"].replace(mod_mode="scale_only", num_steps=5,
                                          tau_schedule=(1.0, 0.97, 0.6, 0.3, 0.02, 0.0))
    w, sk, sv, frames = _setup(cfg, 3)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    for t in range(3):
        eng.write_frame(frames[t])
    state, noise = WL.make_state(cfg, 2), WL.make_noise(cfg, 2)
    got = eng.denoise(state, noise, taus=cfg.taus())
    eng.synchronize()
    ref = O.denoise_chunk(cfg, w, sk, sv, frames, 3, state, noise, cfg.taus())
    assert np.max(np.abs(got.cpu().numpy() - ref)) <= FP32_TOL
    eng.close()


@pytest.mark.parametrize("frame_dim", [72, 0])
def test_ragged_multi_env(frame_dim):
    """Partial key tiles (Ls = 40, F = 24), partial query blocks (T*Hq = 18),
    three independent envs, a 3-slot ring wrapped twice, both frame paths."""
    cfg = RAGGED.replace(frame_dim=frame_dim)
    w, sk, sv, frames = _setup(cfg, 7)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    for t in range(7):
        eng.write_frame(frames[t])
        if t in (0, 2, 6):
            state, noise = WL.make_state(cfg, t), WL.make_noise(cfg, t)
            got = eng.denoise(state, noise)
            eng.synchronize()
            ref = O.denoise_chunk(cfg, w, sk, sv, frames, t + 1, state, noise, cfg.taus())
            assert np.max(np.abs(got.cpu().numpy() - ref)) <= FP32_TOL, t
    eng.close()


BF16_REL, BF16_ABS = 1e-2, 5e-2


@pytest.mark.parametrize("attn", ["rows16", "rows16p", "pair"])
@pytest.mark.parametrize("head_dim,frame_dim", [(64, 72), (128, 0), (256, 48)])
def test_ragged_bf16(head_dim, frame_dim, attn):
    """The bf16 path (bf16 attention tiles, bf16 GEMM operands) at every head
    width it supports, with both attention kernels, ragged tiles and blocks:
    Ls = 40 and F = 24 leave partial 64-key tiles, T*Hq = 18 a partial query
    block; three envs; a 3-slot ring wrapped twice.  Tolerance: relative-L2
    1e-2 and max-abs 5e-2 on the action chunk (bf16 operands, fp32
    accumulation)."""
    cfg = RAGGED.replace(name=f"ragged_bf16_{head_dim}", dtype="bf16", head_dim=head_dim, frame_dim=frame_dim,
                         attn_kernel=attn)
    w, sk, sv, frames = _setup(cfg, 7)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    for t in range(7):
        eng.write_frame(frames[t])
        if t in (0, 2, 6):
            state, noise = WL.make_state(cfg, t), WL.make_noise(cfg, t)
            got = eng.denoise(state, noise).cpu().numpy()
            eng.synchronize()
            ref = O.denoise_chunk(cfg, w, sk, sv, frames, t + 1, state, noise, cfg.taus())
            rel = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
            mx = float(np.max(np.abs(got - ref)))
            print(f"bf16 dh={head_dim} {attn} tick {t}: rel-L2 {rel:.2e} max-abs {mx:.2e}", flush=True)
            assert rel <= BF16_REL and mx <= BF16_ABS, (t, rel, mx)
    eng.close()


@pytest.mark.parametrize("head_dim,heads,horizon", [(64, 2, 7), (256, 2, 7), (64, 8, 50)])
def test_multi_tile_splits_pipelined_equals_rows16(head_dim, heads, horizon):
    """Key splits of several tiles each: two envs and a 20-frame ring of
    200-token frames give 21 to 65 key tiles over 16 splits, so a split runs
    2, 3, 4 or 5 tiles (odd and even counts, the pipelined kernel's loop and
    its tail).  Frame keys are scaled by 1, 2 and 4 for frames 0-6, 7-13 and
    14-19 (exact in bf16), so tile maxima grow by more than the lazy-rescale
    threshold inside a split.  16 query rows per env fill one wave of one
    block; 408 rows (51 tokens x 8 heads) spread 26 row waves over four blocks
    as 7, 7, 6 and 6.  The pipelined 16-row kernel must equal the plain one
    bit for bit (same rows per wave, same operations in the same order per
    row), and both must match the oracle within the bf16 tolerance."""
    cfg = RAGGED.replace(name=f"multi_tile_{head_dim}_{heads}x{horizon}", dtype="bf16", batch=2, static_len=40,
                         frame_tokens=200, window_frames=20, action_horizon=horizon, n_q_heads=heads,
                         head_dim=head_dim, frame_dim=0, num_steps=2)
    w, sk, sv, frames = _setup(cfg, 20)
    for f in frames:
        frames[f][:, :, 0] *= float(2 ** (f // 7))
    engs = {a: R.ReflexEngine(cfg.replace(attn_kernel=a), w, sk, sv) for a in ("rows16", "rows16p")}
    for t in range(20):
        for e in engs.values():
            e.write_frame(frames[t])
        if t + 1 in (6, 11, 16, 20):
            state, noise = WL.make_state(cfg, t), WL.make_noise(cfg, t)
            got = {a: e.denoise(state, noise).cpu().numpy().copy() for a, e in engs.items()}
            assert np.array_equal(got["rows16"], got["rows16p"]), t
            ref = O.denoise_chunk(cfg, w, sk, sv, frames, t + 1, state, noise, cfg.taus())
            rel = float(np.linalg.norm(got["rows16p"] - ref) / np.linalg.norm(ref))
            mx = float(np.max(np.abs(got["rows16p"] - ref)))
            print(f"multi-tile dh={head_dim} rows {heads * (horizon + 1)} frames {t + 1}: rel-L2 {rel:.2e} "
                  f"max-abs {mx:.2e}", flush=True)
            assert rel <= BF16_REL and mx <= BF16_ABS, (t, rel, mx)
    for e in engs.values():
        e.close()


@pytest.mark.parametrize("batch,width", [(1, 512), (8, 512), (8, 2048)])
def test_gemm_row_tilings_bf16(batch, width):
    """51 dynamic rows per env with 128-wide heads.  Eight envs (M = 408 GEMM
    rows): the packed QKV (RoPE epilogue), gate|up (gated GELU) and down (fp32
    output) GEMMs take the tiled path with 64-row tiles on the four-stage
    pipeline, 8 stages of 64 over K = 512 at width 512 and 32 stages at width
    2048 (QKV and gate|up with two waves per output block).  One env (M = 51):
    the unsplit skinny GEMMs with few column strips (QKV, gate|up) take their
    rows in two 32-row halves, and the split merge its 4-byte form.  Every env
    is checked against the oracle within the bf16 tolerance."""
    cfg = RAGGED.replace(name=f"rowtile_bf16_b{batch}_w{width}", dtype="bf16", batch=batch, action_horizon=50, width=width,
                         mlp_dim=512, n_q_heads=2, head_dim=128, frame_dim=0, n_layers=1, num_steps=2,
                         window_frames=2)
    w, sk, sv, frames = _setup(cfg, 2)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    for t in range(2):
        eng.write_frame(frames[t])
    state, noise = WL.make_state(cfg, 1), WL.make_noise(cfg, 1)
    got = eng.denoise(state, noise).cpu().numpy()
    eng.synchronize()
    ref = O.denoise_chunk(cfg, w, sk, sv, frames, 2, state, noise, cfg.taus())
    rel = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    mx = float(np.max(np.abs(got - ref)))
    print(f"row tilings B={batch} width {width}: rel-L2 {rel:.2e} max-abs {mx:.2e}", flush=True)
    assert rel <= BF16_REL and mx <= BF16_ABS, (rel, mx)
    eng.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_limits_t64_no_static_prefix(dtype):
    """Boundary shapes: 63 actions (T = 64, a full dynamic tile and T*Hq = 192
    query rows), no static prefix (the cached keys are ring rows only),
    state and action widths of 64, a 5-slot ring of 8-token frames."""
    cfg = RAGGED.replace(name=f"limits_{dtype}", dtype=dtype, batch=2, static_len=0, frame_tokens=8,
                         window_frames=5, action_horizon=63, action_dim=64, state_dim=64, n_q_heads=3,
                         head_dim=64, width=128, mlp_dim=128, cond_hidden=64, frame_dim=0, num_steps=2)
    w, sk, sv, frames = _setup(cfg, 7)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    for t in range(7):
        eng.write_frame(frames[t])
        if t in (0, 6):
            state, noise = WL.make_state(cfg, t), WL.make_noise(cfg, t)
            got = eng.denoise(state, noise).cpu().numpy()
            eng.synchronize()
            ref = O.denoise_chunk(cfg, w, sk, sv, frames, t + 1, state, noise, cfg.taus())
            if dtype == "f32":
                assert np.max(np.abs(got - ref)) <= FP32_TOL, t
            else:
                rel = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
                assert rel <= BF16_REL and float(np.max(np.abs(got - ref))) <= BF16_ABS, (t, rel)
    eng.close()


@pytest.mark.parametrize("dtype,horizon,attn", [("f32", 100, "auto"), ("bf16", 100, "rows16"),
                                                ("bf16", 127, "rows16"), ("bf16", 100, "pair"),
                                                ("bf16", 127, "pair"), ("bf16", 100, "rows16p"),
                                                ("bf16", 127, "rows16p")])
def test_long_chunks_two_dynamic_tiles(dtype, horizon, attn):
    """Action chunks longer than one 64-key tile: T = 101 (a ragged second
    dynamic tile) and T = 128 (the largest supported), so the dynamic keys
    span two tiles and the query rows several query blocks."""
    cfg = RAGGED.replace(name=f"long_{dtype}_{horizon}", dtype=dtype, batch=2, action_horizon=horizon,
                         n_q_heads=2, head_dim=64, width=128, mlp_dim=128, cond_hidden=64, frame_dim=0,
                         window_frames=2, num_steps=2, attn_kernel=attn)
    w, sk, sv, frames = _setup(cfg, 3)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    for t in range(3):
        eng.write_frame(frames[t])
    state, noise = WL.make_state(cfg, 2), WL.make_noise(cfg, 2)
    got = eng.denoise(state, noise).cpu().numpy()
    eng.synchronize()
    ref = O.denoise_chunk(cfg, w, sk, sv, frames, 3, state, noise, cfg.taus())
    if dtype == "f32":
        assert np.max(np.abs(got - ref)) <= FP32_TOL
    else:
        rel = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
        assert rel <= BF16_REL and float(np.max(np.abs(got - ref))) <= BF16_ABS, rel
    eng.close()


def test_norm_precision_variants():
    """The two baselines of the stability stress test (a bf16 residual stream
    with bf16 or fp32 RMS statistics) stay finite and close to the oracle on a
    short chunk, differ from the method, and the method is unchanged by the
    option's existence (checked by every other test)."""
    cfg = RAGGED.replace(name="normprec", dtype="bf16", head_dim=128, frame_dim=0)
    w, sk, sv, frames = _setup(cfg, 3)
    state, noise = WL.make_state(cfg, 2), WL.make_noise(cfg, 2)
    ref = O.denoise_chunk(cfg, w, sk, sv, frames, 3, state, noise, cfg.taus())
    got = {}
    for prec in ("fp32", "bf16_fp32_stats", "bf16"):
        eng = R.ReflexEngine(cfg.replace(norm_precision=prec), w, sk, sv)
        for t in range(3):
            eng.write_frame(frames[t])
        got[prec] = eng.denoise(state, noise).cpu().numpy()
        eng.close()
        rel = float(np.linalg.norm(got[prec] - ref) / np.linalg.norm(ref))
        print(prec, f"rel-L2 vs oracle {rel:.2e}", flush=True)
        assert np.isfinite(got[prec]).all()
        assert rel <= (BF16_REL if prec == "fp32" else 5e-2), (prec, rel)
    for prec in ("bf16_fp32_stats", "bf16"):
        assert np.max(np.abs(got[prec] - got["fp32"])) > 0.0, prec


def test_dtype_probe_rejects_mismatch(tiny):
    cfg, w, sk, sv, frames = tiny
    with pytest.raises(R.ReflexError) as ei:
        R.ReflexEngine(cfg, w, sk, sv, weight_dtype_override=torch.bfloat16)
    assert ei.value.status == R.REFLEX_EDTYPE


def test_denoise_rejects_bad_steps(tiny):
    cfg, w, sk, sv, frames = tiny
    eng = R.ReflexEngine(cfg, w, sk, sv)
    with pytest.raises(R.ReflexError) as ei:
        eng.denoise(WL.make_state(cfg, 0), WL.make_noise(cfg, 0), num_steps=cfg.num_steps + 1)
    assert ei.value.status == R.REFLEX_EINVAL
    eng.close()


def test_engine_waits_for_inputs_made_on_the_callers_stream():
    """The static K/V handed to the engine may still be being computed on the
    caller's stream (here behind a ~50 ms busy kernel); the prefix written at
    init must still be the finished values."""
    cfg = WL.CONFIGS["tiny_fp32"]
    w, sk, sv, frames = _setup(cfg, 1)
    sk_ref = torch.from_numpy(sk).cuda()
    sv_ref = torch.from_numpy(sv).cuda()
    torch.cuda.synchronize()
    sk_d = torch.zeros_like(sk_ref)
    sv_d = torch.zeros_like(sv_ref)
    torch.cuda._sleep(100_000_000)  # keeps the caller's stream busy
    sk_d.copy_(sk_ref)
    sv_d.copy_(sv_ref)
    eng = R.ReflexEngine(cfg, w, sk_d, sv_d)
    K, Vt = eng.cache_views()
    K, Vt = K.cpu().numpy(), Vt.cpu().numpy()
    ks, vs = O.static_kv(cfg, sk, sv, 0, 0)
    np.testing.assert_allclose(K[0, 0, :cfg.static_len], ks[:, 0], rtol=1e-5, atol=1e-5)
    np.testing.assert_allclose(Vt[0, 0, :, :cfg.static_len], vs[:, 0].T, rtol=0, atol=0)
    eng.close()


@pytest.mark.parametrize("shape", ["qkv_gelu", "o_proj"])
def test_gemm_160_row_tiles_bf16(shape):
    """32 envs of 51 rows (M = 1632), so a GEMM with 20 column tiles has 260
    128-row tiles, just over one wave, and takes 220 160-row tiles on the
    four-stage pipeline with two waves per output block (K = 1024).
    "qkv_gelu": width 1024, eight 256-wide heads: the packed QKV (N = 2560,
    RoPE epilogue on head pairs) and gate|up (1280 gated-GELU pairs) take that
    path.  "o_proj": width 2560, four heads: the output projection (N = 2560,
    K = 1024, one split, fp32 epilogue) takes it.  Envs 0, 17 and 31 (the
    last, partial tile) against the oracle."""
    if shape == "qkv_gelu":
        width, heads, mlp = 1024, 8, 1280
    else:
        width, heads, mlp = 2560, 4, 512
    cfg = RAGGED.replace(name="tile160_" + shape, dtype="bf16", batch=32, action_horizon=50, width=width,
                         mlp_dim=mlp, n_q_heads=heads, head_dim=256, state_dim=8, action_dim=5, cond_hidden=64,
                         frame_dim=0, n_layers=1, num_steps=1, window_frames=1, static_len=40, frame_tokens=24)
    w, sk, sv, frames = _setup(cfg, 1)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    eng.write_frame(frames[0])
    envs = [0, 17, 31]
    state, noise = WL.make_state(cfg, 1), WL.make_noise(cfg, 1)
    got = eng.denoise(state, noise).cpu().numpy()[envs]
    eng.synchronize()
    ref = O.denoise_chunk(cfg, w, sk, sv, {0: frames[0]}, 1, state, noise, cfg.taus(), envs=envs)
    for i, e in enumerate(envs):
        rel = float(np.linalg.norm(got[i] - ref[i]) / np.linalg.norm(ref[i]))
        mx = float(np.max(np.abs(got[i] - ref[i])))
        print(f"160-row tiles ({shape}) env {e}: rel-L2 {rel:.2e} max-abs {mx:.2e}", flush=True)
        assert rel <= BF16_REL and mx <= BF16_ABS, (e, rel, mx)
    eng.close()


def test_gemm_32x32_blocks_bf16():
    """41 envs of 51 rows (M = 2091) at width 512 with six 128-wide heads: the
    packed QKV (N = 1024, RoPE epilogue) and gate|up (gated GELU) GEMMs have
    8 column tiles of 17 128-row tiles, one wave, but 264 64-row ones, so they
    take 128-row tiles on the four-stage pipeline with 32x32x16 MFMAs (8
    stages).  Envs 0, 20 and 40 (the last, partial tile) against the oracle."""
    cfg = RAGGED.replace(name="mfma32_bf16", dtype="bf16", batch=41, action_horizon=50, width=512,
                         mlp_dim=512, n_q_heads=6, head_dim=128, state_dim=8, action_dim=5, cond_hidden=64,
                         frame_dim=0, n_layers=1, num_steps=2, window_frames=1, static_len=40, frame_tokens=24)
    w, sk, sv, frames = _setup(cfg, 1)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    eng.write_frame(frames[0])
    envs = [0, 20, 40]
    state, noise = WL.make_state(cfg, 1), WL.make_noise(cfg, 1)
    got = eng.denoise(state, noise).cpu().numpy()[envs]
    eng.synchronize()
    ref = O.denoise_chunk(cfg, w, sk, sv, {0: frames[0]}, 1, state, noise, cfg.taus(), envs=envs)
    for i, e in enumerate(envs):
        rel = float(np.linalg.norm(got[i] - ref[i]) / np.linalg.norm(ref[i]))
        mx = float(np.max(np.abs(got[i] - ref[i])))
        print(f"32x32 blocks env {e}: rel-L2 {rel:.2e} max-abs {mx:.2e}", flush=True)
        assert rel <= BF16_REL and mx <= BF16_ABS, (e, rel, mx)
    eng.close()


@pytest.mark.parametrize("shape", ["rows320", "width1152"])
def test_embedding_kernel_every_step_fp32(shape):
    """Chunks outside the final kernel's fused-embedding range launch the
    embedding kernel at every Euler step: 5 envs x 64 tokens (320 rows) and
    one env at width 1152.  fp32 against the oracle."""
    if shape == "rows320":
        cfg = RAGGED.replace(name="embed_rows320", batch=5, action_horizon=63, num_steps=3)
    else:
        cfg = RAGGED.replace(name="embed_w1152", batch=1, width=1152, mlp_dim=256, num_steps=3)
    w, sk, sv, frames = _setup(cfg, 2)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    for t in range(2):
        eng.write_frame(frames[t])
    state, noise = WL.make_state(cfg, 1), WL.make_noise(cfg, 1)
    prof = eng.profile(state, noise)
    assert prof["embed_norm"][1] == cfg.num_steps
    got = eng.denoise(state, noise).cpu().numpy()
    eng.synchronize()
    ref = O.denoise_chunk(cfg, w, sk, sv, frames, 2, state, noise, cfg.taus())
    assert np.max(np.abs(got - ref)) <= FP32_TOL, np.max(np.abs(got - ref))
    eng.close()
