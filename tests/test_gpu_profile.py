"""In-graph class timing (reflex_profile_graph): the stamped launches of one
kernel class are exactly the launches the eager profile counts for it, each
gets a positive duration, and the classes' durations add up to at most the
chunk; the stamped graph computes the chunk bit for bit; the context's own
denoise is unchanged afterwards; malformed requests are rejected."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2607_14695_amd import reflex as R
from paper_2607_14695_amd import workloads as WL

pytestmark = pytest.mark.gpu


def _engine(cfg):
    w = WL.make_weights(cfg)
    sk, sv = WL.make_static_kv(cfg)
    eng = R.ReflexEngine(cfg, w, sk, sv)
    for t in range(cfg.window_frames):
        eng.write_frame(WL.make_frame(cfg, t))
    return eng, WL.make_state(cfg, 0), WL.make_noise(cfg, 0)


@pytest.mark.parametrize("dtype", [WL.DTYPE_F32, WL.DTYPE_BF16])
def test_class_graphs_count_the_profiled_launches(dtype):
    cfg = WL.CONFIGS["tiny_fp32"].replace(name=f"tiny_{dtype}", dtype=dtype)
    eng, state, noise = _engine(cfg)
    ref = eng.denoise(state, noise).clone()
    eager = eng.profile(state, noise)
    names = eng.class_names()
    assert set(eager) == set(names)
    for cls, (ms, n) in eager.items():
        if n == 0 or cls in ("frame_proj", "ring_write"):
            continue
        g_ms, g_n = eng.profile_graph(state, noise, [cls], reps=3)
        assert g_n == n, cls
        assert g_ms > 0.0, cls
    chunk = [c for c, (_, n) in eager.items() if n > 0]
    g_ms, g_n = eng.profile_graph(state, noise, chunk, reps=2)
    assert g_n == sum(n for _, n in eager.values())
    assert g_ms > 0.0
    # the stamped graph wrote the engine's output buffer: the whole chunk again
    torch.testing.assert_close(eng._keep_io[2], ref, rtol=0, atol=0)
    again = eng.denoise(state, noise)
    torch.testing.assert_close(again, ref, rtol=0, atol=0)
    eng.close()


def test_class_graph_rejects_bad_requests():
    cfg = WL.CONFIGS["tiny_fp32"]
    eng, state, noise = _engine(cfg)
    eng.denoise(state, noise)
    with pytest.raises(ValueError):
        eng.profile_graph(state, noise, ["no_such_class"])
    s, n, out = eng._keep_io
    ms, cnt = ctypes.c_double(0.0), ctypes.c_int32(0)
    call = eng.lib.reflex_profile_graph
    assert call(eng.ctx, s.data_ptr(), n.data_ptr(), cfg.num_steps, None, out.data_ptr(), 0, 3,
                ctypes.byref(ms), ctypes.byref(cnt)) == R.REFLEX_EINVAL
    assert call(eng.ctx, s.data_ptr(), n.data_ptr(), cfg.num_steps, None, out.data_ptr(), 1 << 2, 0,
                ctypes.byref(ms), ctypes.byref(cnt)) == R.REFLEX_EINVAL
    assert call(eng.ctx, s.data_ptr(), n.data_ptr(), 0, None, out.data_ptr(), 1 << 2, 3,
                ctypes.byref(ms), ctypes.byref(cnt)) == R.REFLEX_EINVAL
    assert call(eng.ctx, s.data_ptr(), n.data_ptr(), cfg.num_steps, None, out.data_ptr(), 1 << 2, 3,
                None, ctypes.byref(cnt)) == R.REFLEX_EINVAL
    eng.close()
