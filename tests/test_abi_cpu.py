"""Host-only checks of the C ABI: the library loads, exports every function the
header declares, and its pure host functions (ring bookkeeping, size query,
validation, status text) behave as documented.  No device calls."""
import ctypes
import os
import subprocess

import pytest

from paper_2607_14695_amd import reflex as R
from paper_2607_14695_amd import workloads as WL

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_library_exports_every_header_symbol():
    lib = R.load_library()
    names = R.header_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n


def test_ring_plan_matches_golden_trace():
    rows = []
    with open(os.path.join(GOLDEN, "ring_trace_w2_f32_ls64.txt")) as fh:
        for line in fh:
            if line.strip() and not line.startswith("#"):
                rows.append([int(t) for t in line.split()])
    for f, slot, p0, p1, nv, ev, dyn in rows:
        st = R.ring_plan(f, 2, 32, 64)
        assert st["frame_index"] == f and st["slot"] == slot and st["pos0"] == p0
        assert st["pos0"] + 31 == p1 and st["n_valid"] == nv and st["evicted"] == ev
        assert st["dyn_pos0"] == dyn


def test_ring_plan_long_streams_and_errors():
    # 500 ticks of 768-token frames in a 2-slot ring after a 48-token prefix
    st = R.ring_plan(499, 2, 768, 48)
    assert st["slot"] == 1 and st["pos0"] == 48 + 499 * 768 and st["evicted"] == 768
    assert st["dyn_pos0"] == 48 + 500 * 768 and st["n_valid"] == 2
    st = R.ring_plan(5, 8, 768, 256)
    assert st["slot"] == 5 and st["n_valid"] == 6 and st["evicted"] == 0
    # int64 positions far beyond 2^31
    st = R.ring_plan(3_000_000, 2, 768, 48)
    assert st["pos0"] == 48 + 3_000_000 * 768
    lib = R.load_library()
    out = R.RingStepC()
    assert lib.reflex_ring_plan(-1, 2, 32, 64, ctypes.byref(out)) == R.REFLEX_EINVAL
    assert lib.reflex_ring_plan(0, 0, 32, 64, ctypes.byref(out)) == R.REFLEX_EINVAL
    assert lib.reflex_ring_plan(0, 2, 32, 64, None) == R.REFLEX_EINVAL


@pytest.mark.parametrize("name", sorted(WL.CONFIGS))
def test_query_sizes_every_workload(name):
    cfg = WL.CONFIGS[name]
    cache, ws = R.query_sizes(cfg)
    esz = 2 if cfg.bf16 else 4
    per = cfg.batch * cfg.n_layers * cfg.cache_rows * cfg.head_dim * esz
    assert cache >= 2 * per and cache % 256 == 0
    assert ws > 0 and ws % 256 == 0


def test_query_sizes_rejects_bad_configs():
    base = R.config_to_c(WL.CONFIGS["tiny_fp32"])
    assert R.query_sizes_status(base) == R.REFLEX_OK
    for field, bad in [("n_kv_heads", 2), ("head_dim", 96), ("action_horizon", 128), ("width", 100),
                       ("dtype", 7), ("max_steps", 0), ("max_steps", 65), ("frame_tokens", 12),
                       ("static_len", -8), ("batch", 0), ("window_frames", 0), ("state_dim", 5),
                       ("spare_slot", 2), ("spare_slot", -1), ("norm_precision", 3), ("norm_precision", -1),
                       ("attn_kernel", 4), ("attn_kernel", -1)]:
        c = R.config_to_c(WL.CONFIGS["tiny_fp32"])
        setattr(c, field, bad)
        assert R.query_sizes_status(c) == R.REFLEX_EINVAL, field


def test_spare_slot_adds_one_frame_of_rows():
    """A ring with a spare slot holds window_frames + 1 frames per layer and env."""
    for name in ("tiny_fp32", "pi0_stream_bf16"):
        cfg = WL.CONFIGS[name]
        c0, w0 = R.query_sizes(cfg)
        c1, w1 = R.query_sizes(cfg.replace(spare_slot=1))
        esz = 2 if cfg.bf16 else 4
        extra = 2 * cfg.batch * cfg.n_layers * cfg.frame_tokens * cfg.head_dim * esz
        assert abs((c1 - c0) - extra) <= 512, name
        assert w1 >= w0  # the key split count may grow with the row count


def test_null_and_state_errors_without_device():
    lib = R.load_library()
    assert lib.reflex_cache_write_frame(None, None, None, None) == R.REFLEX_ESTATE
    assert lib.reflex_denoise_chunk(None, None, None, 10, None, None) == R.REFLEX_ESTATE
    assert lib.reflex_destroy(None) == 0
    assert lib.reflex_frames_written(None) < 0
    c = R.config_to_c(WL.CONFIGS["tiny_fp32"])
    out = ctypes.c_void_p(None)
    # null weights / buffers are rejected before any device call
    assert lib.reflex_cache_init(ctypes.byref(c), None, None, None, None, None, None, ctypes.byref(out)) \
        == R.REFLEX_EINVAL
    assert out.value is None


def test_strerror_texts():
    for code in (R.REFLEX_OK, R.REFLEX_EINVAL, R.REFLEX_EDTYPE, R.REFLEX_EHIP, R.REFLEX_ESTATE, -99):
        assert isinstance(R.strerror(code), str) and R.strerror(code)


def test_struct_sizes_match_c_layout(tmp_path):
    """Every ctypes mirror has the size and field offsets the C compiler gives
    the header's struct (a small host program built with gcc prints them)."""
    structs = {"reflex_config": R.ConfigC, "reflex_weights": R.WeightsC, "reflex_ring_step": R.RingStepC,
               "reflex_sources": R.SourcesC}
    lines = ['#include <stddef.h>', '#include <stdio.h>', f'#include "{R.HEADER_PATH}"', "int main(void) {"]
    for cname, py in structs.items():
        lines.append(f'  printf("{cname} size %zu\\n", sizeof({cname}));')
        for fname, _ in py._fields_:
            lines.append(f'  printf("{cname} {fname} %zu\\n", offsetof({cname}, {fname}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-o", str(exe), str(src)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l.strip()}
    for cname, py in structs.items():
        assert got[(cname, "size")] == ctypes.sizeof(py), cname
        for fname, _ in py._fields_:
            assert got[(cname, fname)] == getattr(py, fname).offset, (cname, fname)
