"""Host-side checks of the rocprofv3 summary tools (no GPU)."""
import json

from paper_2607_14695_amd import profiling as P


def _rec(kernel_class, digest, nbytes):
    return {"kernel_class": kernel_class, "digest": digest, "hbm_bytes_per_launch": nbytes}


def test_traffic_record_is_used_only_while_its_sources_match(tmp_path):
    path = tmp_path / "traffic.json"
    doc = {"workload": "w", "records": {
        "attention": _rec("attention", P.source_digest("attention"), 1234),
        "resid_norm": _rec("resid_norm", "0" * 64, 99),  # counters from older sources
    }}
    path.write_text(json.dumps(doc))
    assert P.load_traffic(str(path), "attention") == 1234
    assert P.load_traffic(str(path), "resid_norm") is None   # stale: never attached
    assert P.load_traffic(str(path), "gemm_o") is None       # no record for the class
    assert P.load_traffic(str(tmp_path / "missing.json"), "attention") is None


def test_counter_per_dispatch_sums_instances_and_reads_the_copy(tmp_path):
    # two counter instances of one dispatch are summed; the calibration copy
    # (a multiply over 64 Mi fp32 elements) is reported separately, and other
    # multiplies of the same kernel name (weight initialisation) are not
    # taken for it, however many there are
    mul = '"at::native::vectorized_elementwise_kernel<4, MulFunctor<float>>"'
    rows = [
        "Dispatch_Id,Grid_Size,Kernel_Name,Counter_Name,Counter_Value",
        "1,4096,reflex::k<1>(args),FETCH_SIZE,10",
        "1,4096,reflex::k<1>(args),FETCH_SIZE,5",
        "2,4096,reflex::k<1>(args),FETCH_SIZE,30",
        f"3,{P.COPY_GRID},{mul},FETCH_SIZE,400",
    ] + [f"{4 + i},11796480,{mul},FETCH_SIZE,300" for i in range(5)]
    path = tmp_path / "c.csv"
    path.write_text("\n".join(rows) + "\n")
    avg, n, copy = P.counter_per_dispatch(str(path), "FETCH_SIZE", r"reflex::k<1>")
    assert n == 2 and avg == 22.5 and copy == 400


def test_counter_per_dispatch_requires_the_copy(tmp_path):
    rows = ["Dispatch_Id,Grid_Size,Kernel_Name,Counter_Name,Counter_Value",
            "1,4096,reflex::k<1>(args),FETCH_SIZE,10",
            '2,11796480,"at::native::vectorized_elementwise_kernel<4, MulFunctor<float>>",FETCH_SIZE,300']
    path = tmp_path / "c.csv"
    path.write_text("\n".join(rows) + "\n")
    try:
        P.counter_per_dispatch(str(path), "FETCH_SIZE", r"reflex::k<1>")
    except ValueError as e:
        assert "calibration copy" in str(e)
    else:
        raise AssertionError("a run without the calibration copy must not yield a factor")


def _counter_csv(path, dispatches):
    """Counter-collection CSV: dispatches = [(name, grid, start, end, {counter: value})]."""
    hdr = ("Correlation_Id,Dispatch_Id,Agent_Id,Queue_Id,Process_Id,Thread_Id,Grid_Size,Kernel_Id,Kernel_Name,"
           "Workgroup_Size,LDS_Block_Size,Scratch_Size,VGPR_Count,Accum_VGPR_Count,SGPR_Count,Counter_Name,"
           "Counter_Value,Start_Timestamp,End_Timestamp")
    lines = [hdr]
    for i, (name, grid, t0, t1, cs) in enumerate(dispatches, 1):
        for c, v in cs.items():
            lines.append(f'{i},{i},"Agent 1",1,1,1,{grid},{i},"{name}",256,0,0,8,0,16,"{c}",{v},{t0},{t1}')
    path.write_text("\n".join(lines) + "\n")


def _trace_csv(path, dispatches):
    hdr = "Kind,Kernel_Name,Grid_Size_X,Grid_Size_Y,Grid_Size_Z,Start_Timestamp,End_Timestamp"
    lines = [hdr] + [f'KERNEL_DISPATCH,"{n}",{g},1,1,{t0},{t1}' for n, g, t0, t1, _ in dispatches]
    path.write_text("\n".join(lines) + "\n")


def test_classify_orders_the_fp32_projections():
    seq = ["reflex::gemm_skinny_lds<2, 1, 4, 8>(x)", "reflex::attn_pair_kernel<256>(x)",
           "reflex::attn_merge_kernel<unsigned short, 256, 2>(x)", "reflex::gemm_skinny_lds<4, 2, 0, 4>(x)",
           "reflex::resid_norm_kernel<unsigned short, 1>(x)", "reflex::gemm_skinny_lds<4, 1, 2, 8>(x)",
           "reflex::gemm_skinny_lds<4, 2, 0, 8>(x)", "reflex::gemm_big5<5, 64>(x)", "at::native::foo"]
    assert P.classify(seq) == ["gemm_qkv", "attention", "attn_merge", "gemm_o", "resid_norm", "gemm_gate_up",
                               "gemm_down", "frame_proj", "other"]


def test_summarize_calibrates_bytes_and_mfma_busy(tmp_path):
    copy = "at::native::vectorized_elementwise_kernel<4, MulFunctor<float>>"
    gemm = "reflex::gemm_dma<4, 2, 0, 96>(reflex::GemmArgs)"
    dur = 10_000  # ns
    busy = 0.25 * dur * P.CLOCK_GHZ * P.SIMDS   # a quarter of the MFMA cycles
    mops = 0.5 * 2500e12 * dur * 1e-9 / 512   # half the bf16 peak
    d_fetch = [(copy, P.COPY_GRID, 0, 50_000, {"FETCH_SIZE": 131072.0}),
               (gemm, 88064, 100_000, 100_000 + dur, {"FETCH_SIZE": 1000.0})]
    d_write = [(copy, P.COPY_GRID, 0, 50_000, {"WRITE_SIZE": 262144.0}),
               (gemm, 88064, 100_000, 100_000 + dur, {"WRITE_SIZE": 500.0})]
    d_mfma = [(copy, P.COPY_GRID, 0, 50_000, {"SQ_VALU_MFMA_BUSY_CYCLES": 0.0, "SQ_INSTS_VALU_MFMA_MOPS_BF16": 0.0}),
              (gemm, 88064, 100_000, 100_000 + dur, {"SQ_VALU_MFMA_BUSY_CYCLES": busy,
                                                     "SQ_INSTS_VALU_MFMA_MOPS_BF16": mops})]
    for name, d in (("fetch", d_fetch), ("write", d_write), ("mfma", d_mfma)):
        _counter_csv(tmp_path / f"{name}.csv", d)
    _trace_csv(tmp_path / "trace.csv", d_fetch)
    out = P.summarize("w", str(tmp_path / "trace.csv"), str(tmp_path / "fetch.csv"), str(tmp_path / "write.csv"),
                      str(tmp_path / "mfma.csv"), {"kt": "cmd"}, str(tmp_path / "s.md"), str(tmp_path / "t.json"))
    row = [r for r in out["rows"] if r["class"] == "gemm_qkv"][0]
    # fetch factor 2 (the copy reads 256 MiB but counts 128 Mi KiB-units), write factor 1
    assert row["hbm_bytes"] == 1000.0 * 1024 * 2 + 500.0 * 1024
    assert abs(row["mfma_busy"] - 0.25) < 1e-9
    assert abs(row["mfma_tflops"] - 1250.0) < 1e-6
    doc = json.loads((tmp_path / "t.json").read_text())
    assert doc["records"]["gemm_qkv"]["hbm_bytes_per_launch"] == round(row["hbm_bytes"])
    assert P.load_traffic(str(tmp_path / "t.json"), "gemm_qkv") == round(row["hbm_bytes"])


def test_stamp_validation_takes_only_the_stamped_dispatches(tmp_path):
    stamp = "(anonymous namespace)::stamp_kernel(unsigned long long*)"
    attn = "reflex::attn_pair_kernel<256>(reflex::AttnArgs)"
    merge = "reflex::attn_merge_kernel<unsigned short, 256, 2>(reflex::AttnArgs)"
    seq, t = [], 0

    def add(name, dur):
        nonlocal t
        seq.append((name, 64, t, t + dur, None))
        t += dur + 100

    add(attn, 9000)           # unstamped: ignored
    add(merge, 4000)
    for _ in range(3):        # stamped attention launches of 8 and 10 us
        add(stamp, 500)
        add(stamp, 500)
        add(attn, 8000 if _ % 2 == 0 else 10000)
        add(stamp, 500)
    add(merge, 3000)          # after the last launch's trailing stamp only: not stamped
    path = tmp_path / "kt.csv"
    _trace_csv(path, seq)
    rows = P.stamp_validation(str(path), {"attention": 8.5, "attn_merge": 3.0})
    assert [r["class"] for r in rows] == ["attention"]
    r = rows[0]
    assert r["stamped"] == 3
    assert abs(r["trace_us"] - (8.0 + 10.0 + 8.0) / 3) < 1e-9
    assert abs(r["ratio"] - 8.5 / r["trace_us"]) < 1e-12
