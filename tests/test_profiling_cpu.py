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
