"""Host logic of the counter summaries (paper_2607_16673_amd.traffic) on
synthetic rocprofv3 counter files: the FETCH_SIZE / WRITE_SIZE calibration
against a copy of known size, per-dispatch sums over counter instances,
skipped leading dispatches, and the read check by request size."""
import csv
import json
import os

import pytest

from paper_2607_16673_amd import traffic as T


def _write(dirname, rows):
    os.makedirs(os.path.join(dirname, "host"), exist_ok=True)
    fn = os.path.join(dirname, "host", "1_counter_collection.csv")
    with open(fn, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for r in rows:
            w.writerow(r)


def _rows(kernel, counter, per_dispatch, instances=2, first=1):
    out = []
    for i, v in enumerate(per_dispatch):
        for _ in range(instances):  # the value split over counter instances
            out.append(dict(Dispatch_Id=first + i, Kernel_Name=kernel, Counter_Name=counter,
                            Counter_Value=v / instances))
    return out


COPY_KIB = T.COPY_MIB * 1024


def test_calibrated_bytes_and_read_check(tmp_path):
    d = str(tmp_path)
    # the copy: FETCH_SIZE reads half the known bytes (128-byte requests
    # counted as 64), WRITE_SIZE exactly the known bytes
    _write(os.path.join(d, "copy_fetch"), _rows("void at::native::mul_kernel", "FETCH_SIZE", [COPY_KIB / 2] * 5))
    _write(os.path.join(d, "copy_write"), _rows("void at::native::mul_kernel", "WRITE_SIZE", [COPY_KIB] * 5))
    # the kernel: a first dispatch to skip, then two at 1000 / 3000 KiB raw
    kern = "void sla::verify_tile_kernel<128, 16, 4, 2, 0, false, true>(sla::VerifyArgs)"
    _write(os.path.join(d, "bench_fetch"), _rows(kern, "FETCH_SIZE", [7.0, 1000.0, 3000.0]))
    _write(os.path.join(d, "bench_write"), _rows(kern, "WRITE_SIZE", [5.0, 500.0, 1500.0]))
    js = os.path.join(d, "traffic.json")
    out = T.summarize(d, "w", "auto", "fused", 1, js)
    e = out["w/auto/fused"]
    assert e["copy_scale_fetch"] == pytest.approx(2.0) and e["copy_scale_write"] == pytest.approx(1.0)
    assert e["fetch_bytes_per_launch"] == 2000 * 1024 * 2
    assert e["write_bytes_per_launch"] == 1000 * 1024
    assert e["dispatches"] == [2, 2]
    # read requests by size: the copy all 128-byte requests; the kernel's
    # mix gives exactly the calibrated figure
    nreq = T.COPY_MIB * (1 << 20) // 128
    copy_rows = (_rows("mul_kernel", "TCC_EA0_RDREQ_32B_sum", [0] * 5)
                 + _rows("mul_kernel", "TCC_EA0_RDREQ_64B_sum", [0] * 5)
                 + _rows("mul_kernel", "TCC_EA0_RDREQ_128B_sum", [nreq] * 5))
    _write(os.path.join(d, "copy_sizes"), copy_rows)
    target = 2000 * 1024 * 2  # bytes
    n64 = 1024
    n128 = (target - 64 * n64) // 128
    krows = (_rows(kern, "TCC_EA0_RDREQ_32B_sum", [9, 0, 0]) + _rows(kern, "TCC_EA0_RDREQ_64B_sum", [9, n64, n64])
             + _rows(kern, "TCC_EA0_RDREQ_128B_sum", [9, n128, n128]))
    _write(os.path.join(d, "bench_sizes"), krows)
    chk = T.summarize_sizes(d, "w/auto/fused", 1, js)["w/auto/fused"]
    assert chk["fetch_bytes_by_request_size"] == target
    assert chk["ratio_to_calibrated_fetch"] == pytest.approx(1.0)
    assert chk["copy_bytes_by_request_size_over_known"] == pytest.approx(1.0)
    assert chk["request_mix"]["32"] == 0.0 and chk["dispatches"] == 2
    with open(js) as f:
        assert json.load(f)["w/auto/fused"]["read_check"] == chk


def test_mixed_runs_in_one_folder_are_refused(tmp_path):
    d = str(tmp_path / "bench_fetch")
    _write(d, _rows("k", "FETCH_SIZE", [1.0]))
    os.makedirs(os.path.join(d, "other"))
    with open(os.path.join(d, "other", "2_counter_collection.csv"), "w") as f:
        f.write("Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value\n")
    with pytest.raises(RuntimeError):
        T._rows(d, "FETCH_SIZE")


def test_missing_kernel_is_an_error(tmp_path):
    d = str(tmp_path / "bench_fetch")
    _write(d, _rows("other_kernel", "FETCH_SIZE", [1.0]))
    with pytest.raises(ValueError):
        T._per_dispatch_kib(T._rows(d, "FETCH_SIZE"), "verify_tile_kernel")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_mfma_summary_counts_the_dtype_operations(tmp_path, dtype):
    d = str(tmp_path / "mfma")
    kern = "void sla::verify_tile_kernel<128, 64, 8, 2, 0, true, false>(sla::VerifyArgs)"
    names = T.mfma_counters(dtype)
    rows = []
    for name, vals in zip(names, [[0, 4096.0, 4096.0], [0, 1000.0, 3000.0], [0, 7.0, 7.0], [0, 50.0, 70.0]]):
        rows += _rows(kern, name, vals, instances=1)
    _write(d, rows)
    e = T.summarize_mfma(d, "w", 1, str(tmp_path / "t.json"), dtype=dtype)
    assert e["%s_mfma_flops" % dtype] == 2000.0 * 512
    assert e["mfma_busy_cycles_per_simd"] == 4096.0 / 1024
    assert e["dispatches"] == 2
