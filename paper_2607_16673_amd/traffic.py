"""Measured HBM traffic of the verify kernel from rocprofv3 counters.

Two steps, each run under its own `rocprofv3 --pmc <counter>` pass (one
pass for FETCH_SIZE, one for WRITE_SIZE; the counters cannot share a pass):

  copy      a plain device copy of a known size (reads N bytes, writes N
            bytes), the calibration: the counters' KiB per dispatch are
            scaled so that this copy reads and writes exactly N bytes;
  summarize reads the counter CSVs of the copy passes and of the bench
            passes and writes the calibrated HBM bytes per verify launch to
            profiles/traffic.json, which bench.py reports as
            roofline.traffic;
  sizes     checks the read calibration against the L2's read requests to
            HBM counted by size (32, 64 and 128 bytes), one more pass each
            over the copy and the bench.

Example (the full commands are recorded next to the numbers in profiles/):

  rocprofv3 --pmc FETCH_SIZE -d OUT/copy_fetch --output-format csv -- \\
      python3 -m paper_2607_16673_amd.traffic copy
  rocprofv3 --pmc FETCH_SIZE -d OUT/bench_fetch --output-format csv -- \\
      python3 bench.py --no-graph --steps 2 --warmup 1 --no-cpu-baseline
  (the same two with WRITE_SIZE)
  python3 -m paper_2607_16673_amd.traffic summarize --out-dir OUT \\
      --workload batched_tree_serving
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
COPY_MIB = 512
KERNEL_TAG = "verify_tile_kernel"
COPY_TAG = "mul"  # the elementwise multiply of run_copy (not the fill before it)


# the sources each counted kernel is built from (with the host code that
# chooses its launch): counters taken on other sources are stale
_COMMON = ["device.hpp", "kernels.hpp", "api.cpp"]
SOURCES = {
    "verify_tile_kernel": ["verify_tile.hip"] + _COMMON,
    "verify_serial_kernel": ["verify_serial.hip"] + _COMMON,
    "decode_kernel": ["decode.hip"] + _COMMON,
    "commit_kernel": ["commit.hip"] + _COMMON,
    "conv_verify_kernel": ["conv.hip", "device.hpp", "layer_ops.hpp", "api.cpp"],
    "conv_node_kernel": ["conv.hip", "device.hpp", "layer_ops.hpp", "api.cpp"],
}


def source_digest(kernel: str = KERNEL_TAG) -> str:
    """sha256 over the sources of one counted kernel."""
    h = hashlib.sha256()
    files = [os.path.join(HERE, "csrc", f) for f in SOURCES[kernel]]
    for fn in files:
        with open(fn, "rb") as f:
            h.update(os.path.basename(fn).encode() + b"\0" + f.read())
    return h.hexdigest()


def run_copy(mib: int = COPY_MIB) -> None:
    """Elementwise device copy of `mib` MiB (fp32), five dispatches."""
    import torch

    n = mib * (1 << 20) // 4
    a = torch.empty(n, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(5):
        torch.mul(a, 1.0, out=b)  # one elementwise kernel: reads a, writes b
    torch.cuda.synchronize()
    print("copy: %d MiB x 5 dispatches" % mib, flush=True)


def _rows(dirname: str, counter: str):
    files = glob.glob(os.path.join(dirname, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError("no counter_collection.csv under %s" % dirname)
    if len(files) > 1:
        # one pass is one process: more files mean results of several runs mixed in one folder
        raise RuntimeError("%d counter files under %s; give each pass a fresh folder" % (len(files), dirname))
    out = []
    for fn in files:
        with open(fn, newline="") as f:
            for r in csv.DictReader(f):
                if r.get("Counter_Name") == counter:
                    out.append(r)
    out.sort(key=lambda r: int(r.get("Dispatch_Id") or r.get("Correlation_Id") or 0))
    return out


def _per_dispatch_kib(rows, tag, skip=0):
    # a counter may be reported per XCD / per instance: sum per dispatch
    acc = {}
    order = []
    for r in rows:
        if tag.lower() not in r.get("Kernel_Name", "").lower():
            continue
        d = r.get("Dispatch_Id") or r.get("Correlation_Id")
        if d not in acc:
            acc[d] = 0.0
            order.append(d)
        acc[d] += float(r["Counter_Value"])
    vals = [acc[d] for d in order][skip:]
    if not vals:
        raise ValueError("no dispatch of a kernel matching %r" % tag)
    return sum(vals) / len(vals), len(vals)


def summarize(out_dir: str, workload: str, route: str, mode: str, skip: int, json_path: str,
              kernel: str = KERNEL_TAG, family: str = "gdn") -> dict:
    copy_bytes = COPY_MIB * (1 << 20)  # per copy dispatch, read and written
    cf, _ = _per_dispatch_kib(_rows(os.path.join(out_dir, "copy_fetch"), "FETCH_SIZE"), COPY_TAG, 0)
    cw, _ = _per_dispatch_kib(_rows(os.path.join(out_dir, "copy_write"), "WRITE_SIZE"), COPY_TAG, 0)
    scale_f = copy_bytes / (cf * 1024.0)
    scale_w = copy_bytes / (cw * 1024.0)
    bf, nf = _per_dispatch_kib(_rows(os.path.join(out_dir, "bench_fetch"), "FETCH_SIZE"), kernel, skip)
    bw, nw = _per_dispatch_kib(_rows(os.path.join(out_dir, "bench_write"), "WRITE_SIZE"), kernel, skip)
    fetch = bf * 1024.0 * scale_f
    write = bw * 1024.0 * scale_w
    key = "%s/%s/%s" % (workload, route, mode)
    if family != "gdn":
        key += "/" + family
    entry = {
        "kernel": kernel,
        "bytes_per_launch": int(round(fetch + write)),
        "fetch_bytes_per_launch": int(round(fetch)),
        "write_bytes_per_launch": int(round(write)),
        "fetch_kib_raw": round(bf, 1), "write_kib_raw": round(bw, 1),
        "copy_scale_fetch": round(scale_f, 4), "copy_scale_write": round(scale_w, 4),
        "dispatches": [nf, nw],
        "source_sha256": source_digest(kernel),
    }
    data = {}
    if os.path.exists(json_path):
        with open(json_path) as f:
            data = json.load(f)
    data[key] = entry
    with open(json_path, "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
        f.write("\n")
    return {key: entry}


SIZE_COUNTERS = {32: "TCC_EA0_RDREQ_32B_sum", 64: "TCC_EA0_RDREQ_64B_sum", 128: "TCC_EA0_RDREQ_128B_sum"}


def _bytes_by_request_size(dirname: str, tag: str, skip: int):
    """Read bytes per dispatch from the L2's read requests to HBM counted by
    size (one pass holding the three SIZE_COUNTERS), and the request counts."""
    counts = {}
    n = 0
    for size, name in SIZE_COUNTERS.items():
        v, n = _per_dispatch_kib(_rows(dirname, name), tag, skip)
        counts[size] = v
    return sum(size * c for size, c in counts.items()), counts, n


def summarize_sizes(out_dir: str, key: str, skip: int, json_path: str, kernel: str = KERNEL_TAG) -> dict:
    """Checks the FETCH_SIZE calibration with a direct count.  The copy and
    the bench each get one rocprofv3 --pmc pass over SIZE_COUNTERS (folders
    copy_sizes and bench_sizes); the read bytes are 32, 64 and 128 times the
    requests of each size.  Recorded beside the calibrated entry `key` of
    traffic.json: the direct count per launch, the request mix, and its
    ratio to the calibrated FETCH_SIZE figure (1.0 when the copy's scale
    holds for this kernel) and to the copy's known bytes."""
    copy_bytes = COPY_MIB * (1 << 20)
    cb, ccounts, _ = _bytes_by_request_size(os.path.join(out_dir, "copy_sizes"), COPY_TAG, 0)
    kb, kcounts, n = _bytes_by_request_size(os.path.join(out_dir, "bench_sizes"), kernel, skip)
    with open(json_path) as f:
        data = json.load(f)
    if key not in data:
        raise KeyError("no calibrated entry %r in %s" % (key, json_path))
    entry = data[key]
    tot = sum(kcounts.values()) or 1.0
    entry["read_check"] = {
        "fetch_bytes_by_request_size": int(round(kb)),
        "request_mix": {str(s): round(c / tot, 4) for s, c in kcounts.items()},
        "ratio_to_calibrated_fetch": round(kb / entry["fetch_bytes_per_launch"], 4),
        "copy_bytes_by_request_size_over_known": round(cb / copy_bytes, 4),
        "dispatches": n,
        "source_sha256": source_digest(kernel),
    }
    with open(json_path, "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
        f.write("\n")
    return {key: entry["read_check"]}


def mfma_counters(dtype: str = "bf16"):
    """The counters of one matrix-core pass: busy cycles, the MFMA operations
    of the activation dtype's products (bf16 or f32), CU and GPU activity."""
    return ["SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU_MFMA_MOPS_%s" % dtype.upper(), "SQ_BUSY_CU_CYCLES",
            "GRBM_GUI_ACTIVE"]


MFMA_COUNTERS = mfma_counters("bf16")


def summarize_mfma(out_dir: str, workload: str, skip: int, json_path: str, kernel: str = KERNEL_TAG,
                   simds: int = 1024, dtype: str = "bf16") -> dict:
    """Matrix-core use of the verify kernel from one rocprofv3 --pmc pass with
    mfma_counters(dtype), per launch: MFMA busy cycles per SIMD (busy cycles
    summed over the SIMDs / simds) and the MFMA operations of that dtype
    (SQ_INSTS_VALU_MFMA_MOPS_* counts multiply and add operations / 512).
    GRBM_GUI_ACTIVE is kept for reference only: under counter collection it
    spans more than the kernel (dispatches are serialised and sampled), so
    utilisation is taken against the kernel-trace duration instead."""
    files = glob.glob(os.path.join(out_dir, "**", "*counter_collection.csv"), recursive=True)
    if len(files) != 1:
        raise RuntimeError("expected one counter file under %s, found %d" % (out_dir, len(files)))
    acc = {}
    order = []
    with open(files[0], newline="") as f:
        for r in csv.DictReader(f):
            if kernel.lower() not in r.get("Kernel_Name", "").lower():
                continue
            d = r.get("Dispatch_Id") or r.get("Correlation_Id")
            if d not in acc:
                acc[d] = {}
                order.append(d)
            c = r["Counter_Name"]
            v = float(r["Counter_Value"])
            # GRBM_GUI_ACTIVE is per XCD: the launch's span is the largest one
            acc[d][c] = max(acc[d].get(c, 0.0), v) if c == "GRBM_GUI_ACTIVE" else acc[d].get(c, 0.0) + v
    rows = [acc[d] for d in order][skip:]
    if not rows:
        raise ValueError("no dispatch of %r" % kernel)
    counters = mfma_counters(dtype)
    mean = {c: sum(r.get(c, 0.0) for r in rows) / len(rows) for c in counters}
    entry = {
        "kernel": kernel, "dispatches": len(rows), "simds": simds,
        "mfma_busy_cycles_per_simd": mean["SQ_VALU_MFMA_BUSY_CYCLES"] / simds,
        "%s_mfma_flops" % dtype.lower(): mean[counters[1]] * 512,
        "gui_active_cycles_under_collection": mean["GRBM_GUI_ACTIVE"],
        "source_sha256": source_digest(kernel),
    }
    data = {}
    if os.path.exists(json_path):
        with open(json_path) as f:
            data = json.load(f)
    data["%s/mfma" % workload] = entry
    with open(json_path, "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
        f.write("\n")
    return entry


def main(argv=None) -> None:
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    c = sub.add_parser("copy")
    c.add_argument("--mib", type=int, default=COPY_MIB)
    s = sub.add_parser("summarize")
    s.add_argument("--out-dir", required=True)
    s.add_argument("--workload", required=True)
    s.add_argument("--route", default="auto", help="auto, serial, parallel, or conv for the convolution")
    s.add_argument("--kernel", default=KERNEL_TAG, help="kernel name substring to average")
    s.add_argument("--mode", default="fused")
    s.add_argument("--family", default="gdn", help="layer family the bench ran (bench.py --family)")
    s.add_argument("--skip", type=int, default=0,
                   help="leading verify dispatches to ignore (the first step has no pending path)")
    s.add_argument("--json", default=os.path.join(ROOT, "profiles", "traffic.json"))
    m = sub.add_parser("mfma")
    m.add_argument("--out-dir", required=True)
    m.add_argument("--workload", required=True)
    m.add_argument("--skip", type=int, default=0)
    m.add_argument("--dtype", default="bf16", help="bf16 or f32: the MFMA operations counted")
    m.add_argument("--json", default=os.path.join(ROOT, "profiles", "traffic.json"))
    z = sub.add_parser("sizes", help="check the FETCH_SIZE calibration with read requests counted by size")
    z.add_argument("--out-dir", required=True)
    z.add_argument("--key", required=True, help="traffic.json entry, e.g. batched_tree_serving/auto/fused")
    z.add_argument("--kernel", default=KERNEL_TAG)
    z.add_argument("--skip", type=int, default=0)
    z.add_argument("--json", default=os.path.join(ROOT, "profiles", "traffic.json"))
    a = ap.parse_args(argv)
    if a.cmd == "sizes":
        print(json.dumps(summarize_sizes(a.out_dir, a.key, a.skip, a.json, a.kernel), indent=1))
    elif a.cmd == "copy":
        run_copy(a.mib)
    elif a.cmd == "mfma":
        print(json.dumps(summarize_mfma(a.out_dir, a.workload, a.skip, a.json, dtype=a.dtype), indent=1))
    else:
        print(json.dumps(summarize(a.out_dir, a.workload, a.route, a.mode, a.skip, a.json, a.kernel, a.family),
                         indent=1))


if __name__ == "__main__":
    sys.exit(main())
