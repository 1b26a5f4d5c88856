"""Benchmark: cache-cold batched FFT throughput on one MI355X, plus the SAR chain.

One step is one forward FFT of the N = 4096, batch 32768, complex FP32 batch
(1 GiB in, 1 GiB out: the whole working set is eight times the 256 MiB
Infinity Cache, so every step streams from HBM).  ``value`` is algorithmic
bytes (one read and one write per point, Section IV eq. (1)) over the wall
time of the K timed steps.  The JSON line also carries:

  roofline      the FFT kernel's algorithmic bytes per launch over its average
                duration (HIP events around the timed launches on the launch
                stream), against the 8 TB/s HBM peak; ``traffic`` comes from the
                committed rocprofv3 FETCH_SIZE/WRITE_SIZE measurement when it
                was taken on the current kernel sources, else null;
  cpu_baseline  the fp64 oracle timed on this host on a bounded sample of the
                same workload;
  breakdown     the other workloads (N = 1024 latency case, 8192, 16384, FP16
                storage, a 2^20-point transform in the two-pass four-step form, the 4096 x 4096 two-pass SAR image and the 4096 x
                4096 full range-Doppler image of the paper's L-band scene, with
                FP32 and FP16 intermediates), each a median of cache-flushed
                samples.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "batched FFT GB/s and % HBM peak at N=4096/8192/16384 (cache-cold); SAR ms/image"
WORKLOAD = "fft_n4096_b32768_fp32"
HBM_PEAK_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_digest() -> str:
    """sha256 over the kernel sources; a traffic measurement is valid only for it."""
    csrc = os.path.join(ROOT, "paper_2609_32237_amd", "csrc")
    h = hashlib.sha256()
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".hpp", ".h")):
            h.update(name.encode())
            h.update(open(os.path.join(csrc, name), "rb").read())
    return h.hexdigest()[:16]


def gflops(n, batch, seconds):
    return 5.0 * n * np.log2(n) * batch / seconds / 1e9


class Flusher:
    """Reads a 1 GiB buffer on the current stream: evicts the 256 MiB Infinity
    Cache and every L2 before a cache-cold sample (Section III's cold runs).
    A read leaves clean lines behind; a write-based flush would leave dirty
    lines whose write-back lands inside the next timed call."""

    def __init__(self, torch):
        self.buf = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        self.acc = torch.empty((), dtype=torch.float32, device="cuda")
        self.torch = torch

    def __call__(self):
        self.torch.sum(self.buf, dim=0, out=self.acc)


def time_samples(torch, fn, flush, samples, warmup=2):
    """Median and quartiles (ms) of single calls, each after a cache flush."""
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(samples)]
    for _ in range(warmup):
        flush()
        fn()
    for a, b in ev:
        flush()
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    ms = np.array([a.elapsed_time(b) for a, b in ev])
    return float(np.median(ms)), float(np.percentile(ms, 25)), float(np.percentile(ms, 75))


def fft_breakdown(torch, api, flush, name, samples):
    import workloads

    w = workloads.FFT_WORKLOADS[name]
    n, batch, storage = w["n"], w["batch"], w["storage"]
    x = torch.from_numpy(workloads.fft_workload(name)).cuda()
    out = torch.empty_like(x)
    plan = api.Plan(n, batch, 1, n, 0 if storage == "fp32" else 1, -1)
    med, q1, q3 = time_samples(torch, lambda: plan.execute(x, out), flush, samples)
    plan.close()
    bytes_ = 2 * n * batch * (8 if storage == "fp32" else 4)
    del x, out
    torch.cuda.empty_cache()
    gbs = bytes_ / (med * 1e-3) / 1e9
    return {"n": n, "batch": batch, "storage": storage, "ms_median": round(med, 5), "ms_iqr": [round(q1, 5), round(q3, 5)],
            "GB/s": round(gbs, 1), "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
            "GFLOPS": round(gflops(n, batch, med * 1e-3), 1)}


def matrix_unit_experiment(torch, api, flush, samples):
    """FP16 storage, 1 GiB batches: the vector kernels (FP32 exchange), the FP16
    exchange and the radix-16 butterflies on the matrix cores (Section VIII)."""
    res = {"experiment": "matrix-units", "storage": "fp16", "results": []}
    g = torch.Generator(device="cuda").manual_seed(12)
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < 2.0:  # a fresh process: bring the clocks up first
        for _ in range(20):
            flush()
        torch.cuda.synchronize()
    for n in (4096, 16384):
        batch = (1 << 30) // (n * 4)
        x = (torch.rand(batch, n, 2, device="cuda", generator=g) * 2 - 1).half()
        out = torch.empty_like(x)
        for name, flags in (("vector", 0), ("fp16_exchange", api._lib.FFT_FLAG_FP16_EXCHANGE),
                            ("matrix_units", api._lib.FFT_FLAG_MATRIX_UNITS)):
            plan = api.Plan(n, batch, 1, n, 1, -1, flags=flags)
            med, q1, q3 = time_samples(torch, lambda: plan.execute(x, out), flush, samples)
            plan.close()
            gbs = 8 * n * batch / (med * 1e-3) / 1e9
            res["results"].append({"n": n, "batch": batch, "kernels": name, "ms_median": round(med, 5),
                                   "ms_iqr": [round(q1, 5), round(q3, 5)], "GB/s": round(gbs, 1),
                                   "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4)})
        del x, out
        torch.cuda.empty_cache()
    return res


def long_breakdown(torch, api, flush, n, batch, samples):
    """A transform longer than the chip holds: the two-pass four-step form.
    GB/s counts the method's own 16 bytes per point (one read, one write);
    the two passes move twice that."""
    g = torch.Generator(device="cuda").manual_seed(11)
    x = torch.view_as_complex(torch.rand(batch, n, 2, device="cuda", generator=g) * 2 - 1)
    out = torch.empty_like(x)
    plan = api.Plan(n, batch, 1, n, 0, -1)
    med, q1, q3 = time_samples(torch, lambda: plan.execute(x, out), flush, samples)
    plan.close()
    gbs = 16 * n * batch / (med * 1e-3) / 1e9
    return {"n": n, "batch": batch, "storage": "fp32", "passes": 2, "ms_median": round(med, 5),
            "ms_iqr": [round(q1, 5), round(q3, 5)], "GB/s": round(gbs, 1), "moved_GB/s": round(2 * gbs, 1),
            "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4), "GFLOPS": round(gflops(n, batch, med * 1e-3), 1)}


def sar_breakdown(torch, api, flush, inter, samples):
    import workloads

    sc = workloads.sar_scene()
    raw = torch.from_numpy(sc.raw).cuda()
    hr = torch.from_numpy(sc.range_ref).cuda()
    ha = torch.from_numpy(sc.az_ref).cuda()
    out = torch.empty_like(raw)
    ws = torch.empty(api._lib.sar_workspace_bytes(4096, 4096, inter), dtype=torch.uint8, device="cuda")
    fn = lambda: api.sar_form_image(raw, hr, ha, inter, out=out, workspace=ws)  # noqa: E731
    med, q1, q3 = time_samples(torch, fn, flush, samples)
    bpp = 32 if inter == 0 else 24  # raw read + intermediate write + read + image write
    bytes_ = bpp * 4096 * 4096
    gbs = bytes_ / (med * 1e-3) / 1e9
    return {"image": "4096x4096", "intermediate": "fp32" if inter == 0 else "fp16", "ms_median": round(med, 5),
            "ms_iqr": [round(q1, 5), round(q3, 5)], "algorithmic_bytes_per_point": bpp, "GB/s": round(gbs, 1),
            "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4)}


def rd_breakdown(torch, api, flush, inter, samples):
    """The paper's full range-Doppler chain on its 4096 x 4096 L-band scene."""
    import workloads

    sc = workloads.rd_scene()
    raw = torch.from_numpy(sc.raw).cuda()
    hr = torch.from_numpy(sc.range_ref).cuda()
    out = torch.empty_like(raw)
    ws = torch.empty(api._lib.sar_rd_workspace_bytes(4096, 4096, inter), dtype=torch.uint8, device="cuda")
    fn = lambda: api.sar_rd_form_image(raw, hr, sc.geometry, inter, out=out, workspace=ws)  # noqa: E731
    med, q1, q3 = time_samples(torch, fn, flush, samples)
    # raw read, range-compressed write + read, range-Doppler write + read, image write
    bpp = 48 if inter == 0 else 32
    gbs = bpp * 4096 * 4096 / (med * 1e-3) / 1e9
    return {"image": "4096x4096", "scene": "L-band stripmap, 6 targets (Section X)",
            "intermediate": "fp32" if inter == 0 else "fp16", "passes": 3, "ms_median": round(med, 5),
            "ms_iqr": [round(q1, 5), round(q3, 5)], "algorithmic_bytes_per_point": bpp, "GB/s": round(gbs, 1),
            "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4)}


def cpu_baseline(x_host, n, target_s=10.0):
    """The fp64 oracle on a bounded sample of the workload, on this host's cores
    (median of three timings of the same sample)."""
    import oracle

    threads = oracle.default_threads()
    probe = 256
    t0 = time.perf_counter()
    oracle.fft(x_host[:probe], nthreads=threads)
    t_probe = time.perf_counter() - t0
    count = int(min(x_host.shape[0], max(probe, probe * target_s / 3 / max(t_probe, 1e-6))))
    xs = x_host[:count].astype(np.complex128)  # widening is not timed
    times = []
    for _ in range(3):
        t0 = time.perf_counter()
        oracle.fft_layout(xs, n, count, 1, n, -1, nthreads=threads)
        times.append(time.perf_counter() - t0)
    dt = float(np.median(times))
    return {"value": round(16.0 * n * count / dt / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"first {count} of {x_host.shape[0]} transforms (N={n}, fp64 radix-2), median of 3 "
                      f"timings, {dt:.2f} s each"}


def copy_reference(torch):
    """Read+write bandwidth of a plain streaming kernel on this GPU: an in-place
    scale of a 1 GiB buffer (reads and writes every byte once), median of 10."""
    buf = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    for _ in range(3):
        buf.mul_(1.0)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(10)]
    for a, b in ev:
        a.record()
        buf.mul_(1.0)
        b.record()
    torch.cuda.synchronize()
    ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    del buf
    torch.cuda.empty_cache()
    return 2.0 * (1 << 30) / (ms * 1e-3) / 1e9


def load_traffic(digest: str):
    path = os.path.join(PROFILES, f"traffic_{WORKLOAD}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("kernel_source_digest") != digest:
        return None
    return rec.get("bytes_per_launch")


def summarize(prof_dir: str, command: str) -> str:
    """Text summary of rocprofv3 CSV output: per-kernel durations (kernel trace)
    or per-dispatch counter values (--pmc), for committing under profiles/."""
    import csv
    import glob
    from collections import defaultdict

    lines = [f"command: {command}", f"source: {prof_dir}"]
    traces = glob.glob(os.path.join(prof_dir, "**", "*kernel_trace.csv"), recursive=True)
    pmcs = glob.glob(os.path.join(prof_dir, "**", "*counter_collection.csv"), recursive=True)
    for path in traces:
        groups = defaultdict(list)
        for r in csv.DictReader(open(path)):
            key = (r["Kernel_Name"], r["Grid_Size_X"], r["Workgroup_Size_X"], r["LDS_Block_Size"],
                   r["VGPR_Count"], r["Scratch_Size"])
            groups[key].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
        lines.append("kernel trace (durations in us): calls, mean, median, min, max | grid, wg, lds, vgpr, scratch | name")
        for key, d in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
            d = np.array(d)
            lines.append(f"{len(d):5d} {d.mean():10.2f} {np.median(d):10.2f} {d.min():10.2f} {d.max():10.2f} | "
                         f"{key[1]} {key[2]} {key[3]} {key[4]} {key[5]} | {key[0][:200]}")
    for path in pmcs:
        groups = defaultdict(list)
        for r in csv.DictReader(open(path)):
            groups[(r["Kernel_Name"], r["Grid_Size"], r["Counter_Name"])].append(float(r["Counter_Value"]))
        lines.append("counters per dispatch: dispatches, mean value | grid | counter | name")
        for key, v in sorted(groups.items()):
            lines.append(f"{len(v):5d} {np.mean(v):16.1f} | {key[1]} | {key[2]} | {key[0][:200]}")
    return "\n".join(lines) + "\n"


def _pmc_means(prof_dir: str, counter: str):
    """{(kernel name, grid): mean counter value per dispatch} from a --pmc run."""
    import csv
    import glob
    from collections import defaultdict

    vals = defaultdict(list)
    for path in glob.glob(os.path.join(prof_dir, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] == counter:
                vals[(r["Kernel_Name"], int(r["Grid_Size"]))].append(float(r["Counter_Value"]))
    return {k: float(np.mean(v)) for k, v in vals.items()}


def make_traffic(fetch_dir: str, write_dir: str, commands: list) -> dict:
    """HBM-side bytes per launch of the benchmarked FFT kernel from two --pmc runs
    (FETCH_SIZE, WRITE_SIZE; KiB per dispatch), each scaled by what the same
    counter reads for the copy-reference kernel, which reads and writes exactly
    1 GiB per dispatch."""
    rec = {"workload": WORKLOAD, "kernel_source_digest": kernel_source_digest(), "commands": commands}
    n, batch = 4096, 32768
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        means = _pmc_means(d, counter)
        fft = [v for (name, grid), v in means.items() if "fft_kernel<mi355fft::KCfg<4096," in name
               and grid == batch * 256 and "(mi355fft::EPI" not in name]
        calib = [v for (name, grid), v in means.items() if "MulFunctor" in name and grid >= (1 << 26)]
        if not fft or not calib:
            raise RuntimeError(f"{counter}: benchmark or reference kernel missing in {d}")
        factor = ((1 << 30) / 1024.0) / calib[0]
        key = "fetch" if counter == "FETCH_SIZE" else "write"
        rec[f"{key}_kib_per_dispatch_raw"] = fft[0]
        rec[f"{key}_reference_kib_per_dispatch_raw"] = calib[0]
        rec[f"{key}_scale"] = factor
        rec[f"{key}_bytes_per_launch"] = fft[0] * 1024.0 * factor
    rec["algorithmic_bytes_per_launch"] = 16 * n * batch
    rec["bytes_per_launch"] = rec["fetch_bytes_per_launch"] + rec["write_bytes_per_launch"]
    return rec


def main():
    if len(sys.argv) > 1 and sys.argv[1] == "--summarize":
        print(summarize(sys.argv[2], " ".join(sys.argv[3:])), end="")
        return
    if len(sys.argv) > 1 and sys.argv[1] == "--make-traffic":
        print(json.dumps(make_traffic(sys.argv[2], sys.argv[3], sys.argv[4:]), indent=1))
        return
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--samples", type=int, default=11, help="cache-flushed samples per breakdown workload")
    ap.add_argument("--no-breakdown", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--experiment", choices=["matrix-units"], default=None,
                    help="instead of the benchmark: FP16-storage N = 4096 / 16384 with the vector kernels, the "
                         "FP16 exchange and the matrix-core butterflies (one JSON line)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU; --gpus must be 1",
                          "note": "batched transforms shard by batch with no communication"}))
        sys.exit(2)

    import torch

    import workloads
    from paper_2609_32237_amd import torch_api as api

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.experiment == "matrix-units":
        print(json.dumps(matrix_unit_experiment(torch, api, Flusher(torch), args.samples)), flush=True)
        return
    w = workloads.FFT_WORKLOADS[WORKLOAD]
    n, batch = w["n"], w["batch"]
    log(f"generating {WORKLOAD}")
    x_host = workloads.fft_workload(WORKLOAD)
    x = torch.from_numpy(x_host).cuda()
    out = torch.empty_like(x)
    plan = api.Plan(n, batch, 1, n, 0, -1)
    step_bytes = 2 * 8 * n * batch

    for _ in range(args.warmup):
        plan.execute(x, out)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        plan.execute(x, out)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kernel_ms = e0.elapsed_time(e1) / args.steps
    value = step_bytes * args.steps / wall / 1e9
    achieved = step_bytes / (kernel_ms * 1e-3) / 1e9

    digest = kernel_source_digest()
    plan.close()
    del x, out
    torch.cuda.empty_cache()
    copy_gbs = copy_reference(torch)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": load_traffic(digest),
                "kernel": "fft_kernel rows N=4096 fp32 forward", "algorithmic_bytes_per_launch": step_bytes,
                "avg_launch_ms": round(kernel_ms, 5), "kernel_source_digest": digest,
                "measured_copy_GBs": round(copy_gbs, 1), "frac_of_measured_copy": round(achieved / copy_gbs, 4)}
    result = {
        "metric": METRIC, "value": round(value, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(wall * 1e3 / args.steps, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": WORKLOAD, "n": n, "batch": batch, "storage": "fp32", "direction": "forward",
                   "layout": "contiguous rows", "cache": "cold: 2 GiB working set vs 256 MiB Infinity Cache",
                   "gflops_5nlog2n": round(gflops(n, batch, wall / args.steps), 1)},
        "roofline": roofline,
    }

    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        result["cpu_baseline"] = cpu_baseline(x_host, n)
    del x_host

    if not args.no_breakdown:
        flush = Flusher(torch)
        bd = {}
        for name in ("fft_n1024_b64_fp32", "fft_n4096_b32768_fp32", "fft_n8192_b16384_fp32",
                     "fft_n16384_b8192_fp32", "fft_n16384_b16384_fp16"):
            log(f"breakdown {name}")
            bd[name] = fft_breakdown(torch, api, flush, name, args.samples)
        log("breakdown fft_n1048576_b128_fp32 (four-step)")
        bd["fft_n1048576_b128_fp32"] = long_breakdown(torch, api, flush, 1 << 20, 128, args.samples)
        for inter in (0, 1):
            log(f"breakdown sar inter={inter}")
            bd[f"sar_4096x4096_{'fp32' if inter == 0 else 'fp16'}_inter"] = sar_breakdown(
                torch, api, flush, inter, args.samples)
        for inter in (0, 1):
            log(f"breakdown range-Doppler inter={inter}")
            bd[f"rd_4096x4096_{'fp32' if inter == 0 else 'fp16'}_inter"] = rd_breakdown(
                torch, api, flush, inter, args.samples)
        result["breakdown"] = bd
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
