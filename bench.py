"""Benchmark of the 1xN-pruned convolution forward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c1] [--no-cpu]

A step is one forward pass of the workload's pruned layer(s) (Eq. 8 on the
GPU) over one batch of synthetic input already resident in HBM.  Mask
building and packing are the offline part of the method (done once per layer
before deployment) and run before the timed region.  To keep timed steps from
hitting the 256 MB Infinity Cache with the previous step's data, the input and
output buffers rotate over enough copies to exceed 512 MB.

Prints one JSON line.  value = actual TFLOP/s (2 * pixels * N * kh * kw * t
per layer, summed) over the timed steps; the dense-equivalent rate and the
HBM rate are reported beside it.
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import paper_2105_14713_amd as onexn  # noqa: E402
import workloads  # noqa: E402

PEAK_HBM_GBPS = 8000.0
PEAK_TFLOPS = {"f32": 157.3, "bf16": 2516.6}
METRIC = "1×N sparse conv fwd: actual & dense-equiv TFLOP/s, % of MFMA/HBM roofline"
ROTATE_BYTES = 512 << 20

WORKLOADS = {
    "c0": workloads.config0,
    "c1": workloads.config1,
    "c2": workloads.config2,
    "c4": lambda: workloads.config4("bf16"),
    "c4f32": lambda: workloads.config4("f32"),
}
for _N in (4, 8, 16, 32):
    for _p in (0.3, 0.5, 0.7):
        WORKLOADS[f"c3_n{_N}_p{int(_p * 100)}"] = (lambda N=_N, p=_p: workloads.config3(N, p))

_ESIZE = {"f32": 4, "bf16": 2}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
COPY_BYTES = 256 << 20
_TDT = {"f32": torch.float32, "bf16": torch.bfloat16}


def layer_work(layer, packed, batch, dtype, out_dtype):
    """Algorithmic flops and HBM bytes of one forward of one layer."""
    px = layer.out_pixels(batch)
    kk = layer.k * layer.k
    f_act = 2.0 * px * layer.N * kk * packed.t
    f_dense = 2.0 * px * layer.cout * layer.cin * kk
    used_ch = int((packed.mask.sum(dim=1) > 0).sum())
    e = _ESIZE[dtype]
    b_x = batch * layer.H * layer.H * used_ch * e
    b_y = px * layer.cout * _ESIZE[out_dtype]
    b_w = packed.t * layer.N * kk * e + packed.t * 4 + (packed.P.numel()) * 4
    return f_act, f_dense, b_x + b_y + b_w


def source_hash(files):
    """sha256 over the named source files (paths relative to the repository
    root): byte counters taken on an older build of a kernel are not reported
    for a newer one."""
    h = hashlib.sha256()
    for name in sorted(files):
        h.update(name.encode())
        with open(os.path.join(ROOT, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per launch of the workload's kernel from the committed
    rocprofv3 counter summary (FETCH_SIZE and WRITE_SIZE in KiB per dispatch,
    each scaled by the factor the same counter shows for a copy kernel of
    known size), or None when there is none, or when any source file the
    kernel is built from (listed in the record) has changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    w = rec.get("workloads", {}).get(workload)
    if not w:
        return None
    try:
        if w.get("source_sha256") != source_hash(w["sources"]):
            return None
    except (OSError, KeyError):
        return None
    return 1024.0 * (w["fetch_kib"] * rec["fetch_scale"] + w["write_kib"] * rec["write_scale"])


def copy_calibration(dev):
    """A plain copy-like kernel of known size (elementwise negate of a 256 MiB
    fp32 buffer into another) for scaling the rocprofv3 byte counters."""
    src = torch.randn(COPY_BYTES // 4, device=dev)
    dst = torch.empty_like(src)
    for _ in range(5):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_kernel": "torch.neg fp32", "bytes_read": COPY_BYTES,
                      "bytes_written": COPY_BYTES, "launches": 5}), flush=True)


def cpu_baseline(layers, batch, wl, budget_s):
    """The oracle (direct 7-loop over the masked dense weight, fp64) on the host
    cores, over a bounded sample: single images through all the workload's
    layers, cycling over the batch until the time budget is spent."""
    import oracle
    done_f, spent, imgs = 0.0, 0.0, 0
    lw = []
    for layer in layers:
        w, x = workloads.gen_layer(layer, 1, wl.dtype)
        pr = oracle.prune(w.double().numpy(), layer.N, layer.p, layer.rearrange)
        lw.append((layer, pr, x.double().numpy()))
    while spent < budget_s:
        for layer, pr, x in lw:
            t0 = time.perf_counter()
            oracle.conv2d(x, pr.wbar, (layer.stride,) * 2, (layer.pad,) * 2)
            spent += time.perf_counter() - t0
            done_f += 2.0 * layer.Ho * layer.Ho * layer.N * layer.k * layer.k * pr.t
        imgs += 1
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": done_f / spent / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "cpu_model": cpu_model, "host_cpus": os.cpu_count(),
            "kind": "oracle",
            "sample": f"{imgs} single-image passes (the workload has batch {batch}) through all "
                      f"{len(layers)} layer(s): fp64 direct convolution over the masked dense "
                      f"weight, {spent:.1f} s; rate counts the 1xN kernel's actual flops"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="c1", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle work")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a copy kernel of known size (for scaling byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the 1xN conv path here is single-GPU "
              "(multi-GPU sharding is a design note, not built); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration:
        copy_calibration(dev)
        return
    wl = WORKLOADS[args.workload]()
    batch = wl.batch
    odt = _TDT[wl.out_dtype]

    # Offline: generate, build masks, pack, copy to the device.
    prepared = []
    f_act = f_dense = b_alg = 0.0
    t_host = 0.0
    for layer in wl.layers:
        w, x = workloads.gen_layer(layer, batch, wl.dtype)
        t0 = time.perf_counter()
        packed = onexn.prepare_layer(w, layer.N, layer.p, layer.rearrange, dev)
        t_host += time.perf_counter() - t0
        fa, fd, bb = layer_work(layer, packed, batch, wl.dtype, wl.out_dtype)
        f_act, f_dense, b_alg = f_act + fa, f_dense + fd, b_alg + bb
        xd = x.to(dev)
        Ho = layer.Ho
        copies = max(1, math.ceil(ROTATE_BYTES / max(bb, 1)))
        copies = min(copies, 16)
        xs = [xd] + [xd.clone() for _ in range(copies - 1)]
        ys = [torch.empty((batch, layer.cout, Ho, Ho), dtype=odt, device=dev) for _ in range(copies)]
        prepared.append((layer, packed, xs, ys))
        del x, w

    stream = torch.cuda.current_stream(dev)
    # One pre-marshalled launch per (layer, buffer copy); a step issues one per layer.
    calls = []
    for layer, packed, xs, ys in prepared:
        calls.append([onexn.BoundConv(packed.P, packed.I, packed.D, packed.n, xs[r], ys[r],
                                      layer.stride, layer.pad, "nchw", stream.cuda_stream)
                      for r in range(len(xs))])

    def step(i):
        for per_layer in calls:
            per_layer[i % len(per_layer)]()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # Host-side launch cost per step, to size the stall that keeps the GPU from
    # draining the queue while the timed steps are being enqueued.
    h0 = time.perf_counter()
    for i in range(10):
        step(i)
    host_step_s = (time.perf_counter() - h0) / 10
    torch.cuda.synchronize()
    cyc0 = torch.cuda.Event(enable_timing=True)
    cyc1 = torch.cuda.Event(enable_timing=True)
    cyc0.record(stream)
    torch.cuda._sleep(1_000_000)
    cyc1.record(stream)
    torch.cuda.synchronize()
    cycles_per_ms = 1_000_000 / max(cyc0.elapsed_time(cyc1), 1e-3)
    stall_ms = 2.0 * host_step_s * 1e3 * (args.steps + 2) + 5.0

    # Timed region: the stream is held by a spin kernel while all K steps (and
    # an event pair around each) are enqueued, so the GPU then runs them back
    # to back and the events time the kernels, not the host.
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    t_all0 = torch.cuda.Event(enable_timing=True)
    t_all1 = torch.cuda.Event(enable_timing=True)
    stall_end = torch.cuda.Event()
    torch.cuda.synchronize()
    torch.cuda._sleep(int(stall_ms * cycles_per_ms))
    stall_end.record(stream)
    t_all0.record(stream)
    for i in range(args.steps):
        ev[i][0].record(stream)
        step(args.warmup + i)
        ev[i][1].record(stream)
    t_all1.record(stream)
    host_ahead = not stall_end.query()     # the stall was still running: no gaps
    torch.cuda.synchronize()
    total_ms = t_all0.elapsed_time(t_all1)
    per_step = sorted(a.elapsed_time(b) for a, b in ev)
    avg_step_ms = sum(per_step) / len(per_step)
    ms_per_step = total_ms / args.steps

    dtype = wl.dtype
    peak = PEAK_TFLOPS[dtype]
    t_compute = f_act / (peak * 1e12)
    t_hbm = b_alg / (PEAK_HBM_GBPS * 1e9)
    bound = "mfma" if t_compute >= t_hbm else "hbm"
    avg_s = avg_step_ms / 1e3
    if bound == "mfma":
        achieved, pk, unit = f_act / avg_s / 1e12, peak, "TFLOP/s"
    else:
        achieved, pk, unit = b_alg / avg_s / 1e9, PEAK_HBM_GBPS, "GB/s"
    traffic = measured_traffic(args.workload) if len(wl.layers) == 1 else None

    rec = {
        "metric": METRIC,
        "value": round(f_act * args.steps / (total_ms / 1e3) / 1e12, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "description": wl.description, "batch": batch,
                   "layers": len(wl.layers), "out_dtype": wl.out_dtype, "layout": "nchw"},
        "dense_equiv_tflops": round(f_dense * args.steps / (total_ms / 1e3) / 1e12, 3),
        "hbm_gbps": round(b_alg * args.steps / (total_ms / 1e3) / 1e9, 1),
        "kernel_us": {"mean": round(avg_step_ms * 1e3, 2), "p10": round(per_step[len(per_step) // 10] * 1e3, 2),
                      "p50": round(per_step[len(per_step) // 2] * 1e3, 2),
                      "p90": round(per_step[(9 * len(per_step)) // 10] * 1e3, 2)},
        "flops_actual_per_step": f_act,
        "flops_dense_per_step": f_dense,
        "bytes_alg_per_step": b_alg,
        "t_roof_us": round(max(t_compute, t_hbm) * 1e6, 2),
        "frac_of_roofline": round(max(t_compute, t_hbm) / avg_s, 4),
        "roofline": {"bound": bound, "achieved": round(achieved, 3), "peak": pk, "unit": unit,
                     "frac": round(achieved / pk, 4), "traffic": traffic},
        "host_prepare_s": round(t_host, 3),
        "host_enqueued_ahead": host_ahead,
        "host_launch_us_per_step": round(host_step_s * 1e6, 1),
    }
    if not args.no_cpu:
        rec["cpu_baseline"] = cpu_baseline(wl.layers, batch, wl, args.cpu_budget)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
