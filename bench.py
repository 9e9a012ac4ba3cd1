"""Benchmark of the 1xN-pruned convolution forward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c2] [--no-cpu]

A step is one forward pass of the workload's pruned layer(s) (Eq. 8 on the
GPU) over one batch of synthetic input already resident in HBM.  The default
workload is every convolution of a ResNet-50-shaped network at batch 64 in
fp32 (N = 32, p = 0.5, the 7x7 stem dense).  Mask building and packing are
the offline part of the method (done once per layer before deployment) and
run before the timed region.  To keep timed steps from hitting the 256 MB
Infinity Cache with the previous step's data, the input and output buffers
rotate over enough copies to exceed 512 MB.

Before anything is timed, every layer's output is checked against the oracle
on at least 10^4 sampled outputs (random ones plus one in every tile of
pixels and col-group); a miss exits with status 3 and prints no result.

Prints one JSON line.  value = actual TFLOP/s (2 * pixels * N * kh * kw * t
per layer, summed) over the timed steps; the dense-equivalent rate and the
HBM rate are reported beside it.  The roofline fraction is the sum over
layers of each layer's roofline time, max(F_act / peak, B_alg / 8 TB/s),
divided by the measured step time; per-layer rows give each layer's share.
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
DEFAULT_WORKLOAD = "c2"
PARITY_SAMPLES = 10000
PAPER_CPU_CONTEXT = ("the paper's only latency figure: 1xN (N = 4) saves 56.04 ms of MobileNet-V2 "
                     "inference against weight pruning on an Arm Cortex-A7 (Zeropi board, "
                     "TVM/Ansor); a network latency difference on another machine, not a target")

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
for _N in (4, 32):
    for _lay in ("rows", "cols"):
        WORKLOADS[f"fc_n{_N}_{_lay}"] = (lambda N=_N, lay=_lay: workloads.fc_resnet50(N, lay))
WORKLOADS["c1_nhwc"] = lambda: workloads.nhwc(workloads.config1())
for _N in (16, 32):
    WORKLOADS[f"c3_n{_N}_p50_nhwc"] = (lambda N=_N: workloads.nhwc(workloads.config3(N, 0.5)))

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
    """HBM bytes per step of the workload from the committed rocprofv3 counter
    summary (FETCH_SIZE and WRITE_SIZE in KiB, summed over the step's
    dispatches, each scaled by the factor the same counter shows for a copy
    kernel of known size), or None when there is none, or when any source
    file the kernels are built from (listed in the record) has changed since."""
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


def epilogue_params(layer, li):
    """Seeded per-channel parameters of a folded batch norm for layer ``li``
    (scale in [0.5, 1.5), bias ~ N(0, 0.25^2), channel order of the layer's
    output), as host float32 tensors."""
    g = torch.Generator().manual_seed(10_000 + li)
    scale = 0.5 + torch.rand(layer.cout, generator=g)
    bias = 0.25 * torch.randn(layer.cout, generator=g)
    return scale, bias


def parity_gate(prepared, wl, fused=False):
    """Each layer's output (from one launch of the same call the timed steps
    make) against the oracle at sampled outputs (with the oracle's epilogue
    when the layers carry a folded batch norm and ReLU).  Returns per-layer
    records; exits with status 3 on the first layer over the bar."""
    import oracle
    bar = 2e-2 if wl.out_dtype == "bf16" else 1e-5
    recs = []
    for li, (layer, packed, xs, ys, w_cpu, x_cpu, call0) in enumerate(prepared):
        call0()
        torch.cuda.synchronize()
        y = ys[0]
        if wl.fc_layout == "cols":        # [n][batch] -> [batch][n]
            y = y.t().contiguous()
        if wl.layout == "nhwc":           # [batch][Ho][Wo][n] -> [batch][n][Ho][Wo]
            y = y.permute(0, 3, 1, 2).contiguous()
        y = y.reshape(x_cpu.shape[0], layer.cout, layer.Ho, layer.Ho)
        idx = workloads.sample_outputs(tuple(y.shape), layer.N, PARITY_SAMPLES, seed=li)
        got = y.reshape(-1)[torch.from_numpy(idx).to(y.device)].double().cpu().numpy()
        pr = oracle.prune(w_cpu.double().numpy(), layer.N, layer.p, layer.rearrange)
        ref = oracle.conv2d_at(x_cpu.double().numpy(), pr.wbar, idx, (layer.stride,) * 2,
                               (layer.pad,) * 2)
        if fused:
            # Each sample as a channel of its own: act(scale[o] * v + bias[o]).
            o = (idx // (layer.Ho * layer.Ho)) % layer.cout
            sc, bi = epilogue_params(layer, li)
            ref = oracle.epilogue(ref.reshape(1, -1, 1), sc.double().numpy()[o],
                                  bi.double().numpy()[o], "relu").reshape(-1)
        den = float(abs(ref).max()) if ref.size else 0.0
        num = float(abs(got - ref).max()) if ref.size else 0.0
        err = num / den if den > 0 else (0.0 if num == 0 else float("inf"))
        ok = packed.t == pr.t and err <= bar and bool(torch.isfinite(torch.from_numpy(got)).all())
        recs.append({"layer": layer.name, "samples": int(idx.size), "rel_err": err, "ok": ok})
        if not ok:
            print(json.dumps({"parity": "FAIL", "workload": wl.name, "layer": layer.name,
                              "t": packed.t, "t_oracle": pr.t, "rel_err": err, "bar": bar,
                              "samples": int(idx.size)}), flush=True)
            sys.exit(3)
    return recs


def cpu_rate(lw, budget_s):
    """Oracle flops (the 1xN kernel's actual flops) per second over single-image
    passes through all layers until ``budget_s`` seconds are spent."""
    import oracle
    done_f, spent, imgs = 0.0, 0.0, 0
    while spent < budget_s:
        for layer, pr, x in lw:
            t0 = time.perf_counter()
            oracle.conv2d(x, pr.wbar, (layer.stride,) * 2, (layer.pad,) * 2)
            spent += time.perf_counter() - t0
            done_f += 2.0 * layer.Ho * layer.Ho * layer.N * layer.k * layer.k * pr.t
            if spent >= budget_s:
                break
        imgs += 1
    return done_f / spent / 1e12, spent, imgs


def cpu_baseline(layers, batch, wl, budget_s, single_budget_s):
    """The oracle (direct 7-loop over the masked dense weight, fp64) on the host
    cores, over a bounded sample: single images through the workload's layers,
    cycling over the layers until the time budget is spent; first on all the
    threads OpenMP takes, then on one thread."""
    import oracle
    lw = []
    for layer in layers:
        w, x = workloads.gen_layer(layer, 1, wl.dtype)
        pr = oracle.prune(w.double().numpy(), layer.N, layer.p, layer.rearrange)
        lw.append((layer, pr, x.double().numpy()))
    threads = oracle.num_threads()
    rate, spent, imgs = cpu_rate(lw, budget_s)
    oracle.set_num_threads(1)
    rate1, spent1, imgs1 = cpu_rate(lw, single_budget_s)
    oracle.set_num_threads(threads)
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": rate, "unit": "TFLOP/s", "cores": threads,
            "cpu_model": cpu_model, "host_cpus": os.cpu_count(),
            "kind": "oracle",
            "sample": f"{imgs} single-image passes (the workload has batch {batch}) over the "
                      f"workload's {len(layers)} layer(s) in order: fp64 direct convolution over "
                      f"the masked dense weight, {spent:.1f} s; rate counts the 1xN kernel's "
                      f"actual flops",
            "single_thread": {"value": rate1, "unit": "TFLOP/s", "cores": 1,
                              "sample": f"{imgs1} single-image passes, {spent1:.1f} s"},
            "paper_context": PAPER_CPU_CONTEXT}


def mask_bench(wl, dev, reps):
    """Times onexn_build_mask_dev (GPU mask building: filter norms, ranks, block
    scores, top-(1-p) selection) on every layer of a workload against the host
    library's onexn_build_mask, after checking that both agree bit for bit."""
    stream = torch.cuda.current_stream(dev)
    rows, t_gpu, t_host, b_alg = [], 0.0, 0.0, 0.0
    for layer in wl.layers:
        w, _ = workloads.gen_layer(layer, 1, wl.dtype)
        wd = w.to(dev)
        ws = torch.empty(max(onexn.mask_workspace_bytes(*w.shape[:2], layer.N), 8), dtype=torch.uint8,
                         device=dev)
        h0 = time.perf_counter()
        perm_h, mask_h, t_h = onexn.build_mask(w, layer.N, layer.p, layer.rearrange)
        th = time.perf_counter() - h0
        perm_d, mask_d, t_d = onexn.build_mask_dev(wd, layer.N, layer.p, layer.rearrange, ws)
        torch.cuda.synchronize()
        if not (t_d == t_h and torch.equal(perm_d.cpu(), perm_h) and torch.equal(mask_d.cpu(), mask_h)):
            print(json.dumps({"parity": "FAIL", "layer": layer.name}), flush=True)
            sys.exit(3)
        for _ in range(3):
            onexn.build_mask_dev(wd, layer.N, layer.p, layer.rearrange, ws)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            onexn.build_mask_dev(wd, layer.N, layer.p, layer.rearrange, ws)
        e1.record(stream)
        torch.cuda.synchronize()
        tg = e0.elapsed_time(e1) / reps / 1e3
        # Algorithmic bytes: W once for the block scores (once more for the
        # filter norms), the scores written and read by the selection, the mask.
        K = layer.cin * -(-layer.cout // layer.N)
        wb = w.numel() * w.element_size()
        bb = wb * (2 if layer.rearrange else 1) + 16 * K + K + 4 * layer.cout
        rows.append({"layer": layer.name, "n": layer.cout, "m": layer.cin, "k": layer.k, "N": layer.N,
                     "blocks": K, "gpu_us": round(tg * 1e6, 2), "host_us": round(th * 1e6, 1),
                     "mb_alg": round(bb / 1e6, 3)})
        t_gpu, t_host, b_alg = t_gpu + tg, t_host + th, b_alg + bb
    t_roof = b_alg / (PEAK_HBM_GBPS * 1e9)
    print(json.dumps({
        "metric": "1xN mask building on the GPU (rearrangement, block l1 scores, top-(1-p)): "
                  "time per workload, bit-exact with the host",
        "value": round(t_gpu * 1e6, 2), "unit": "us", "higher_is_better": False, "n_gpus": 1,
        "config": {"workload": wl.name, "layers": len(wl.layers)},
        "host_us": round(t_host * 1e6, 1), "speedup_vs_host": round(t_host / t_gpu, 2),
        "roofline": {"bound": "hbm", "achieved": round(b_alg / t_gpu / 1e9, 1), "peak": PEAK_HBM_GBPS,
                     "unit": "GB/s", "frac": round(t_roof / t_gpu, 4), "traffic": None},
        "per_layer": rows}), flush=True)


def backward_bench(wl, dev, reps):
    """Times one backward pass (onexn_conv2d_bwd_data and onexn_conv2d_bwd_weight
    on every layer) with HIP events, after checking each layer's gradients on
    the first image against the oracle (every entry of the timed launch's dX
    there, and of dD over that image alone).  Each of the
    two gradients does the forward's actual flops (2 * pixels * N * kh * kw * t)."""
    import oracle
    stream = torch.cuda.current_stream(dev)
    rows, t_sum, f_sum, troof = [], 0.0, 0.0, 0.0
    peak = PEAK_TFLOPS[wl.dtype]
    for li, layer in enumerate(wl.layers):
        w, x = workloads.gen_layer(layer, wl.batch, wl.dtype)
        packed = onexn.prepare_layer(w, layer.N, layer.p, layer.rearrange, dev)
        gen = torch.Generator().manual_seed(layer.seed + 7)
        dy = torch.randn((wl.batch, layer.cout, layer.Ho, layer.Ho), generator=gen).to(_TDT[wl.dtype])
        xd, dyd = x.to(dev), dy.to(dev)
        kk = (layer.k, layer.k)

        def run():
            dx = onexn.conv2d_bwd_data(packed.P, packed.I, packed.D, layer.cout, layer.cin, dyd,
                                       (layer.H, layer.H), layer.stride, layer.pad)
            dD = onexn.conv2d_bwd_weight(packed.P, packed.I, layer.cout, layer.N, kk, xd, dyd,
                                         layer.stride, layer.pad)
            return dx, dD
        dx, dD = run()
        torch.cuda.synchronize()
        # Parity before timing, against the oracle on the first image: every
        # entry of that image's dX from the timed launch (images are
        # independent), and every dD entry of a launch on that image alone.
        pr = oracle.prune(w.double().numpy(), layer.N, layer.p, layer.rearrange)
        x0, dy0 = x[:1].double().numpy(), dy[:1].double().numpy()
        ref_dx = oracle.conv2d_bwd_data(dy0, pr.wbar, (layer.H, layer.H), (layer.stride,) * 2,
                                        (layer.pad,) * 2)
        dx1 = dx[:1]
        dD1 = onexn.conv2d_bwd_weight(packed.P, packed.I, layer.cout, layer.N, kk, xd[:1].contiguous(),
                                      dyd[:1].contiguous(), layer.stride, layer.pad)
        torch.cuda.synchronize()
        dw = oracle.conv2d_bwd_weight(x0, dy0, pr.T, layer.N, kk, (layer.stride,) * 2, (layer.pad,) * 2)
        _, _, ref_dD = oracle.pack(dw, pr.T, layer.N)
        bar = 2e-2 if wl.dtype == "bf16" else 1e-5

        def rel(a, b):
            return float(abs(a - b).max() / max(abs(b).max(), 1e-300))
        e1 = rel(dx1.double().cpu().numpy(), ref_dx)
        e2 = rel(dD1.double().cpu().numpy(), ref_dD)
        if not (e1 <= bar and e2 <= bar):
            print(json.dumps({"parity": "FAIL", "layer": layer.name, "dx": e1, "dD": e2}), flush=True)
            sys.exit(3)
        errs = {"dx_rel_err": float(f"{e1:.3g}"), "dD_rel_err": float(f"{e2:.3g}")}
        for _ in range(2):
            run()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            run()
        e1.record(stream)
        torch.cuda.synchronize()
        tl = e0.elapsed_time(e1) / reps / 1e3
        fa = 2.0 * 2.0 * layer.out_pixels(wl.batch) * layer.N * layer.k * layer.k * packed.t
        rows.append({"layer": layer.name, "us": round(tl * 1e6, 1), "gflop": round(fa / 1e9, 3),
                     "tflops": round(fa / tl / 1e12, 3), **errs})
        t_sum, f_sum, troof = t_sum + tl, f_sum + fa, troof + fa / (peak * 1e12)
        del dx, dD, xd, dyd
    print(json.dumps({
        "metric": "1xN sparse conv backward (input and kept-block weight gradients): TFLOP/s",
        "value": round(f_sum / t_sum / 1e12, 3), "unit": "TFLOP/s", "higher_is_better": True, "n_gpus": 1,
        "dtype": wl.dtype, "config": {"workload": wl.name, "layers": len(wl.layers), "batch": wl.batch},
        "ms_per_pass": round(t_sum * 1e3, 3),
        "roofline": {"bound": "mfma", "achieved": round(f_sum / t_sum / 1e12, 3), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(troof / t_sum, 4), "traffic": None},
        "per_layer": rows}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle work")
    ap.add_argument("--cpu-single-budget", type=float, default=8.0,
                    help="seconds of single-threaded oracle work")
    ap.add_argument("--backward", action="store_true",
                    help="time the backward kernels on the workload's layers instead of the forward")
    ap.add_argument("--mask", action="store_true",
                    help="time the GPU mask building of the workload's layers instead of the conv")
    ap.add_argument("--fused", action="store_true",
                    help="every layer with a folded batch norm and ReLU in its store stage "
                         "(the fused entry point)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a copy kernel of known size (for scaling byte counters)")
    ap.add_argument("--tune", action="append", default=[], metavar="NAME=VALUE",
                    help="a kernel-choice override of the library (onexn_set_tuning), for A/B timing")
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
    for kv in args.tune:
        name, _, value = kv.partition("=")
        onexn.set_tuning(name, int(value))
    if args.copy_calibration:
        copy_calibration(dev)
        return
    wl = WORKLOADS[args.workload]()
    if args.mask:
        mask_bench(wl, dev, max(args.steps, 5))
        return
    if args.backward:
        backward_bench(wl, dev, max(min(args.steps, 10), 2))
        return
    batch = wl.batch
    odt = _TDT[wl.out_dtype]
    stream = torch.cuda.current_stream(dev)
    print(f"bench: {wl.name}: preparing {len(wl.layers)} layer(s)", file=sys.stderr, flush=True)

    # Offline: generate, build masks, pack, copy to the device.
    prepared = []
    rows = []
    f_act = f_dense = b_alg = 0.0
    t_host = 0.0
    peak = PEAK_TFLOPS[wl.dtype]
    for li, layer in enumerate(wl.layers):
        w, x = workloads.gen_layer(layer, batch, wl.dtype)
        t0 = time.perf_counter()
        packed = onexn.prepare_layer(w, layer.N, layer.p, layer.rearrange, dev)
        t_host += time.perf_counter() - t0
        fa, fd, bb = layer_work(layer, packed, batch, wl.dtype, wl.out_dtype)
        ep = {}
        if args.fused:
            sc, bi = epilogue_params(layer, li)
            ep = {"scale": sc.to(dev), "bias": bi.to(dev), "act": "relu"}
            bb += 2 * 4 * layer.cout
        f_act, f_dense, b_alg = f_act + fa, f_dense + fd, b_alg + bb
        t_c, t_m = fa / (peak * 1e12), bb / (PEAK_HBM_GBPS * 1e9)
        rows.append({"layer": layer.name, "k": layer.k, "stride": layer.stride, "cin": layer.cin,
                     "cout": layer.cout, "H": layer.H, "N": layer.N, "p": layer.p, "t": packed.t,
                     "gflop_act": fa / 1e9, "mb_alg": bb / 1e6,
                     "bound": "mfma" if t_c >= t_m else "hbm", "t_roof_us": max(t_c, t_m) * 1e6})
        Ho = layer.Ho
        copies = max(1, math.ceil(ROTATE_BYTES / max(bb, 1)))
        copies = min(copies, 16)
        if wl.fc_layout:
            # A fully connected layer: x [batch][m] ("rows") or [m][batch] ("cols").
            x2 = x.reshape(batch, layer.cin)
            xd = (x2 if wl.fc_layout == "rows" else x2.t().contiguous()).to(dev)
            yshape = (batch, layer.cout) if wl.fc_layout == "rows" else (layer.cout, batch)
        else:
            if wl.layout == "nhwc":
                xd = x.permute(0, 2, 3, 1).contiguous().to(dev)
                yshape = (batch, Ho, Ho, layer.cout)
            else:
                xd = x.to(dev)
                yshape = (batch, layer.cout, Ho, Ho)
        xs = [xd] + [xd.clone() for _ in range(copies - 1)]
        ys = [torch.empty(yshape, dtype=odt, device=dev) for _ in range(copies)]
        if wl.fc_layout:
            calls = [(lambda r=r: onexn.fc_fwd(packed.P, packed.I, packed.D, packed.n, xs[r],
                                               wl.fc_layout, odt, ys[r], stream.cuda_stream, **ep))
                     for r in range(copies)]
        else:
            calls = [onexn.BoundConv(packed.P, packed.I, packed.D, packed.n, xs[r], ys[r],
                                     layer.stride, layer.pad, wl.layout, stream.cuda_stream, **ep)
                     for r in range(copies)]
        prepared.append((layer, packed, xs, ys, w, x, calls))

    # Parity before timing: the same bound calls the timed steps issue.
    print("bench: parity gate against the oracle", file=sys.stderr, flush=True)
    gate = parity_gate([(l, pk, xs, ys, w, x, calls[0]) for l, pk, xs, ys, w, x, calls in prepared], wl,
                       args.fused)
    calls = [item[6] for item in prepared]
    del prepared    # the host copies of the inputs are no longer needed

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

    def stalled(n_events):
        """Holds the stream with a spin kernel long enough for the host to
        enqueue everything that follows, so the GPU runs it back to back."""
        stall_ms = 2.0 * host_step_s * 1e3 * (args.steps + 2) * n_events + 5.0
        torch.cuda.synchronize()
        torch.cuda._sleep(int(stall_ms * cycles_per_ms))
        end = torch.cuda.Event()
        end.record(stream)
        return end

    # Timed region: one event pair around each of the K back-to-back steps.
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    t_all0 = torch.cuda.Event(enable_timing=True)
    t_all1 = torch.cuda.Event(enable_timing=True)
    stall_end = stalled(1)
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

    # Per-layer times: the same steps again with an event between consecutive
    # launches (one chain per step, so the layer times add up to the step).
    per_layer_ms = [0.0] * len(calls)
    if len(calls) > 1:
        lsteps = max(5, min(args.steps, 20))
        chains = [[torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)]
                  for _ in range(lsteps)]
        stalled(2)
        for i in range(lsteps):
            chains[i][0].record(stream)
            for li, per_layer in enumerate(calls):
                per_layer[(args.warmup + i) % len(per_layer)]()
                chains[i][li + 1].record(stream)
        torch.cuda.synchronize()
        for ch in chains:
            for li in range(len(calls)):
                per_layer_ms[li] += ch[li].elapsed_time(ch[li + 1]) / lsteps
    else:
        per_layer_ms[0] = avg_step_ms
    for r, t_ms, g in zip(rows, per_layer_ms, gate):
        r["t_meas_us"] = round(t_ms * 1e3, 2)
        r["frac"] = round(r["t_roof_us"] / max(t_ms * 1e3, 1e-9), 4)
        r["t_roof_us"] = round(r["t_roof_us"], 2)
        r["gflop_act"] = round(r["gflop_act"], 4)
        r["mb_alg"] = round(r["mb_alg"], 3)
        r["parity_samples"] = g["samples"]
        r["parity_rel_err"] = float(f"{g['rel_err']:.3g}")

    dtype = wl.dtype
    t_roof_sum_us = sum(r["t_roof_us"] for r in rows)
    t_roof_mfma = sum(r["t_roof_us"] for r in rows if r["bound"] == "mfma")
    bound = "mfma" if t_roof_mfma >= t_roof_sum_us - t_roof_mfma else "hbm"
    frac = t_roof_sum_us / (avg_step_ms * 1e3)
    if bound == "mfma":
        pk, unit = peak, "TFLOP/s"
    else:
        pk, unit = PEAK_HBM_GBPS, "GB/s"
    traffic = None if args.fused else measured_traffic(args.workload)

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
                   "layers": len(wl.layers), "out_dtype": wl.out_dtype,
                   "layout": wl.fc_layout or wl.layout},
        "dense_equiv_tflops": round(f_dense * args.steps / (total_ms / 1e3) / 1e12, 3),
        "hbm_gbps": round(b_alg * args.steps / (total_ms / 1e3) / 1e9, 1),
        "kernel_us": {"mean": round(avg_step_ms * 1e3, 2), "p10": round(per_step[len(per_step) // 10] * 1e3, 2),
                      "p50": round(per_step[len(per_step) // 2] * 1e3, 2),
                      "p90": round(per_step[(9 * len(per_step)) // 10] * 1e3, 2)},
        "flops_actual_per_step": f_act,
        "flops_dense_per_step": f_dense,
        "bytes_alg_per_step": b_alg,
        "t_roof_us": round(t_roof_sum_us, 2),
        "frac_of_roofline": round(frac, 4),
        "roofline": {"bound": bound, "achieved": round(frac * pk, 3), "peak": pk, "unit": unit,
                     "frac": round(frac, 4), "traffic": traffic,
                     "definition": "sum over layers of max(F_act/peak, B_alg/8 TB/s) over the "
                                   "measured step time; achieved = frac x peak"},
        "parity": {"ok": True, "samples_min": min(g["samples"] for g in gate),
                   "rel_err_max": max(g["rel_err"] for g in gate),
                   "bar": 2e-2 if wl.out_dtype == "bf16" else 1e-5},
        "per_layer": rows,
        "host_prepare_s": round(t_host, 3),
        "host_enqueued_ahead": host_ahead,
        "host_launch_us_per_step": round(host_step_s * 1e6, 1),
    }
    if args.fused:
        rec["config"]["epilogue"] = "folded batch norm (per-channel scale and bias) + ReLU, fused"
    if args.tune:
        rec["config"]["tuning"] = args.tune
    if not args.no_cpu:
        print("bench: CPU oracle baseline", file=sys.stderr, flush=True)
        rec["cpu_baseline"] = cpu_baseline(wl.layers, batch, wl, args.cpu_budget,
                                           args.cpu_single_budget)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
