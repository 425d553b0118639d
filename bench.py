"""Benchmark of the pattern-sparse 3x3 convolution forward on one MI355X.

A step is one forward pass of a whole workload through the HIP path: for the
VGG-16 stack (the headline workload) the 13 pattern-sparse conv layers with
fused ReLU and the four 2x2 max-pools (fused into the conv launch they follow
where that is faster, as timed at start-up) on a 1x3x224x224 synthetic
image; for the other workloads every listed layer on its own resident input.
Weights are pruned and packed on the GPU (projection, selection, packing)
before timing.  The timed steps are eager launches on one stream; the same
run also captures the step once in a HIP graph, checks a replay against the
eager output and times the replays (--launch graph reports those instead;
on this path graph replay measures 2-5 % slower than eager launches, whose
host-side submission stays ahead of the GPU).

The same run measures the other workloads the metric is quoted on (by
default the 16 ResNet-50 3x3 layers in fp16 at batch 1 and 32).  For every
workload it reports, per layer, the median, p10 and p90 of 30 samples of 5
back-to-back launches timed with HIP events on the launch stream (after 10
warm-up launches), the nonzero-MAC GFLOP/s, the roofline fraction, and the
time of MIOpen's dense convolution of the same masked weights (torch
conv2d) with the speedup over it; and the oracle's fp32-accumulating conv
loop timed on the host cores, on all threads and on one.

It also times the retraining kernels of each workload (dx through the
transposed packing and the masked weight gradient) and one iteration of the
data-free ADMM pruning of a layer (Algorithm 1) on the two ADMM workloads.

Prints ONE JSON line: the headline workload's nonzero-MAC GFLOP/s and
ms/step, its conv kernels' roofline, the CPU baseline, a "configs" object
with the per-workload results and an "admm" object.
"""
import argparse
import hashlib
import glob
import json
import os
import sys
import time
from types import SimpleNamespace

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "nonzero-MAC GFLOP/s + ms/layer, pattern-sparse 3x3 conv fwd, batch 1 and 32"
# MI355X published fp32 vector peak (256 CUs x 2.4 GHz).  The kernels issue
# non-packed v_fmac_f32 (the library is compiled with packed fp32 disabled); the measured
# ceilings in the bench line give the rate that instruction reaches here.
PEAK_VALU_TFLOPS = 157.3
PEAK_MFMA_F32_TFLOPS = 157.3   # MI355X published dense fp32 matrix peak (the same figure)
PEAK_HBM_GBS = 8000.0
DEFAULT_CONFIGS = "vgg16_224_b1_f32,resnet50_3x3_b1_f16,resnet50_3x3_b32_f16"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="vgg16_224_b1_f32", help="the headline workload")
    ap.add_argument("--configs", default=DEFAULT_CONFIGS,
                    help="workloads measured in the same run (comma-separated); 'all' for every one")
    ap.add_argument("--algo", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-miopen", action="store_true")
    ap.add_argument("--details", default=None, help="also write the per-layer results to this JSON file")
    ap.add_argument("--jsonl", default=None,
                    help="also write one JSON line per (workload, layer) to this file")
    ap.add_argument("--no-ceilings", dest="ceilings", action="store_false",
                    help="skip the measured ceilings (FMA probe, HBM copy, launch latency)")
    ap.add_argument("--list", action="store_true")
    ap.add_argument("--launch", choices=("eager", "graph"), default="eager",
                    help="the timed steps: eager launches, or replays of a captured HIP graph of the step "
                         "(both are timed and reported)")
    ap.add_argument("--fuse-pool", default="auto",
                    help="pooled layers whose pool runs inside the conv launch: auto (the faster form, "
                         "timed at start-up), all, none, or layer names separated by commas")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a 256 MiB device-to-device copy (reference for HBM counters)")
    ap.add_argument("--no-backward", dest="backward", action="store_false",
                    help="skip the retraining kernels (dx through the transposed packing, masked dW)")
    ap.add_argument("--no-admm", dest="admm", action="store_false",
                    help="skip the ADMM pruning iteration timings")
    ap.add_argument("--profile-only", action="store_true",
                    help="only the headline workload's warm-up and timed eager steps (for profiler runs)")
    ap.add_argument("--profile-part", choices=("forward", "backward", "admm"), default="forward",
                    help="with --profile-only: the forward step, the retraining kernels (dx and masked dW of "
                         "every stride-1 layer) or ADMM iterations of the ADMM workload --workload names")
    return ap.parse_args()


def find_workload(name):
    from synthetic import inputs
    for wl in inputs.all_workloads():
        if wl.name == name:
            return wl
    raise SystemExit("unknown workload %s; --list shows the names" % name)


class Net:
    """Prepared layers + resident activations of one workload."""

    def __init__(self, wl, algo):
        import torch
        from paper_2003_06513_amd import binding as B
        from synthetic import inputs
        self.wl, self.algo = wl, algo
        tdt = torch.float16 if wl.dtype == "f16" else torch.float32
        self.tdt = tdt
        allk = inputs.all_kernels(wl)
        self.masks = B.select_library(allk, wl.m)
        self.layers = []
        n = wl.batch
        x = torch.from_numpy(inputs.layer_input(wl, 0)).cuda()
        for li, lay in enumerate(wl.layers):
            w = torch.from_numpy(inputs.layer_weights(wl, li)).cuda()
            prep = B.prepare(w, self.masks, lay.keep)
            if not wl.chained and li > 0:
                x = torch.from_numpy(inputs.layer_input(wl, li)).cuda()
            y = torch.empty((n, lay.cout) + lay.out_hw, dtype=tdt, device="cuda")
            pooled = None
            if lay.pool_after:
                pooled = torch.empty((n, lay.cout, lay.h // 2, lay.w // 2), dtype=tdt, device="cuda")
            cfg = B.conv3x3_config(prep.layer, prep.layer.dtype, n, lay.h, lay.w, False, lay.stride, algo)
            self.layers.append(dict(lay=lay, w=w, prep=prep, x=x, y=y, pooled=pooled, fused=False, cfg=cfg))
            if wl.chained:
                x = pooled if pooled is not None else y
        torch.cuda.synchronize()

    def launch(self, L):
        from paper_2003_06513_amd import binding as B
        if L["fused"]:
            # conv, ReLU and the 2x2 max-pool in one launch
            B.conv3x3_fwd_pool2(L["prep"].layer, L["prep"].packed, L["x"], L["pooled"], relu=L["lay"].relu,
                                algo=self.algo)
        elif L["lay"].stride != 1:
            B.conv3x3_fwd_strided(L["prep"].layer, L["prep"].packed, L["x"], L["y"], L["lay"].stride,
                                  relu=L["lay"].relu, algo=self.algo)
        else:
            B.conv3x3_fwd(L["prep"].layer, L["prep"].packed, L["x"], L["y"], relu=L["lay"].relu, algo=self.algo)

    def step(self):
        from paper_2003_06513_amd import binding as B
        for L in self.layers:
            self.launch(L)
            if L["pooled"] is not None and not L["fused"]:
                B.maxpool2x2(L["y"], L["pooled"])

    def choose_fusion(self, mode="auto", reps=20):
        """Per pooled layer, the fused conv + pool launch or the conv launch
        followed by the pool kernel: with mode "auto" the fused launch unless
        the separate pair times more than 3 % faster on this device (the fused
        launch saves a launch and a round trip of the unpooled output; the
        margin keeps near-ties from flipping between runs); else "all",
        "none" or a list of layer names."""
        import torch
        names = [n for n in mode.split(",") if n] if mode not in ("auto", "all", "none") else []
        for L in self.layers:
            L["fused"] = False
            if L["pooled"] is None:
                continue
            if mode != "auto":
                L["fused"] = mode == "all" or L["lay"].name in names
                continue
            t = {}
            for fused in (False, True):
                L["fused"] = fused
                one = [dict(L)]
                run = lambda: Net.step(SimpleNamespace(layers=one, algo=self.algo, launch=self.launch))
                for _ in range(3):
                    run()
                s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                s.record()
                for _ in range(reps):
                    run()
                e.record()
                torch.cuda.synchronize()
                t[fused] = s.elapsed_time(e)
            L["fused"] = t[True] <= 1.03 * t[False]
            L["fusion_us"] = [round(t[False] * 1e3 / reps, 2), round(t[True] * 1e3 / reps, 2)]

    def output(self):
        L = self.layers[-1]
        return L["pooled"] if L["pooled"] is not None else L["y"]

    def nz_flops(self, li):
        lay = self.layers[li]["lay"]
        oh, ow = lay.out_hw
        return 8.0 * self.wl.batch * oh * ow * lay.keep


def time_launches(fn, warm=10, samples=30, reps=5):
    """Median, p10, p90 and mean in ms of one launch of fn: ``samples``
    samples of ``reps`` back-to-back launches bracketed by HIP events on the
    current stream (the one the launches use), after ``warm`` launches."""
    import torch
    for _ in range(warm):
        fn()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(samples)]
    for s, e in ev:
        s.record()
        for _ in range(reps):
            fn()
        e.record()
    torch.cuda.synchronize()
    t = np.array([s.elapsed_time(e) / reps for s, e in ev])
    return float(np.median(t)), float(np.percentile(t, 10)), float(np.percentile(t, 90)), float(t.mean())


def time_step(net, steps, warmup):
    """ms per step, eager and as replays of a HIP graph of the step (whose
    output is checked against the eager step's): ``warmup`` untimed steps,
    then ``steps`` timed ones between two device synchronisations."""
    import torch
    for _ in range(warmup):
        net.step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        net.step()
    torch.cuda.synchronize()
    ms_eager = (time.perf_counter() - t0) * 1e3 / steps
    eager_out = net.output().clone()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        net.step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        net.step()
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    if not torch.equal(net.output(), eager_out):
        raise SystemExit("graph replay of the step differs from the eager step")
    t0 = time.perf_counter()
    for _ in range(steps):
        g.replay()
    torch.cuda.synchronize()
    return ms_eager, (time.perf_counter() - t0) * 1e3 / steps


def layer_table(net, miopen):
    """Per layer: the sparse conv launch as the step runs it, and MIOpen's
    dense conv of the same masked weights (torch conv2d, + ReLU where the
    layer has it; stride as the layer's)."""
    import torch
    from paper_2003_06513_amd import binding as B
    rows = []
    for li, L in enumerate(net.layers):
        lay, prep = L["lay"], L["prep"]
        med, p10, p90, mean = time_launches(lambda: net.launch(L))
        nz = net.nz_flops(li)
        row = dict(layer=lay.name, cin=lay.cin, cout=lay.cout, h=lay.h, w=lay.w, stride=lay.stride, keep=lay.keep,
                   fused_pool=bool(L["fused"]), ms=round(med, 5), p10=round(p10, 5), p90=round(p90, 5),
                   mean_ms=round(mean, 5), nz_gflops=round(nz / (med * 1e-3) / 1e9, 1),
                   kernel=["stream", "wide", "simple", "stride2", "rows"][L["cfg"]["kernel"]] + ("-staged" if L["cfg"]["staged"] else ""),
                   R=L["cfg"]["rows_per_lane"], KS=L["cfg"]["shares"])
        if "fusion_us" in L:
            row["pool_separate_fused_us"] = L["fusion_us"]
        if miopen:
            wd = torch.empty(L["w"].shape, dtype=net.tdt, device="cuda")
            B.unpack_dense(prep.layer, prep.packed, wd)
            torch.cuda.synchronize()
            st = lay.stride

            def dense():
                y = torch.nn.functional.conv2d(L["x"], wd, padding=1, stride=st)
                return torch.relu_(y) if lay.relu else y
            if L["fused"]:
                def dense_pool():
                    return torch.nn.functional.max_pool2d(dense(), 2)
                dmed = time_launches(dense_pool, warm=3)[0]
            else:
                dmed = time_launches(dense, warm=3)[0]
            row["miopen_ms"] = round(dmed, 5)
            row["speedup_vs_miopen"] = round(dmed / med, 3)
        rows.append(row)
    return rows


def cpu_baseline(net, budget_s=8.0):
    """The oracle's conv loop built with fp32 accumulation (-O3, x86-64-v3: AVX2 + FMA)
    on the host cores: one full step of the workload (every layer, every
    image, on the inputs the GPU layers received) on all threads, median of
    up to 5 runs within budget_s; and on 1 thread the first image's pass,
    median of up to 3 runs."""
    import oracle
    oracle.build(force=False)
    host = [(L["lay"], L["prep"].packed.to_host(), L["x"].cpu().numpy()) for L in net.layers]
    flops = sum(8.0 * x.shape[0] * lay.out_hw[0] * lay.out_hw[1] * lay.keep for lay, _, x in host)
    flops1 = sum(8.0 * lay.out_hw[0] * lay.out_hw[1] * lay.keep for lay, _, _ in host)

    def run(images):
        t0 = time.perf_counter()
        for lay, packed, x in host:
            oracle.conv_sparse_f32acc(x[:images], packed, net.masks, lay.cout, lay.stride, relu=lay.relu)
        return time.perf_counter() - t0

    ncores = os.cpu_count() or 1
    oracle.bench_set_num_threads(ncores)
    cores = oracle.bench_num_threads()
    ts, spent = [], 0.0
    while len(ts) < 5 and (spent < budget_s or len(ts) < 1):
        ts.append(run(net.wl.batch))
        spent += ts[-1]
    oracle.bench_set_num_threads(1)
    t1, spent = [], 0.0
    while len(t1) < 3 and (spent < budget_s or len(t1) < 1):
        t1.append(run(1))
        spent += t1[-1]
    oracle.bench_set_num_threads(ncores)
    t, tt = float(np.median(ts)), float(np.median(t1))
    return {"value": round(flops / t / 1e9, 3), "unit": "GFLOP/s", "cores": cores, "kind": "oracle",
            "sample": "fp32-accumulating build of the oracle's sparse conv loop (-O3 x86-64-v3, OpenMP over "
                      "(image, filter)); all %d threads: one full step (%d layers x %d images, %.3f nonzero-MAC "
                      "GFLOP), median of %d runs = %.2f ms; 1 thread: image 0 of every layer, median of %d runs"
                      % (cores, len(host), net.wl.batch, flops / 1e9, len(ts), t * 1e3, len(t1)),
            "ms_per_step": round(t * 1e3, 3),
            "value_1thread": round(flops1 / tt / 1e9, 3)}


def backward_calls(net):
    """One retraining pass over the stride-1 layers of a prepared workload
    (dx through the transposed packing, then dv and db), as a callable."""
    import torch
    from paper_2003_06513_amd import binding as B
    calls = []
    for L in net.layers:
        lay = L["lay"]
        if lay.stride != 1:
            continue
        pt = B.prepare_transposed(L["prep"], L["w"])
        dy = torch.randn((net.wl.batch, lay.cout, lay.h, lay.w), device="cuda").to(net.tdt)
        dx = torch.empty((net.wl.batch, lay.cin, lay.h, lay.w), dtype=net.tdt, device="cuda")
        dv = torch.empty(4 * lay.keep, dtype=torch.float32, device="cuda")
        db = torch.empty(lay.cout, dtype=torch.float32, device="cuda")
        ws = B.conv3x3_bwd_weight_workspace(L["prep"].layer, L["prep"].layer.dtype, net.wl.batch, lay.h, lay.w)
        calls.append((pt, L, dy, dx, dv, db, ws))

    def run():
        for pt, L, dy, dx, dv, db, ws in calls:
            B.conv3x3_fwd(pt.layer, pt.packed, dy, dx)
            B.conv3x3_bwd_weight(L["prep"].layer, L["prep"].packed, L["x"], dy, dv, db, ws=ws)
    return run


def measure_backward(net):
    """Retraining kernels (Sec. 3.3) on every stride-1 layer of a prepared
    workload: dx through the transposed packing (the tuned forward kernels)
    and the masked weight gradient; flops 8*N*H*W*keep each, as the
    forward."""
    import torch
    from paper_2003_06513_amd import binding as B
    rows, tot = [], {"dx": [0.0, 0.0], "dw": [0.0, 0.0]}
    for li, L in enumerate(net.layers):
        lay = L["lay"]
        if lay.stride != 1:
            continue
        pt = B.prepare_transposed(L["prep"], L["w"])
        dy = torch.randn((net.wl.batch, lay.cout, lay.h, lay.w), device="cuda").to(net.tdt)
        dx = torch.empty((net.wl.batch, lay.cin, lay.h, lay.w), dtype=net.tdt, device="cuda")
        dv = torch.empty(4 * lay.keep, dtype=torch.float32, device="cuda")
        db = torch.empty(lay.cout, dtype=torch.float32, device="cuda")
        ws = B.conv3x3_bwd_weight_workspace(L["prep"].layer, L["prep"].layer.dtype, net.wl.batch, lay.h, lay.w)
        torch.cuda.synchronize()
        t_dx = time_launches(lambda: B.conv3x3_fwd(pt.layer, pt.packed, dy, dx))[0]
        t_dw = time_launches(lambda: B.conv3x3_bwd_weight(L["prep"].layer, L["prep"].packed, L["x"], dy, dv, db,
                                                          ws=ws))[0]
        fl = 8.0 * net.wl.batch * lay.h * lay.w * lay.keep
        tot["dx"][0] += fl
        tot["dx"][1] += t_dx
        tot["dw"][0] += fl
        tot["dw"][1] += t_dw
        rows.append(dict(layer=lay.name, dx_ms=round(t_dx, 5), dw_ms=round(t_dw, 5),
                         dx_gflops=round(fl / (t_dx * 1e-3) / 1e9, 1), dw_gflops=round(fl / (t_dw * 1e-3) / 1e9, 1)))
    out = {"layers": rows}
    for k, (fl, ms) in tot.items():
        if ms > 0:
            out[k + "_ms_per_step"] = round(ms, 4)
            out[k + "_tflops"] = round(fl / (ms * 1e-3) / 1e12, 3)
            out[k + "_roofline_frac"] = round(fl / (ms * 1e-3) / 1e12 / PEAK_VALU_TFLOPS, 4)
    return out


def measure_admm(wl, iters=10, parts=True):
    """One ADMM iteration of one layer (Algorithm 1): the pre-trained target,
    the current layer, the loss gradient, the dense weight gradient, the SGD
    step, the projection (project + select) and the dual step, on a new
    synthetic batch per iteration (batches drawn and uploaded beforehand)."""
    import torch
    from paper_2003_06513_amd import binding as B
    w0 = torch.from_numpy(wl.weights()).cuda()
    b0 = torch.from_numpy(wl.bias()).cuda()
    masks = B.select_library(wl.weights(), wl.m)
    st = B.AdmmLayer(w0, b0, masks, wl.layer.keep, lr=wl.lr)
    xs = [torch.from_numpy(wl.batch_input(k)).cuda() for k in range(1, 3)]
    shape = (wl.batch, wl.layer.cout, wl.layer.h, wl.layer.w)
    tgt = torch.empty(shape, dtype=torch.float32, device="cuda")
    scale = 1.0 / tgt.numel()

    def one(k):
        x = xs[k % 2]
        st.target(x, out=tgt)
        st.iteration(x, tgt, B.admm_rho(k + 1), scale)
    for k in range(3):
        one(k)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for k in range(iters):
        one(k)
    e.record()
    torch.cuda.synchronize()
    ms_iter = s.elapsed_time(e) / iters
    if not parts:
        return {"ms_per_iteration": round(ms_iter, 4)}
    x = xs[0]
    z = st._bufs["z"]
    dense_fl = 18.0 * wl.batch * wl.layer.h * wl.layer.w * wl.layer.cin * wl.layer.cout
    parts = {
        "dense_fwd": time_launches(lambda: B.dense3x3_fwd(x, st.w, z, bias=st.b), warm=3, samples=10, reps=2)[0],
        "residual": time_launches(lambda: B.admm_residual(z, tgt, scale, st._bufs["g"], st.loss, st.ws_res),
                                  warm=3, samples=10, reps=2)[0],
        "dense_wgrad": time_launches(lambda: B.dense3x3_bwd_weight(x, st._bufs["g"], st.dw, st.db,
                                                                   ws=st._bufs.get("wgrad_ws")),
                                     warm=3, samples=10, reps=2)[0],
    }
    return {"batch": wl.batch, "layer": "%d->%d %dx%d" % (wl.layer.cin, wl.layer.cout, wl.layer.h, wl.layer.w),
            "keep": wl.layer.keep, "m": wl.m, "ms_per_iteration": round(ms_iter, 4),
            "loss_after": float(st.loss.item()),
            "ms": {k: round(v, 4) for k, v in parts.items()},
            "dense_fwd_tflops": round(dense_fl / (parts["dense_fwd"] * 1e-3) / 1e12, 3),
            "dense_wgrad_tflops": round(dense_fl / (parts["dense_wgrad"] * 1e-3) / 1e12, 3),
            "dense_fwd_roofline_frac": round(dense_fl / (parts["dense_fwd"] * 1e-3) / 1e12 / PEAK_MFMA_F32_TFLOPS, 4),
            "dense_wgrad_roofline_frac": round(dense_fl / (parts["dense_wgrad"] * 1e-3) / 1e12 / PEAK_MFMA_F32_TFLOPS, 4)}


def conv_sources_digest():
    """sha256 over the conv kernel sources (a committed counter summary is
    valid only for the kernels it measured)."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2003_06513_amd", "csrc")
    for f in sorted(glob.glob(os.path.join(csrc, "conv_*.h")) + glob.glob(os.path.join(csrc, "conv_*.hip"))):
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode() + b"\0" + fh.read())
    return h.hexdigest()


def profiled_traffic(workload, fused):
    """HBM bytes per conv launch from the committed rocprofv3 counter summary
    of this workload, or None when the conv sources or the set of layers with
    the pool fused into the conv launch differ from the profiled ones."""
    paths = glob.glob(os.path.join(ROOT, "profiles", "*_%s.md" % workload))
    for path in paths:
        fields = {}
        with open(path) as f:
            for line in f:
                if line.startswith("- ") and ": " in line:
                    k, v = line[2:].strip().split(": ", 1)
                    fields[k.strip("`")] = v.strip().strip("`")
        if "hbm bytes per conv launch" not in fields:
            continue
        if fields.get("conv sources sha256") != conv_sources_digest():
            return None
        if fields.get("pool fused into") not in (None, ",".join(fused) or "none"):
            return None
        try:
            return int(fields["hbm bytes per conv launch"])
        except ValueError:
            return None
    return None


def measure(wl, args, headline):
    """Everything reported for one workload."""
    net = Net(wl, args.algo)
    net.choose_fusion(args.fuse_pool)
    ms_eager, ms_graph = time_step(net, args.steps, args.warmup)
    ms_step = ms_graph if args.launch == "graph" else ms_eager
    rows = layer_table(net, not args.no_miopen)
    nz = [net.nz_flops(li) for li in range(len(net.layers))]
    conv_ms = sum(r["mean_ms"] for r in rows)
    achieved = sum(nz) / (conv_ms * 1e-3) / 1e12
    res = {
        "batch": wl.batch, "dtype": wl.dtype, "m": wl.m, "layers": len(wl.layers),
        "ms_per_step": round(ms_step, 4), "ms_per_step_eager": round(ms_eager, 4),
        "ms_per_step_graph": round(ms_graph, 4),
        "step_launch": "hip graph replay" if args.launch == "graph" else "eager, one stream",
        "nz_gflops": round(sum(nz) / (ms_step * 1e-3) / 1e9, 2),
        "conv_ms_per_step": round(conv_ms, 4),
        "roofline_frac": round(achieved / PEAK_VALU_TFLOPS, 4),
        "pool_fused_into": [L["lay"].name for L in net.layers if L["fused"]],
        "ms_per_layer": {r["layer"]: r["ms"] for r in rows},
        "layer_detail": rows,
    }
    if not args.no_miopen:
        dense_ms = sum(r["miopen_ms"] for r in rows)
        sparse_ms = sum(r["ms"] for r in rows)
        res["miopen_ms_per_step"] = round(dense_ms, 4)
        res["speedup_vs_miopen"] = round(dense_ms / sparse_ms, 3)
    if args.backward:
        res["backward"] = measure_backward(net)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(net)
    roof = {"bound": "alu", "achieved": round(achieved, 3), "peak": PEAK_VALU_TFLOPS, "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_VALU_TFLOPS, 4),
            "traffic": profiled_traffic(wl.name, res["pool_fused_into"]),
            "kernel": ", ".join(sorted({r["kernel"] for r in rows})),
            "per_launch": "8*N*H*W*keep nonzero-MAC flops averaged over the %d conv launches of a step, / their "
                          "mean duration (HIP events around back-to-back launches on the launch stream); peak: "
                          "MI355X published fp32 vector rate" % len(rows),
            "avg_launch_us": round(conv_ms * 1e3 / len(rows), 3)}
    return net, res, roof


def measure_ceilings():
    """Measured ceilings beside the published ones: the fp32 FMA rate of the
    vector ALUs as the library issues it (psc_probe_fma: v_fmac_f32, packed
    fp32 disabled), the fp32 matrix-core rate of the dense kernels'
    instruction (psc_probe_mfma), the HBM bandwidth of a 1 GiB device copy (read + write
    bytes), and the launch latency of a tiny library kernel, eager and as a
    HIP graph replay."""
    import torch
    from paper_2003_06513_amd import binding as B
    blocks, iters = 4096, 20000
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    for _ in range(2):
        B.probe_fma(blocks, iters, out)
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 5
    s.record()
    for _ in range(reps):
        B.probe_fma(blocks, iters, out)
    e.record()
    torch.cuda.synchronize()
    fma_tflops = 2.0 * 8 * iters * blocks * 256 * reps / (s.elapsed_time(e) * 1e-3) / 1e12
    mblocks, miters = 4096, 4000
    for _ in range(2):
        B.probe_mfma(mblocks, miters, out)
    s.record()
    for _ in range(reps):
        B.probe_mfma(mblocks, miters, out)
    e.record()
    torch.cuda.synchronize()
    mfma_tflops = 32768.0 * miters * mblocks * reps / (s.elapsed_time(e) * 1e-3) / 1e12
    a = torch.ones(256 << 20, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    s.record()
    for _ in range(reps):
        b.copy_(a)
    e.record()
    torch.cuda.synchronize()
    copy_gbs = 2.0 * a.numel() * 4 * reps / (s.elapsed_time(e) * 1e-3) / 1e9
    del a, b
    x = torch.zeros((1, 1, 2, 2), dtype=torch.float32, device="cuda")
    y = torch.empty((1, 1, 1, 1), dtype=torch.float32, device="cuda")
    n = 200
    for _ in range(10):
        B.maxpool2x2(x, y)
    s.record()
    for _ in range(n):
        B.maxpool2x2(x, y)
    e.record()
    torch.cuda.synchronize()
    eager_us = s.elapsed_time(e) * 1e3 / n
    g = torch.cuda.CUDAGraph()
    st = torch.cuda.Stream()
    st.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(st):
        with torch.cuda.graph(g, stream=st):
            for _ in range(n):
                B.maxpool2x2(x, y, stream=st)
    torch.cuda.current_stream().wait_stream(st)
    g.replay()
    torch.cuda.synchronize()
    s.record()
    g.replay()
    e.record()
    torch.cuda.synchronize()
    graph_us = s.elapsed_time(e) * 1e3 / n
    return {"valu_fp32_fma_tflops": round(fma_tflops, 2),
            "valu_fp32_fma_frac_of_peak": round(fma_tflops / PEAK_VALU_TFLOPS, 3),
            "mfma_fp32_tflops": round(mfma_tflops, 2),
            "mfma_fp32_frac_of_peak": round(mfma_tflops / PEAK_MFMA_F32_TFLOPS, 3),
            "hbm_copy_gbs": round(copy_gbs, 1), "hbm_copy_frac_of_8000": round(copy_gbs / 8000.0, 3),
            "launch_us_eager": round(eager_us, 2), "launch_us_graph": round(graph_us, 2),
            "how": "psc_probe_fma 4096x256 lanes x 8 chains x 20000 v_fmac_f32; psc_probe_mfma 4096x4 waves x "
                   "4 chains x 4000 v_mfma_f32_16x16x4_f32; torch copy_ of 1 GiB fp32 "
                   "(2 GiB moved); 200 back-to-back psc_maxpool2x2 launches on a 2x2 image, eager and in one "
                   "HIP graph"}


def write_jsonl(path, results):
    with open(path, "w") as f:
        for name, res in results.items():
            bw = {r["layer"]: r for r in res.get("backward", {}).get("layers", [])}
            for r in res["layer_detail"]:
                row = {"workload": name, "batch": res["batch"], "dtype": res["dtype"]}
                row.update(r)
                if r["layer"] in bw:
                    row.update({k: v for k, v in bw[r["layer"]].items() if k != "layer"})
                f.write(json.dumps(row) + "\n")


def main():
    args = parse()
    if args.list:
        from synthetic import inputs
        for wl in inputs.all_workloads():
            print(wl.name)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the pattern-sparse layer shards by batch with no "
              "exchange, and multi-GPU runs are not implemented", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2003_06513_amd import binding as B
    torch.cuda.set_device(0)
    if args.copy_calibration:
        a = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": a.numel() * 4, "copy_bytes_written": a.numel() * 4,
                          "launches": 5}))
        return
    B.lib()
    if args.profile_only and args.profile_part == "admm":
        from synthetic import inputs
        found = [w for w in inputs.admm_workloads() if w.name == args.workload]
        if not found:
            raise SystemExit("unknown ADMM workload %s; admm workloads: %s"
                             % (args.workload, ", ".join(w.name for w in inputs.admm_workloads())))
        measure_admm(found[0], iters=args.steps, parts=False)
        print(json.dumps({"admm_workload": found[0].name, "steps": args.steps}), flush=True)
        return
    head = find_workload(args.workload)
    if args.profile_only and args.profile_part == "backward":
        net = Net(head, args.algo)
        net.choose_fusion("none")
        run = backward_calls(net)
        for _ in range(args.warmup + args.steps):
            run()
        torch.cuda.synchronize()
        print(json.dumps({"workload": head.name, "part": "backward", "steps": args.steps,
                          "warmup": args.warmup}), flush=True)
        return
    if args.profile_only:
        net = Net(head, args.algo)
        net.choose_fusion(args.fuse_pool)
        for _ in range(args.warmup + args.steps):
            net.step()
        torch.cuda.synchronize()
        print(json.dumps({"workload": head.name, "steps": args.steps, "warmup": args.warmup,
                          "pool_fused_into": [L["lay"].name for L in net.layers if L["fused"]]}), flush=True)
        return
    if args.configs == "all":
        from synthetic import inputs
        names = [wl.name for wl in inputs.all_workloads()]
    else:
        names = [n for n in args.configs.split(",") if n]
    if head.name not in names:
        names.insert(0, head.name)
    results, roofs = {}, {}
    for name in names:
        print("[bench] %s" % name, file=sys.stderr, flush=True)
        _, res, roof = measure(find_workload(name), args, name == head.name)
        results[name] = res
        roofs[name] = roof
    hr = results[head.name]
    line = {
        "metric": METRIC, "value": hr["nz_gflops"], "unit": "GFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": hr["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": head.dtype, "data": "synthetic",
        "config": {"workload": head.name, "batch": head.batch, "layers": len(head.layers), "m": head.m,
                   "stack": "conv+relu, 2x2 max-pool after conv2/4/7/10" if head.chained else "independent layers",
                   "pool_fused_into": hr["pool_fused_into"]},
        "step_launch": hr["step_launch"], "ms_per_step_eager": hr["ms_per_step_eager"],
        "ms_per_step_graph": hr["ms_per_step_graph"],
        "ms_per_layer": hr["ms_per_layer"],
        "roofline": roofs[head.name],
    }
    if "cpu_baseline" in hr:
        line["cpu_baseline"] = hr["cpu_baseline"]
    if args.ceilings:
        print("[bench] ceilings", file=sys.stderr, flush=True)
        line["ceilings"] = measure_ceilings()
        meas = line["ceilings"]["valu_fp32_fma_tflops"]
        line["roofline"]["measured_fma_tflops"] = meas
        line["roofline"]["frac_of_measured_fma"] = round(line["roofline"]["achieved"] / meas, 4)
    line["configs"] = {}
    for name, res in results.items():
        c = {k: v for k, v in res.items() if k not in ("layer_detail", "cpu_baseline", "backward")}
        if "backward" in res:
            c["backward"] = {k: v for k, v in res["backward"].items() if k != "layers"}
        c["roofline"] = {k: roofs[name][k] for k in ("achieved", "peak", "frac", "traffic")}
        if "cpu_baseline" in res:
            c["cpu_gflops_all_cores"] = res["cpu_baseline"]["value"]
            c["cpu_gflops_1thread"] = res["cpu_baseline"]["value_1thread"]
            c["cpu_cores"] = res["cpu_baseline"]["cores"]
        c["layers_detail"] = [{k: r[k] for k in ("layer", "ms", "p10", "p90", "nz_gflops", "kernel", "R", "KS")
                               + (("miopen_ms", "speedup_vs_miopen") if "miopen_ms" in r else ())}
                              for r in res["layer_detail"]]
        line["configs"][name] = c
    if args.admm:
        from synthetic import inputs
        line["admm"] = {}
        for wl in inputs.admm_workloads():
            print("[bench] %s" % wl.name, file=sys.stderr, flush=True)
            line["admm"][wl.name] = measure_admm(wl)
    print(json.dumps(line), flush=True)
    if args.details:
        with open(args.details, "w") as f:
            json.dump({"line": line, "configs": results}, f, indent=1)
    if args.jsonl:
        write_jsonl(args.jsonl, results)


if __name__ == "__main__":
    main()
