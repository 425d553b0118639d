"""Benchmark of the pattern-sparse 3x3 convolution forward on one MI355X.

A step is one forward pass of the whole workload through the HIP path: for
the VGG-16 stack (default) the 13 pattern-sparse conv layers with fused ReLU
and the four 2x2 max-pools (fused into the conv launch they follow where
that is faster, as timed at start-up) on a 1x3x224x224 synthetic image; for
the other workloads every listed layer on its own resident input.  Weights are pruned
and packed on the GPU (projection, selection, packing) before timing.  The
step's launches are captured once in a HIP graph and the timed steps are its
replays (--no-graph times eager launches); per-layer times come from an eager
pass with HIP events.

Prints ONE JSON line: nonzero-MAC GFLOP/s of the step, ms/step, per-layer
ms, the roofline of the conv kernel (measured with HIP events on the stream
it runs on) and the CPU oracle as a baseline.  --details writes per-layer
comparisons with the dense comparators (our dense HIP conv, MIOpen through
torch) to a JSON file.
"""
import argparse
import json
import os
import sys
import time
from types import SimpleNamespace

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "nonzero-MAC GFLOP/s + ms/layer, pattern-sparse 3x3 conv fwd, batch 1 and 32"
PEAK_VALU_TFLOPS = 157.3     # MI355X fp32 vector peak (256 CU x 2.4 GHz x 256 flop/clk)
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="vgg16_224_b1_f32")
    ap.add_argument("--algo", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--details", default=None, help="write per-layer comparisons to this JSON file")
    ap.add_argument("--list", action="store_true")
    ap.add_argument("--no-graph", action="store_true",
                    help="time eager launches instead of replays of a captured HIP graph of the step")
    ap.add_argument("--fuse-pool", default="auto",
                    help="pooled layers whose pool runs inside the conv launch: auto (the faster form, "
                         "timed at start-up), all, none, or layer names separated by commas")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a 256 MiB device-to-device copy (reference for HBM counters)")
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
            self.layers.append(dict(lay=lay, w=w, prep=prep, x=x, y=y, pooled=pooled, fused=False))
            if wl.chained:
                x = pooled if pooled is not None else y
        torch.cuda.synchronize()

    def step(self, events=None):
        from paper_2003_06513_amd import binding as B
        for li, L in enumerate(self.layers):
            if events is not None:
                events[li][0].record()
            if L["fused"]:
                # conv, ReLU and the 2x2 max-pool in one launch
                B.conv3x3_fwd_pool2(L["prep"].layer, L["prep"].packed, L["x"], L["pooled"], relu=L["lay"].relu,
                                    algo=self.algo)
            elif L["lay"].stride != 1:
                B.conv3x3_fwd_strided(L["prep"].layer, L["prep"].packed, L["x"], L["y"], L["lay"].stride,
                                      relu=L["lay"].relu, algo=self.algo)
            else:
                B.conv3x3_fwd(L["prep"].layer, L["prep"].packed, L["x"], L["y"], relu=L["lay"].relu,
                              algo=self.algo)
            if events is not None:
                events[li][1].record()
            if L["pooled"] is not None and not L["fused"]:
                B.maxpool2x2(L["y"], L["pooled"])

    def choose_fusion(self, mode="auto", reps=20):
        """Per pooled layer, the fused conv + pool launch or the conv launch
        followed by the pool kernel: with mode "auto" the faster of the two,
        timed on this device; else "all", "none" or a list of layer names."""
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
                run = lambda: Net.step(SimpleNamespace(layers=one, algo=self.algo))
                for _ in range(3):
                    run()
                s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                s.record()
                for _ in range(reps):
                    run()
                e.record()
                torch.cuda.synchronize()
                t[fused] = s.elapsed_time(e)
            L["fused"] = t[True] < t[False]
            L["fusion_us"] = [round(t[False] * 1e3 / reps, 2), round(t[True] * 1e3 / reps, 2)]

    def output(self):
        L = self.layers[-1]
        return L["pooled"] if L["pooled"] is not None else L["y"]

    def nz_flops(self, li):
        lay = self.layers[li]["lay"]
        oh, ow = lay.out_hw
        return 8.0 * self.wl.batch * oh * ow * lay.keep


def cpu_baseline(net, budget_s=10.0):
    """The oracle's sparse conv, as it stands, on the host cores."""
    import oracle
    oracle.build(force=False)
    # bounded sample: image 0 of the batch through the layers in order,
    # repeated whole passes until about budget_s of CPU work
    host = [(L["lay"], L["prep"].packed.to_host(), L["x"][:1].cpu().numpy()) for L in net.layers]
    flops, secs, passes, layers = 0.0, 0.0, 0, 0
    while secs < budget_s:
        for lay, packed, x in host:
            t0 = time.perf_counter()
            if lay.stride == 1:
                oracle.conv_sparse(x, packed, net.masks, lay.cout, relu=lay.relu)
            else:
                oracle.conv_sparse_strided(x, packed, net.masks, lay.cout, lay.stride, relu=lay.relu)
            secs += time.perf_counter() - t0
            flops += 8.0 * lay.out_hw[0] * lay.out_hw[1] * lay.keep
            layers += 1
            if secs >= budget_s:
                break
        passes += 1
    return {"value": round(flops / secs / 1e9, 3), "unit": "GFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": "fp64-accumulating oracle sparse conv on image 0 of the batch: %d layer runs "
                      "(%d passes over the %d layers), %.2f nonzero-MAC GFLOP in %.2f s"
                      % (layers, passes, len(host), flops / 1e9, secs)}


def profiled_traffic(kernel_src, fused):
    """HBM bytes per conv launch from the committed rocprofv3 counter summary
    of this workload, or None when the kernel source or the set of layers
    with the pool fused into the conv launch differ from the profiled ones."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "k_conv_stream_vgg16_224_b1_f32.md")
    if not os.path.exists(path):
        return None
    with open(kernel_src, "rb") as f:
        digest = hashlib.sha256(f.read()).hexdigest()
    fields = {}
    with open(path) as f:
        for line in f:
            if line.startswith("- ") and ": " in line:
                k, v = line[2:].strip().split(": ", 1)
                fields[k.strip("`")] = v.strip().strip("`")
    if fields.get("conv_stream.hip sha256") != digest:
        return None
    if fields.get("pool fused into") != (",".join(fused) or "none"):
        return None
    try:
        return int(fields["hbm bytes per conv launch"])
    except (KeyError, ValueError):
        return None


def compare_dense(net, reps=20):
    """Per-layer times of the dense comparators on the masked weights."""
    import torch
    from paper_2003_06513_amd import binding as B
    out = []
    for L in net.layers:
        lay, prep = L["lay"], L["prep"]
        if lay.stride != 1:
            continue                     # the dense comparators are stride 1
        wd = torch.empty(L["w"].shape, dtype=net.tdt, device="cuda")
        B.unpack_dense(prep.layer, prep.packed, wd)
        yd = torch.empty_like(L["y"])

        def timeit(fn):
            for _ in range(3):
                fn()
            s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            s.record()
            for _ in range(reps):
                fn()
            e.record()
            torch.cuda.synchronize()
            return s.elapsed_time(e) / reps

        t_sparse = timeit(lambda: B.conv3x3_fwd(prep.layer, prep.packed, L["x"], L["y"], relu=lay.relu))
        t_dense = timeit(lambda: B.dense3x3_fwd(L["x"], wd, yd, relu=lay.relu))
        t_miopen = timeit(lambda: torch.relu_(torch.nn.functional.conv2d(L["x"], wd, padding=1))
                          if lay.relu else torch.nn.functional.conv2d(L["x"], wd, padding=1))
        out.append(dict(layer=lay.name, cin=lay.cin, cout=lay.cout, h=lay.h, w=lay.w, keep=lay.keep,
                        sparse_ms=t_sparse, dense_hip_ms=t_dense, miopen_ms=t_miopen,
                        nz_gflops=8.0 * net.wl.batch * lay.h * lay.w * lay.keep / t_sparse / 1e6))
    return out


def main():
    args = parse()
    if args.list:
        from synthetic import inputs
        for wl in inputs.all_workloads():
            print(wl.name)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the pattern-sparse layer shards by batch with no "
              "exchange, so multi-GPU runs are not part of this build", file=sys.stderr)
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
    wl = find_workload(args.workload)
    net = Net(wl, args.algo)
    net.choose_fusion(args.fuse_pool)

    for _ in range(args.warmup):
        net.step()
    torch.cuda.synchronize()
    K = args.steps
    # eager steps with HIP events around every conv launch (on the stream the
    # launches use): per-layer times and the kernel's roofline
    ev = [[[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)]
           for _ in net.layers] for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(K):
        net.step(ev[k])
    torch.cuda.synchronize()
    ms_eager = (time.perf_counter() - t0) * 1e3 / K
    ms_step, graph = ms_eager, False
    if not args.no_graph:
        # the step's conv and pool launches captured once in a HIP graph
        # and replayed: the timed region is the replays alone
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
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        if not torch.equal(net.output(), eager_out):
            raise SystemExit("graph replay of the step differs from the eager step")
        t0 = time.perf_counter()
        for _ in range(K):
            g.replay()
        torch.cuda.synchronize()
        ms_step, graph = (time.perf_counter() - t0) * 1e3 / K, True
    layer_ms = [float(np.median([ev[k][li][0].elapsed_time(ev[k][li][1]) for k in range(K)]))
                for li in range(len(net.layers))]
    layer_mean_ms = [float(np.mean([ev[k][li][0].elapsed_time(ev[k][li][1]) for k in range(K)]))
                     for li in range(len(net.layers))]
    nz = [net.nz_flops(li) for li in range(len(net.layers))]
    total_nz = sum(nz)
    conv_ms = sum(layer_mean_ms)
    achieved_tf = total_nz / (conv_ms * 1e-3) / 1e12
    traffic = None
    if wl.name == "vgg16_224_b1_f32":
        traffic = profiled_traffic(os.path.join(ROOT, "paper_2003_06513_amd", "csrc", "conv_stream.hip"),
                                   [L["lay"].name for L in net.layers if L["fused"]])
    roof = {"bound": "alu", "achieved": round(achieved_tf, 3), "peak": PEAK_VALU_TFLOPS,
            "unit": "TFLOP/s", "frac": round(achieved_tf / PEAK_VALU_TFLOPS, 4), "traffic": traffic,
            "kernel": ("k_conv_wide (224- and 112-wide layers) + k_conv_stream (the others)"
                   if wl.name == "vgg16_224_b1_f32" else
                   "k_conv_stream / k_conv_wide" + (" + k_conv_simple (stride-2 layers)"
                                                    if any(L["lay"].stride != 1 for L in net.layers) else "")),
            "per_launch": "8*N*H*W*keep nonzero-MAC flops averaged over the %d conv launches of a step, "
                          "/ their mean duration (HIP events on the launch stream)" % len(net.layers),
            "avg_launch_us": round(conv_ms * 1e3 / len(net.layers), 3)}
    line = {
        "metric": METRIC, "value": round(total_nz / (ms_step * 1e-3) / 1e9, 2), "unit": "GFLOP/s",
        "n_gpus": 1, "steps": K, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": wl.name, "batch": wl.batch, "layers": len(wl.layers), "m": wl.m,
                   "stack": "conv+relu, 2x2 max-pool after conv2/4/7/10" if wl.chained else "independent layers",
                   "pool_fused_into": [L["lay"].name for L in net.layers if L["fused"]]},
        "pool_fusion_us_unfused_fused": {L["lay"].name: L["fusion_us"] for L in net.layers if "fusion_us" in L},
        "step_launch": "hip graph replay" if graph else "eager",
        "ms_per_step_eager": round(ms_eager, 4),
        "ms_per_layer": {L["lay"].name: round(t, 4) for L, t in zip(net.layers, layer_ms)},
        "conv_ms_per_step": round(conv_ms, 4),
        "roofline": roof,
    }
    details = {}
    if args.details:
        details["dense_compare"] = compare_dense(net)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(net)
    print(json.dumps(line), flush=True)
    if args.details:
        details["line"] = line
        with open(args.details, "w") as f:
            json.dump(details, f, indent=1)


if __name__ == "__main__":
    main()
