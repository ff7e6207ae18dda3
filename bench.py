"""Benchmark: one training step of the first-stage partition of 3D-ResAttNet
on one MI355X, through the librat3d C ABI.

Workload (the largest single-GPU configuration): stem (7^3 stride-2 conv to
32 channels, BN, ReLU) -> residual unit 32 -> 64 -> residual attention module
on 64 channels, on 48x56x48 maps; 4 micro-batches of 16 single-channel
volumes 96x112x96 (bf16 storage, fp32 accumulation); weight gradients summed
over the micro-batches in fp32, then one SGD step.  The gradient arriving at
the partition's output is a seeded N(0,1) tensor.  Volumes are synthetic
MRI-shaped fields (see paper_2104_05035_amd/synth.py).

Prints one JSON line.  value = algorithmic conv3d fwd+dgrad+wgrad TFLOP/s of
the whole step (conv flops per step / step time); volumes_per_s is the same
step counted in volumes.  An untimed breakdown pass brackets every tagged
launch with hipEvents (kernels_ms_per_step, conv_kernels = conv flops over
the conv kernels' own time, elementwise_hbm) and names the dominant kernel.
In the timed region only the dominant kernel's launches of the last step
carry event pairs (hipEvents recorded by the library on its launch stream):
they give the roofline's average launch duration.  After the timed region:
achievable-peak probes (a bf16 MFMA stream and a 16-byte streaming copy),
whose rates give the `frac_achievable` fields next to the datasheet
fractions, and the throughput of the full network's train step (8 volumes)
and of one attention module (4 x 64 x 48^3), each timed without events.
cpu_baseline times the oracle on a bounded sample.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
METRIC = "conv3d fwd+bwd TFLOP/s (% bf16 MFMA peak) and train volumes/sec, 1 MI355X"


def build_inputs(torch, R, synth, n, mb, vol, c):
    """Seeded parameters, volumes and upstream gradients, resident on the GPU."""
    rng_p, rng_x, rng_dy = synth.streams(4, 3)
    net = R.Net(R.NET_PARTITION1, n, 1, c, *vol, R.BF16, micro_batches=mb, lr=1e-4)
    layout = net.params()
    P0 = synth.init_params(rng_p, [(nm, shp) for nm, _, shp in layout])
    import numpy as np
    arena = np.concatenate([P0[nm].astype(np.float32).ravel() for nm, _, _ in layout])
    P = torch.from_numpy(arena).to("cuda:0")
    G = torch.zeros_like(P)
    ws = torch.empty(net.workspace_size, dtype=torch.uint8, device="cuda:0")
    net.rat3d_net_bind(P, G, ws, ws.numel())
    xs = synth.mri_volumes(rng_x, n * mb, vol)
    x = torch.from_numpy(xs).to(torch.bfloat16).to("cuda:0")
    so = tuple((v + 6 - 7) // 2 + 1 for v in vol)
    dys = []
    for _ in range(mb):  # one micro-batch at a time keeps host memory small
        a = rng_dy.standard_normal((n, c) + so, dtype=np.float32)
        dys.append(torch.from_numpy(a).to(torch.bfloat16).to("cuda:0"))
    dy = torch.cat(dys)
    return net, P, G, ws, x, dy


def cpu_baseline(volumes=2):
    """The oracle as it stands, on a bounded sample of the same workload: the
    partition's forward and backward for `volumes` volumes (same graph and
    shapes, BN statistics over those volumes), bf16 store points, float64
    arithmetic; about 15 s on 16 host cores."""
    import numpy as np
    from oracle import net as onet, ops
    from paper_2104_05035_amd import synth
    rng_p, rng_x, rng_dy = synth.streams(4, 3)
    L = onet.param_layout("partition1", 1, 64)
    P = {k: v.astype(np.float32).astype(np.float64) for k, v in synth.init_params(rng_p, L).items()}
    x = ops.round_bf16(synth.mri_volumes(rng_x, volumes, (96, 112, 96)))
    dy = ops.round_bf16(rng_dy.standard_normal((volumes, 64, 48, 56, 48), dtype=np.float32))
    t0 = time.perf_counter()
    onet.partition1_fwd_bwd(P, x, dy, bf16=True)
    dt = time.perf_counter() - t0
    flops = 8.522e12 / 16.0 * volumes  # conv flops of the volumes through the partition
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": ops.num_threads(),
            "kind": "oracle", "volumes_per_s": round(volumes / dt, 6), "seconds": round(dt, 2),
            "sample": "oracle forward+backward of the partition for %d volumes 96x112x96 "
                      "(%.3f TFLOP of conv work), float64 loops, bf16 store points"
                      % (volumes, flops / 1e12)}


def elementwise_hbm(tags, copy_gbs):
    """Achieved HBM bandwidth of the bandwidth-bound kernels: algorithmic bytes
    (each tensor a kernel must read or write, once) over their hipEvent time,
    overall and per kernel tag, as a fraction of the 8 TB/s peak and of the
    measured streaming-copy rate."""
    ew = [t for t in tags if t[3] == 0 and t[4] > 0]
    tot_b = sum(t[4] for t in ew)
    tot_ms = sum(t[2] for t in ew)
    if tot_ms <= 0:
        return None
    per = sorted(ew, key=lambda t: -t[2])[:10]
    ach = tot_b / (tot_ms * 1e-3) / 1e9
    return {"achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4),
            "frac_achievable": round(ach / copy_gbs, 4),
            "by_kernel": {t[0]: round(t[4] / (t[2] * 1e-3) / 1e9 / PEAK_HBM_GBS, 3)
                          for t in per}}


def achievable_peaks(torch, R, reps=5):
    """Measured ceilings (untimed, after the step): a pure bf16 MFMA stream
    (4 waves per SIMD, independent accumulators) and a 16-byte streaming copy
    of 1 GiB (four times the Infinity Cache); best of `reps`."""
    stream = torch.cuda.current_stream()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    blocks, iters = 4 * cus, 20000
    sink = torch.empty(blocks * 256, dtype=torch.float32, device="cuda:0")
    flops = R.rat3d_probe_mfma_flops(blocks, iters)
    nb = 1 << 30
    src = torch.ones(nb // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)

    def best(fn):
        fn()
        t = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            t.append(e0.elapsed_time(e1))
        return min(t)
    ms_m = best(lambda: R.rat3d_probe_mfma(blocks, iters, sink))
    ms_c = best(lambda: R.rat3d_probe_copy(src, dst, nb))
    del sink, src, dst
    torch.cuda.empty_cache()
    return {"mfma_tflops": round(flops / (ms_m * 1e-3) / 1e12, 1),
            "copy_gbs": round(2.0 * nb / (ms_c * 1e-3) / 1e9, 1),
            "probes": "bf16 MFMA 16x16x32 stream, %d workgroups x 4 waves x %d x 4 MFMA; "
                      "16-byte copy of 1 GiB; best of %d" % (blocks, iters, reps)}


def other_config(torch, R, synth, kind, steps, warmup):
    """Throughput of the other two bf16 workloads: the full network's train
    step (8 volumes 96x112x96, stem, three stages, head, SGD) and one
    attention module's forward + backward (4 x 64 x 48^3).  Conv flops per step
    from one profiled step; the timed steps carry no events."""
    import numpy as np
    stream = torch.cuda.current_stream()
    if kind == "resattnet":
        n, vol = 8, (96, 112, 96)
        net = R.Net(R.NET_RESATTNET, n, 1, 32, *vol, R.BF16, lr=1e-4)
    else:
        n, vol = 4, (48, 48, 48)
        net = R.Net(R.NET_ATTN, n, 64, 64, *vol, R.BF16)
    layout = net.params()
    rng_p, rng_x, rng_l = synth.streams(3 if kind == "resattnet" else 2, 3)
    P0 = synth.init_params(rng_p, [(nm, shp) for nm, _, shp in layout])
    arena = np.concatenate([P0[nm].astype(np.float32).ravel() for nm, _, _ in layout])
    P = torch.from_numpy(arena).to("cuda:0")
    G = torch.zeros_like(P)
    ws = torch.empty(net.workspace_size, dtype=torch.uint8, device="cuda:0")
    net.rat3d_net_bind(P, G, ws, ws.numel())
    if kind == "resattnet":
        x = torch.from_numpy(synth.mri_volumes(rng_x, n, vol)).to(torch.bfloat16).to("cuda:0")
        labels = torch.from_numpy(rng_l.integers(0, 2, n).astype(np.int32)).to("cuda:0")
        step = lambda: net.rat3d_train_step(x, labels, None, None)
    else:
        shp = (n, 64) + vol
        x = torch.from_numpy(rng_x.standard_normal(shp, dtype=np.float32)).to(torch.bfloat16)
        x = x.to("cuda:0")
        dy = torch.from_numpy(rng_l.standard_normal(shp, dtype=np.float32)).to(torch.bfloat16)
        dy = dy.to("cuda:0")
        y, dx = torch.empty_like(x), torch.empty_like(x)
        step = lambda: net.rat3d_block_fwd_bwd(x, dy, y, dx)
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    # the profiled step runs every kernel on one stream (events of concurrent
    # kernels would each count the shared time); the timed steps do not
    net.rat3d_net_set_overlap(0)
    R.rat3d_profile_reset()
    R.rat3d_profile_enable(1)
    step()
    torch.cuda.synchronize()
    R.rat3d_profile_enable(0)
    net.rat3d_net_set_overlap(1)
    tags = [R.rat3d_profile_read(i) for i in range(R.rat3d_profile_count())]
    conv_flops = sum(t[3] for t in tags if t[0].startswith("conv"))
    conv_ms = sum(t[2] for t in tags if t[3] > 0 or t[0] in ("wgrad_reduce", "bias_grad"))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    out = {"workload": ("full network train step: 8 volumes 96x112x96, stem 7^3 s2 -> 32, "
                        "stages 64/128/256 (RU + attention module), GAP, FC, CE, SGD"
                        if kind == "resattnet" else
                        "attention module forward + backward, 4 x 64 x 48^3"),
           "ms_per_step": round(ms, 3), "volumes_per_s": round(n / (ms * 1e-3), 1),
           "conv_tflop_per_step": round(conv_flops / 1e12, 4),
           "conv_tflops": round(conv_flops / (ms * 1e-3) / 1e12, 1),
           "conv_kernels_tflops": round(conv_flops / (conv_ms * 1e-3) / 1e12, 1),
           "launches_per_step": int(sum(t[1] for t in tags)), "steps": steps}
    del net, P, G, ws
    torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="skip the full-network and attention-module throughput lines")
    ap.add_argument("--workload", default="partition1",
                    choices=("partition1", "full_network", "attention_module"),
                    help="partition1 (default): the contract line; the others time only that "
                         "configuration (as the fields of the same name) and print its JSON, "
                         "e.g. for a profiler run of that workload alone")
    ap.add_argument("--calib-copy", action="store_true",
                    help="after the timed steps, copy 256 MiB device-to-device once (the "
                         "reference dispatch that scales rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library runs the per-device training step "
              "on a single MI355X and uses no collectives; run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2104_05035_amd import rat3d as R, synth
    R.lib()
    if args.workload != "partition1":
        kind = "resattnet" if args.workload == "full_network" else "attn"
        print(json.dumps({"workload_name": args.workload,
                          **other_config(torch, R, synth, kind, args.steps, args.warmup)}),
              flush=True)
        return
    n, mb, vol, c = 16, 4, (96, 112, 96), 64
    net, P, G, ws, x, dy = build_inputs(torch, R, synth, n, mb, vol, c)
    stream = torch.cuda.current_stream()

    # Warm-up (untimed) with every kernel on one stream: it loads every
    # kernel and touches every buffer; the schedule of the timed steps does
    # not depend on it.
    net.rat3d_net_set_overlap(0)
    for _ in range(args.warmup):
        net.rat3d_train_step(x, None, dy, None)
    torch.cuda.synchronize()

    # Breakdown pass (untimed): every tagged launch bracketed by hipEvents,
    # which gives the per-kernel table and names the dominant kernel.  It
    # runs the step with every kernel on one stream (the timed steps overlap
    # micro-batch k + 1's forward with micro-batch k's backward, where the
    # events of concurrent kernels would each count the shared time).
    bsteps = max(1, min(args.steps, 3))
    net.rat3d_net_set_overlap(0)
    R.rat3d_profile_reset()
    R.rat3d_profile_filter(None)
    R.rat3d_profile_enable(1)
    for _ in range(bsteps):
        net.rat3d_train_step(x, None, dy, None)
    torch.cuda.synchronize()
    R.rat3d_profile_enable(0)
    net.rat3d_net_set_overlap(1)
    tags = [R.rat3d_profile_read(i) for i in range(R.rat3d_profile_count())]
    dom_tag = max(tags, key=lambda t: t[2])[0]

    # Timed region: K steps.  Only the dominant kernel's launches of the last
    # step carry event pairs (an event pair costs ~10 us of gap; around each
    # of the ~650 launches of every step it would add its own cost to the
    # step time); they give its average launch duration for the roofline.
    # That step runs with micro-batches not overlapped, so the kernel's
    # launches have the GPU to themselves (overlapped, a launch also spans
    # the other micro-batch's concurrent kernels); it stays in ms_per_step.
    R.rat3d_profile_reset()
    R.rat3d_profile_filter(dom_tag)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        if i == args.steps - 1:
            net.rat3d_net_set_overlap(0)
            R.rat3d_profile_enable(1)
        net.rat3d_train_step(x, None, dy, None)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    R.rat3d_profile_enable(0)
    R.rat3d_profile_filter(None)
    net.rat3d_net_set_overlap(1)
    ms_step = ev0.elapsed_time(ev1) / args.steps
    dom = [R.rat3d_profile_read(i) for i in range(R.rat3d_profile_count())][0]
    assert dom[0] == dom_tag and dom[1] > 0

    conv_flops = sum(t[3] for t in tags if t[0].startswith("conv")) / bsteps
    per_launch_ms = dom[2] / dom[1]
    if dom[3] > 0:
        achieved = dom[3] / dom[1] / (per_launch_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 3), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 5),
                "traffic": None}
    else:
        achieved = dom[4] / dom[1] / (per_launch_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 3), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 5), "traffic": None}
    from paper_2104_05035_amd import profsum
    roof["traffic"] = profsum.lookup(dom[0])
    roof["kernel"] = dom[0]
    roof["avg_launch_us"] = round(per_launch_ms * 1e3, 3)
    roof["launches_per_step"] = dom[1]
    roof["timed_in"] = ("last step of the timed region, micro-batches not overlapped "
                        "(hipEvents on the launch stream)")
    del net, P, G, ws, x, dy
    torch.cuda.empty_cache()
    peaks = achievable_peaks(torch, R)
    if roof["bound"] == "mfma":
        roof["frac_achievable"] = round(achieved / peaks["mfma_tflops"], 5)
        roof["achievable_peak"] = peaks["mfma_tflops"]
    else:
        roof["frac_achievable"] = round(achieved / peaks["copy_gbs"], 5)
        roof["achievable_peak"] = peaks["copy_gbs"]

    if args.calib_copy:
        src = torch.empty(256 * 1024 * 1024, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    tflops = conv_flops / (ms_step * 1e-3) / 1e12
    vols = n * mb / (ms_step * 1e-3)
    kernels = sorted(tags, key=lambda t: -t[2])
    # conv kernels proper plus their split-K reductions and bias gradients
    conv_ms = sum(t[2] for t in tags
                  if t[3] > 0 or t[0] in ("wgrad_reduce", "bias_grad")) / bsteps
    conv_rate = conv_flops / (conv_ms * 1e-3) / 1e12 if conv_ms > 0 else 0.0
    out = {
        "metric": METRIC, "value": round(tflops, 3), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "partition1: stem 7^3 s2 1->32, RU 32->64, attention module 64 "
                               "on 48x56x48; 4 micro-batches x 16 volumes 96x112x96",
                   "micro_batches": mb, "volumes_per_micro_batch": n, "volume": list(vol),
                   "channels": c, "parallelism": "none (1 GPU)"},
        "volumes_per_s": round(vols, 3),
        "pct_bf16_mfma_peak": round(100.0 * tflops / PEAK_BF16_TFLOPS, 3),
        "conv_tflop_per_step": round(conv_flops / 1e12, 4),
        "conv_kernels": {"ms_per_step": round(conv_ms, 3), "tflops": round(conv_rate, 1),
                         "frac_bf16_peak": round(conv_rate / PEAK_BF16_TFLOPS, 4)},
        "wall_s_timed": round(wall, 3),
        "kernels_ms_per_step": {t[0]: round(t[2] / bsteps, 3) for t in kernels},
        "breakdown_steps": bsteps,
        "breakdown_schedule": "one stream (micro-batches not overlapped)",
        "timed_schedule": "steps 1..K-1 overlap micro-batch k+1's forward with micro-batch k's "
                          "backward; step K (the roofline's events) does not",
        "roofline": roof,
        "elementwise_hbm": elementwise_hbm(tags, peaks["copy_gbs"]),
        "achievable_peaks": peaks,
    }
    if not args.no_other_configs:
        out["full_network"] = other_config(torch, R, synth, "resattnet", args.steps, args.warmup)
        out["attention_module"] = other_config(torch, R, synth, "attn", args.steps, args.warmup)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
