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
the conv kernels' own time, elementwise_hbm) and names the dominant kernel;
in the timed region only that kernel's launches are bracketed.  The roofline object is for the kernel with the most
time, timed with hipEvents recorded on its own launch stream by the library
during the timed region.  cpu_baseline times the oracle on a bounded sample.
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


def elementwise_hbm(tags):
    """Achieved HBM bandwidth of the bandwidth-bound kernels: algorithmic bytes
    (each tensor a kernel must read or write, once) over their hipEvent time,
    overall and per kernel tag, as a fraction of the 8 TB/s peak."""
    ew = [t for t in tags if t[3] == 0 and t[4] > 0]
    tot_b = sum(t[4] for t in ew)
    tot_ms = sum(t[2] for t in ew)
    if tot_ms <= 0:
        return None
    per = sorted(ew, key=lambda t: -t[2])[:10]
    return {"achieved": round(tot_b / (tot_ms * 1e-3) / 1e9, 1), "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": round(tot_b / (tot_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "by_kernel": {t[0]: round(t[4] / (t[2] * 1e-3) / 1e9 / PEAK_HBM_GBS, 3)
                          for t in per}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy", action="store_true",
                    help="after the timed steps, copy 256 MiB device-to-device once (the "
                         "reference dispatch that scales rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build runs the per-device training step "
              "on a single MI355X and uses no collectives; run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2104_05035_amd import rat3d as R, synth
    R.lib()
    n, mb, vol, c = 16, 4, (96, 112, 96), 64
    net, P, G, ws, x, dy = build_inputs(torch, R, synth, n, mb, vol, c)
    stream = torch.cuda.current_stream()

    for _ in range(args.warmup):
        net.rat3d_train_step(x, None, dy, None)
    torch.cuda.synchronize()

    # Breakdown pass (untimed): every tagged launch bracketed by hipEvents,
    # which gives the per-kernel table and names the dominant kernel.
    bsteps = max(1, min(args.steps, 3))
    R.rat3d_profile_reset()
    R.rat3d_profile_filter(None)
    R.rat3d_profile_enable(1)
    for _ in range(bsteps):
        net.rat3d_train_step(x, None, dy, None)
    torch.cuda.synchronize()
    R.rat3d_profile_enable(0)
    tags = [R.rat3d_profile_read(i) for i in range(R.rat3d_profile_count())]
    dom_tag = max(tags, key=lambda t: t[2])[0]

    # Timed region: only the dominant kernel's launches carry event pairs (an
    # event pair around each of the ~650 launches of a step would add its own
    # cost to the step time).
    R.rat3d_profile_reset()
    R.rat3d_profile_filter(dom_tag)
    R.rat3d_profile_enable(1)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        net.rat3d_train_step(x, None, dy, None)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    R.rat3d_profile_enable(0)
    R.rat3d_profile_filter(None)
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
    roof["launches_per_step"] = dom[1] // args.steps
    roof["timed_in"] = "timed region (hipEvents on the launch stream)"

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
        "roofline": roof,
        "elementwise_hbm": elementwise_hbm(tags),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
