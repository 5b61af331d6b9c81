"""Benchmark: one integer training step (forward, softmax loss, backward,
update) of DeepLabv3-ResNet50 at output stride 16 on a batch of 8 synthetic
512x512 images with 150 classes, on one MI355X.  Other workload graphs
(--workload) are kept for comparison.

Prints ONE JSON line.  `value` is int8 conv throughput: valid-tap MACs x 2 of
the forward, backward-data and backward-weight convolutions per step, divided
by the whole step's wall time (inputs already in HBM); images/s is in
`config`, with the conv throughput over conv time (every conv entry point of
a few extra steps timed by its own events).  `roofline` reports the step's
largest kernel by time, the L1BN backward statistics pass, over every one of
its launches in the timed steps: HIP events that the library records around
each launch on its stream, algorithmic bytes of each launch's layer;
`cpu_baseline` is the CPU oracle timed on a bounded sample.
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "int8 conv TOPS fwd+bwd (% MFMA peak); train images/s DeepLabv3-R50 512²"
INT8_PEAK_TOPS = 5000.0      # MI355X dense int8 MFMA
HBM_PEAK_GBS = 8000.0

# HBM bytes per launch of a timed region, from two rocprofv3 --pmc runs of
# this script (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch, summed over the
# kernels of the region) scaled by what the same counters read for the plain
# copy kernel of --copy-kernel-mib (FETCH_SIZE x 2.0, WRITE_SIZE x 1.0 on
# MI355X).  Keyed by the timed region; `src` is the SHA-256 of the sources the
# region's kernels are built from when the counters were taken: a figure whose
# sources have changed since is reported as null.
TRAFFIC = {
    "bn_bwd_stats:*": dict(bytes=22813441, src="e5bd5c3515a0477a4b8c3f488d6a232dded47085990a998bf84f410cfdc82095",
                           profile="profiles/deeplabv3_r50_512_n8_l1bn_hbm_traffic.md"),
}
TRAFFIC_SRC = {"conv_fwd": ("conv.hip", "quant.hip", "iseg_common.h"),
               "bn_bwd_stats": ("bn.hip", "iseg_common.h")}

WORKLOAD_IDS = {"deeplabv3": 5, "aspp": 4, "resnet-stage": 3, "vgg16": 2, "single-conv": 1, "fcn8s": 6}


def conv_valid_macs(N, H, W, C, K, R, st, pad, dil):
    """Multiply-adds of a conv that touch real (non-padding) input."""
    P = (H + 2 * pad - dil * (R - 1) - 1) // st + 1
    rows = sum(1 for p in range(P) for r in range(R) if 0 <= p * st - pad + r * dil < H)
    Q = (W + 2 * pad - dil * (R - 1) - 1) // st + 1
    cols = sum(1 for q in range(Q) for s in range(R) if 0 <= q * st - pad + s * dil < W)
    return N * rows * cols * C * K


def workload_ops(wl, N=None):
    """Valid-tap int8 ops (2 per MAC) per training step, and per-conv detail:
    forward, backward-weight, and backward-data unless the conv reads the
    input image and no input gradient is wanted."""
    from paper_2011_14504_amd import synth
    wl = synth.scaled(wl, N)
    shapes = synth.node_shapes(wl)
    total, detail = 0, []
    for nd in synth.conv_nodes(wl):
        n, H, W, cin = shapes[nd["src"][0]]
        if nd.get("transposed"):
            # the conv it is the adjoint of (input of the node's output shape),
            # the geometry all three of its passes are launched on
            _, Ho, Wo, cout = shapes[nd["name"]]
            key = (n, Ho, Wo, cout, cin, nd["R"], nd["stride"], nd["pad"], nd["dil"])
        else:
            key = (n, H, W, cin, nd["cout"], nd["R"], nd["stride"], nd["pad"], nd["dil"])
        macs = conv_valid_macs(*key)
        passes = 3 if (nd["src"][0] != "input" or wl["input_grad"]) else 2
        total += 2 * macs * passes
        detail.append(dict(name=nd["name"], key=key, macs=macs))
    return total, detail


BN_FAMILIES = {
    # kernel family: (kernel id, algorithmic bytes per element of the layer's
    # output tensor).  stats1/stats2 read x; apply reads x, writes y; the
    # backward statistics read x and dy; the backward apply reads x, dy, writes dx
    "bn_fwd_stats1": ("ISEG_KID_BN_FWD_STATS1", 1), "bn_fwd_stats2": ("ISEG_KID_BN_FWD_STATS2", 1),
    "bn_fwd_apply": ("ISEG_KID_BN_FWD_APPLY", 2), "bn_bwd_stats": ("ISEG_KID_BN_BWD_STATS", 2),
    "bn_bwd_apply": ("ISEG_KID_BN_BWD_APPLY", 3),
}
CONV_FAMILIES = {"conv_fwd": "ISEG_KID_CONV_FWD", "conv_bwd_data": "ISEG_KID_CONV_BWD_DATA",
                 "conv_wgrad": "ISEG_KID_CONV_WGRAD"}


def timed_kernel_info(name, wl, detail):
    """Kernel family, layer key (None: every launch of the family) and the
    algorithmic work of a launch as a function of its layer key.  Conv
    families: valid-tap ops of the launch's layer.  L1BN families: bytes of
    the layer's tensor moved by the pass."""
    from paper_2011_14504_amd import iseg, synth
    kind, _, layer = name.partition(":")
    shapes = synth.node_shapes(wl)
    if kind in CONV_FAMILIES:
        by_key = {d["key"]: 2 * d["macs"] for d in detail}
        key = None if layer == "*" else next(d for d in detail if d["name"] == layer)["key"]
        what = "every launch" if key is None else f"{layer} (N,H,W,C,K,R,stride,pad,dil = {key})"
        return dict(kid=getattr(iseg, CONV_FAMILIES[kind]), key=key, bound="mfma",
                    work=lambda k: by_key[tuple(k)], name=f"{kind} entry point, {what}")
    kid, bpe = BN_FAMILIES[kind]
    if layer == "*":
        key, what = None, "every L1BN layer of the step"
    else:
        N, P, Q, K = shapes[layer]
        key, what = (N * P * Q, K), f"the L1BN after {layer} (M = {N * P * Q}, C = {K})"
    return dict(kid=getattr(iseg, kid), key=key, bound="hbm", work=lambda k: bpe * k[0] * k[1],
                name=f"{kind} kernel, {what}, {bpe} B per element")


def src_digest(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2011_14504_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(tk):
    """HBM bytes per launch of the timed region from the committed counter
    runs, or None when none were taken or its kernels have changed since."""
    t = TRAFFIC.get(tk)
    kind = tk.partition(":")[0]
    if not t or kind not in TRAFFIC_SRC or src_digest(TRAFFIC_SRC[kind]) != t["src"]:
        return None
    return t["bytes"]


def copy_kernel(mib):
    """The counter calibration: one plain elementwise kernel that reads and
    writes `mib` MiB each (float32 negation), run three times."""
    import torch
    n = mib * (1 << 20) // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda:0")
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    for _ in range(3):
        torch.neg(x, out=y)
    torch.cuda.synchronize()
    print(json.dumps({"copy_kernel_bytes_read": n * 4, "copy_kernel_bytes_written": n * 4}))


def cpu_baseline(wl, sample_hw, widths=None):
    """The oracle's whole training step on one image at sample_hw x sample_hw,
    timed on the host cores; scaled to the benchmark's unit by the ratio of
    valid-tap conv ops."""
    from oracle import oracle as O
    from oracle.model import OracleNet
    from paper_2011_14504_amd import synth
    small = synth.scaled(wl, 1, sample_hw, sample_hw)
    inp = synth.workload_inputs(small)
    net = OracleNet(small, inp, **(widths or {}))
    t0 = time.perf_counter()
    net.step()
    dt = time.perf_counter() - t0
    ops, _ = workload_ops(small)
    full_ops, _ = workload_ops(wl)
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            cpu = next(l.split(":", 1)[1].strip() for l in fh if l.startswith("model name"))
    except (OSError, StopIteration):
        pass
    return dict(value=ops / dt / 1e12, unit="TOPS", cores=O.num_threads(), cpu=cpu, kind="oracle",
                sample=f"one full training step (fwd, loss, bwd, update) of the same network on one "
                       f"{sample_hw}x{sample_hw} image: {dt:.2f} s for {ops / 1e9:.1f} G conv ops",
                images_per_s_est=(ops / full_ops) * wl["N"] / dt)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="deeplabv3", choices=sorted(WORKLOAD_IDS))
    ap.add_argument("--batch", type=int, default=None)
    ap.add_argument("--cpu-sample-hw", type=int, default=128)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--k-w", type=int, default=8, help="weight code width k_W (Table 1 rows: 8, 4)")
    ap.add_argument("--k-a", type=int, default=8, help="activation code width k_A")
    ap.add_argument("--k-e2", type=int, default=16, help="BN error width k_E2 (8 or 16)")
    ap.add_argument("--k-u", type=int, default=24, help="master / update width k_U")
    ap.add_argument("--gq", type=int, default=None, choices=(1, 2),
                    help="weight-gradient quantizer: 1 keeps Scale(G) (Eq. 17), 2 drops it (Eq. 18); "
                         "default: the workload's (2 for FCN8s, 1 otherwise)")
    ap.add_argument("--no-bn", action="store_true", help="the same network without L1BN")
    ap.add_argument("--bn-input", default="q8", choices=("q8", "raw"),
                    help="L1BN on the SQ8 conv output (q8) or on the raw int32 sums (the literal dataflow)")
    ap.add_argument("--copy-kernel-mib", type=int, default=0,
                    help="only run the plain copy kernel used to calibrate the HBM byte counters")
    ap.add_argument("--timed-kernel", default="bn_bwd_stats:*",
                    help="<family>:<layer or *>, family one of conv_fwd, conv_bwd_data, conv_wgrad, "
                         "bn_fwd_stats1, bn_fwd_stats2, bn_fwd_apply, bn_bwd_stats, bn_bwd_apply; * times "
                         "every launch of the family in the timed steps (the default: the L1BN backward "
                         "statistics pass, the step's largest kernel by time)")
    ap.add_argument("--no-replay", action="store_true",
                    help="enqueue every step from Python instead of replaying the recorded last warm-up step")
    ap.add_argument("--conv-steps", type=int, default=2,
                    help="extra steps after the timed ones whose conv entry points are timed one by one "
                         "(conv TOPS over conv time)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the multi-GPU "
              f"sharding of this path is described in DESIGN.md and not built.", file=sys.stderr)
        sys.exit(2)

    if args.copy_kernel_mib:
        copy_kernel(args.copy_kernel_mib)
        return

    import torch
    from paper_2011_14504_amd import iseg, synth
    from paper_2011_14504_amd.model import IntNet

    wl = synth.scaled(synth.WORKLOADS[WORKLOAD_IDS[args.workload]], args.batch)
    if args.no_bn:
        wl = synth.without_bn(wl)
    N = wl["N"]
    if args.gq is None:
        args.gq = wl.get("gq", 1)
    inp = synth.workload_inputs(wl)
    widths = dict(k_W=args.k_w, k_U=args.k_u, bn_cfg={"k_A": args.k_a, "k_E2": args.k_e2}, gq=args.gq)
    # the last warm-up step is recorded into a step tape and the timed steps
    # replay it from native code (the same calls, buffers and stream orderings;
    # the host no longer enqueues each call from Python)
    replay = not args.no_replay and args.warmup >= 1
    net = IntNet(wl, inp, "cuda:0", bn_input=args.bn_input, replay_from=args.warmup - 1 if replay else None,
                 **widths)
    ops, detail = workload_ops(wl)
    tk = args.timed_kernel
    if tk.startswith("bn_") and (args.no_bn or not any(nd.get("bn") for nd in synth.conv_nodes(wl))):
        tk = "conv_fwd:*"
    kinfo = timed_kernel_info(tk, wl, detail)
    prof = iseg.KernelTimer(kinfo["kid"], layer_match=kinfo["key"])

    # the last warm-up step runs with the timer installed, so the events the
    # timed steps record are created before the timed region
    for i in range(args.warmup):
        if i == args.warmup - 1:
            iseg.set_kernel_timer(prof)
        net.step()
    torch.cuda.synchronize()
    iseg.set_kernel_timer(None)
    armed = [(kid, key) for _, _, kid, key in prof.pairs]
    prof.reset()
    if replay:
        # the recorded step armed the timed kernel's launches: each replay of
        # the timed region gets its own (start, stop) events for them
        events = []
        for _ in range(args.steps):
            for kid, key in armed:
                a, b = prof._event(), prof._event()
                prof.pairs.append((a, b, kid, key))
                events.append((a.value, b.value))
        net.tape.set_arm_events(events, args.steps)
    else:
        iseg.set_kernel_timer(prof)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        net.step()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    iseg.set_kernel_timer(None)
    ms = dt / args.steps * 1e3
    value = ops / (dt / args.steps) / 1e12

    # the timed kernel: algorithmic work of each launch over its measured time
    runs = prof.launches()
    prof.close()
    launches = len(runs)
    k_ms = sum(t for _, _, t in runs) / launches if launches else None
    per_launch = sum(kinfo["work"](k) for _, k, _ in runs) / launches if launches else None
    if kinfo["bound"] == "mfma":
        ach = per_launch / (k_ms * 1e-3) / 1e12 if k_ms else None
        roof = dict(kernel=kinfo["name"], bound="mfma", achieved=ach, peak=INT8_PEAK_TOPS,
                    unit="TFLOP/s", frac=(ach / INT8_PEAK_TOPS) if ach else None, traffic=None,
                    algorithmic_ops_per_launch=per_launch, avg_launch_ms=k_ms, launches=launches)
    else:
        ach = per_launch / (k_ms * 1e-3) / 1e9 if k_ms else None
        roof = dict(kernel=kinfo["name"], bound="hbm", achieved=ach, peak=HBM_PEAK_GBS,
                    unit="GB/s", frac=(ach / HBM_PEAK_GBS) if ach else None, traffic=None,
                    algorithmic_bytes_per_launch=per_launch, avg_launch_ms=k_ms, launches=launches)
    traffic = measured_traffic(tk)
    roof["traffic"] = traffic
    roof["traffic_unit"] = "bytes per launch (HBM, rocprofv3 FETCH_SIZE + WRITE_SIZE, calibrated)"
    if tk in TRAFFIC:
        roof["profile"] = TRAFFIC[tk]["profile"]

    # conv throughput over conv time: every conv entry point of a few more
    # steps timed by its own events (the weight gradients overlap other work
    # on their stream, so this sums kernel time, not wall time)
    conv_tops = None
    if args.conv_steps > 0:
        ct = iseg.KernelTimer([iseg.ISEG_KID_CONV_FWD, iseg.ISEG_KID_CONV_BWD_DATA, iseg.ISEG_KID_CONV_WGRAD])
        iseg.set_kernel_timer(ct)
        for _ in range(args.conv_steps):
            net.step(eager=True)
        torch.cuda.synchronize()
        iseg.set_kernel_timer(None)
        conv_ms = sum(t for _, _, t in ct.launches())
        ct.close()
        conv_tops = ops * args.conv_steps / (conv_ms * 1e-3) / 1e12 if conv_ms else None
    cfg = dict(workload=wl["name"], batch=N, image=f"{wl['H']}x{wl['W']}",
               convs=len(detail), conv_ops_per_step=ops, images_per_s=N / (dt / args.steps),
               pct_int8_peak=100.0 * value / INT8_PEAK_TOPS,
               bits=dict(W=args.k_w, A=args.k_a, G=8, E1=8, E2=args.k_e2, U=args.k_u), gq=args.gq,
               l1bn=any(nd.get("bn") for nd in synth.conv_nodes(wl)), bn_input=args.bn_input,
               step_issue="replay of the recorded step tape" if replay else "python",
               conv_tops_over_conv_time=conv_tops,
               conv_pct_int8_peak_over_conv_time=(100.0 * conv_tops / INT8_PEAK_TOPS) if conv_tops else None)
    status = net.read_status()
    if net.loss is not None:
        cfg["loss"] = float(net.loss.item())
    if status != 0 or (net.loss is not None and not math.isfinite(cfg["loss"])):
        print(f"bench.py: the training step flagged device status {status} (loss "
              f"{cfg.get('loss')}); the measurement is not valid", file=sys.stderr)
        sys.exit(3)
    out = dict(metric=METRIC, value=value, unit="TOPS", n_gpus=1, steps=args.steps,
               warmup=args.warmup, ms_per_step=ms, higher_is_better=True, scaling="weak",
               vs_baseline=None, dtype="int8", data="synthetic", config=cfg, roofline=roof)
    if not args.no_cpu_baseline:
        sample = args.cpu_sample_hw if wl["H"] > args.cpu_sample_hw else wl["H"]
        out["cpu_baseline"] = cpu_baseline(wl, sample, widths)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
