"""Benchmark: one integer training step (forward, backward, update) of the
FCN-VGG16 encoder slice (conv1_1, conv1_2, maxpool, conv2_1, conv2_2, L1BN +
ReLU after each conv) at batch 8 and 224x224, on one MI355X.

Prints ONE JSON line.  `value` is int8 conv throughput (valid-tap MACs x 2 of
forward, backward-data and backward-weight, per step) divided by the whole
step's wall time, with inputs already in HBM.  `roofline` reports the
dominant kernel, timed by HIP events bracketing each of its launches inside
the timed steps; `cpu_baseline` is the CPU oracle timed on a bounded sample.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "int8 conv TOPS fwd+bwd (% MFMA peak); train images/s DeepLabv3-R50 512²"
INT8_PEAK_TOPS = 5000.0      # MI355X dense int8 MFMA
HBM_PEAK_GBS = 8000.0


def conv_valid_macs(N, H, W, C, K, R, st, pad, dil):
    """Multiply-adds of a conv that touch real (non-padding) input."""
    P = (H + 2 * pad - dil * (R - 1) - 1) // st + 1
    rows = sum(1 for p in range(P) for r in range(R) if 0 <= p * st - pad + r * dil < H)
    Q = (W + 2 * pad - dil * (R - 1) - 1) // st + 1
    cols = sum(1 for q in range(Q) for s in range(R) if 0 <= q * st - pad + s * dil < W)
    return N * rows * cols * C * K


def workload_ops(wl, N):
    """Valid-tap int8 ops (2 per MAC) per training step, and per-conv detail."""
    H, W = wl["H"], wl["W"]
    total, detail = 0, []
    first = True
    for layer in wl["layers"]:
        if layer[0] == "conv":
            _, cin, cout, R, st, pad, dil = layer
            macs = conv_valid_macs(N, H, W, cin, cout, R, st, pad, dil)
            passes = 3 if (not first or wl["input_grad"]) else 2
            total += 2 * macs * passes
            detail.append(dict(shape=(N, H, W, cin, cout, R, st, pad, dil), macs=macs))
            H = (H + 2 * pad - dil * (R - 1) - 1) // st + 1
            W = (W + 2 * pad - dil * (R - 1) - 1) // st + 1
            first = False
        else:
            _, k, st, pad = layer
            H = (H + 2 * pad - k) // st + 1
            W = (W + 2 * pad - k) // st + 1
    return total, detail


def timed_kernel_info(name, N, detail):
    """Kernel family, layer key and algorithmic work per launch of the kernels
    the benchmark can time in place; all on the conv1_2 layer (64 -> 64 3x3 at
    224x224) or the L1BN that follows it (M = N*224*224 rows, 64 channels)."""
    from paper_2011_14504_amd import iseg
    M, C = N * 224 * 224, 64
    conv_key = (N, 224, 224, 64, 64)
    ops = 2 * detail[1]["macs"]
    table = {
        "conv_fwd": (iseg.ISEG_KID_CONV_FWD, conv_key, "mfma", ops,
                     "k_conv3x3_m32 fwd, max pass (conv1_2, 64->64 3x3, 224x224)"),
        "conv_bwd_data": (iseg.ISEG_KID_CONV_BWD_DATA, conv_key, "mfma", ops,
                          "k_conv3x3_m32 bwd-data, max pass (conv1_2)"),
        "conv_wgrad": (iseg.ISEG_KID_CONV_WGRAD, conv_key, "mfma", ops,
                       "k_conv_wgrad_taps (conv1_2)"),
        # bytes per element: stats reads x and dy; apply reads x, dy and writes dx
        "bn_bwd_stats": (iseg.ISEG_KID_BN_BWD_STATS, (M, C), "hbm", 2 * M * C,
                         "k_bnb_stats (L1BN backward statistics, conv1_2 output)"),
        "bn_bwd_apply": (iseg.ISEG_KID_BN_BWD_APPLY, (M, C), "hbm", 3 * M * C,
                         "k_bnb_apply (L1BN backward output pass, conv1_2 output)"),
        "bn_fwd_stats1": (iseg.ISEG_KID_BN_FWD_STATS1, (M, C), "hbm", M * C,
                          "k_bnf_stats1 (L1BN forward mean pass, conv1_2 output)"),
        "bn_fwd_apply": (iseg.ISEG_KID_BN_FWD_APPLY, (M, C), "hbm", 2 * M * C,
                         "k_bnf_apply (L1BN forward output pass, conv1_2 output)"),
        # reads x (M C) and dy (M C / 4), writes dx (M C)
        "maxpool_bwd": (iseg.ISEG_KID_MAXPOOL_BWD, (N, 224, 224, 64), "hbm", M * C * 9 // 4,
                        "k_maxpool_bwd_win (2x2/2 after conv1_2)"),
    }
    kid, key, bound, work, label = table[name]
    return dict(kid=kid, key=key, bound=bound, work=work, name=label)


def cpu_baseline(wl, n_img):
    """The oracle's training step on n_img images, timed on the host cores."""
    from oracle import oracle as O
    from oracle.model import OracleNet
    from paper_2011_14504_amd import synth
    inp = synth.workload_inputs(wl, n_img)
    net = OracleNet(wl, inp)
    t0 = time.perf_counter()
    net.step()
    dt = time.perf_counter() - t0
    ops, _ = workload_ops(wl, n_img)
    return dict(value=ops / dt / 1e12, unit="TOPS", cores=O.num_threads(), kind="oracle",
                sample=f"one full training step (fwd+bwd+update) of the same workload at batch "
                       f"{n_img}: {dt:.2f} s",
                images_per_s=n_img / dt)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--batch", type=int, default=8)
    ap.add_argument("--cpu-images", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--timed-kernel", default="conv_fwd",
                    choices=["conv_fwd", "conv_bwd_data", "conv_wgrad", "bn_bwd_stats",
                             "bn_bwd_apply", "bn_fwd_stats1", "bn_fwd_apply", "maxpool_bwd"])
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the multi-GPU "
              f"sharding of this path is described in DESIGN.md and not built.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2011_14504_amd import iseg, synth
    from paper_2011_14504_amd.model import IntNet

    wl = synth.VGG16_BLOCKS12
    N = args.batch
    inp = synth.workload_inputs(wl, N)
    net = IntNet(wl, inp, "cuda:0")
    ops, detail = workload_ops(wl, N)

    kinfo = timed_kernel_info(args.timed_kernel, N, detail)
    prof = iseg.KernelTimer(kinfo["kid"], layer_match=kinfo["key"])

    for _ in range(args.warmup):
        net.step()
    torch.cuda.synchronize()
    iseg.set_kernel_timer(prof)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        net.step()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    iseg.set_kernel_timer(None)
    ms = dt / args.steps * 1e3
    value = ops / (dt / args.steps) / 1e12

    k_ms = prof.mean_ms()
    per_launch = kinfo["work"]
    if kinfo["bound"] == "mfma":
        ach = per_launch / (k_ms * 1e-3) / 1e12 if k_ms else None
        roof = dict(kernel=kinfo["name"], bound="mfma", achieved=ach, peak=INT8_PEAK_TOPS,
                    unit="TFLOP/s", frac=(ach / INT8_PEAK_TOPS) if ach else None, traffic=None,
                    algorithmic_ops_per_launch=per_launch, avg_launch_ms=k_ms,
                    launches=prof.count())
    else:
        ach = per_launch / (k_ms * 1e-3) / 1e9 if k_ms else None
        roof = dict(kernel=kinfo["name"], bound="hbm", achieved=ach, peak=HBM_PEAK_GBS,
                    unit="GB/s", frac=(ach / HBM_PEAK_GBS) if ach else None, traffic=None,
                    algorithmic_bytes_per_launch=per_launch, avg_launch_ms=k_ms,
                    launches=prof.count())

    out = dict(metric=METRIC, value=value, unit="TOPS", n_gpus=1, steps=args.steps,
               warmup=args.warmup, ms_per_step=ms, higher_is_better=True, scaling="weak",
               vs_baseline=None, dtype="int8", data="synthetic",
               config=dict(workload=wl["name"], batch=N, image=224, convs=4, bn="L1BN x4",
                           conv_ops_per_step=ops, images_per_s=N / (dt / args.steps),
                           pct_int8_peak=100.0 * value / INT8_PEAK_TOPS),
               roofline=roof)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_images)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
