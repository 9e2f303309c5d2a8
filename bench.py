"""Benchmark of the fused-MLP hot path on one MI355X.

One step = the whole path over one synthetic batch of M rows:
  pack the weights (they change every training step), one inference forward
  pass (Algorithm 1), one training step (Algorithm 2: forward with stash, MSE
  loss and output delta, backward delta propagation, weight gradients).
`value` is M / (time per step) in samples/s with inputs resident in HBM.

The `roofline` object is the inference kernel (one launch per forward
call, so HIP events on its stream around it in every timed step time
exactly that launch): algorithmic flops 2 * sum(fan_in * fan_out) per row
against the dense bf16 MFMA peak.
`roofline_train` is the whole training step against HBM bandwidth, with
its algorithmic bytes per row.  `cpu_baseline` times the fp64 oracle on a
bounded sample of the same step on the host cores.

    python bench.py [--steps K] [--warmup W] [--repeats R] [--width 128 --depth 4 --batch 1048576]
    python bench.py --roofline-plot OUT.svg [--batch M] [--steps K --repeats R]

The timing protocol of the paper's sweeps (section IV-A) is
--steps max(1000 * 2^18 / M, 250) --warmup 10 --repeats 5: the median of
five repeats, each the mean over the steps.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "samples/s + TFLOP/s (% bf16 MFMA peak) for fused MLP fwd and train step"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def flops_per_row(width, depth, in_dim, out_dim):
    shapes = [(in_dim if l == 0 else width, out_dim if l == depth else width)
              for l in range(depth + 1)]
    P = sum(a * b for a, b in shapes)
    fwd = 2 * P
    bwd = 2 * (P - shapes[0][0] * shapes[0][1])  # no input gradient
    return fwd, fwd + bwd + 2 * P  # inference, training step


def fused_backward(width, depth, in_dim, out_dim, act):
    """Whether the library's training step runs the fused backward kernel
    (deltas kept on chip, weight gradients accumulated in the same kernel):
    2 to 5 weight matrices and, at width 128, ReLU hidden layers and at most
    16 outputs; otherwise it runs the three kernels (backward, weight
    gradients, reduce).  The rule of include/ffmlp.h."""
    return 1 <= depth <= 4 and (width != 128 or (act == "relu" and out_dim <= 16))


def fused_step(width, depth):
    """Whether the library runs the whole training step as one kernel
    (widths 16, 32 and 64, 2 to 5 weight matrices): the activations stay on
    chip, so only X and T (and Y when asked for) touch HBM."""
    return width in (16, 32, 64) and 1 <= depth <= 4


def train_bytes_per_row(width, depth, in_dim, out_dim, act, fused=None, masks=True):
    """HBM bytes the training step must move per row.
    One-kernel step (fused=None at widths 16, 32 and 64 with 2 to 5 matrices):
    X and T (the bench asks for no Y).
    Forward (both plans): reads X and T, writes the activations, the output
    delta and (ReLU) the activation masks.
    Fused plan: the backward kernel reads the output delta, X and the
    activations (the weight-gradient operands; at widths up to 64 also the
    ReLU and sigmoid derivative source), plus the masks at width 128 and the
    cos stash of sine nets, and writes no deltas.
    Three-kernel plan: the backward reads the output delta and the
    derivative source of every hidden activation (ReLU: its mask, 16 B per
    row, or with masks=False the activation itself; sigmoid: the
    activation; sine: the stored cos; linear: nothing) and writes the hidden
    deltas; the gradient kernel reads X, the activations, the hidden deltas
    and the output delta."""
    if fused is None:
        if fused_step(width, depth):
            return 2 * in_dim + 4 * out_dim
        fused = fused_backward(width, depth, in_dim, out_dim, act)
    OP = (out_dim + 15) // 16 * 16
    hid = depth * width * 2
    if fused:
        # ReLU masks only at width 128; at widths up to 64 the fused kernel
        # takes relu' (and sigmoid's a (1 - a)) from the activations it reads
        # for the weight gradients: one read of them
        mask = depth * 16 if (act == "relu" and width == 128) else 0
        cos = hid if act == "sine" else 0
        b = 2 * in_dim + 4 * out_dim + hid + 2 * OP + mask + cos   # forward (train)
        return b + 2 * OP + mask + cos + 2 * in_dim + hid           # fused backward
    mask = depth * 16 if (act == "relu" and masks) else 0
    deriv = {"relu": mask if masks else hid, "linear": 0}.get(act, hid)
    b = 2 * in_dim + 4 * out_dim + hid + 2 * OP + mask    # forward (train)
    if act == "sine":
        b += hid                                          # cos stash write
    b += 2 * OP + deriv + hid                             # backward
    b += 2 * in_dim + hid + hid + 2 * OP                  # weight gradients
    return b


def measured_traffic(key):
    """HBM bytes per launch of the inference kernel from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE runs (profiles/traffic.json), or None
    when there are none for this workload or the kernel sources have changed
    since they were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    entry = json.load(open(path)).get(key)
    if entry is None:
        return None
    h = hashlib.sha256()
    for src in entry["sources"]:
        with open(os.path.join(ROOT, src), "rb") as f:
            h.update(f.read())
    if h.hexdigest() != entry["sources_sha256"]:
        return None
    return entry["hbm_bytes_per_launch"]


def cpu_baseline(width, depth, in_dim, out_dim, act, out_act, target_s=12.0):
    """The oracle (fp64, OpenMP over rows) on a bounded sample of the step:
    one inference forward plus one training step per row."""
    import oracle
    import datagen
    acts = {"linear": oracle.LINEAR, "relu": oracle.RELU, "sigmoid": oracle.SIGMOID,
            "sine": oracle.SINE}
    net = oracle.Net(width, depth, in_dim, out_dim, acts[act], acts[out_act])
    W = datagen.xavier_weights(3, width, depth, in_dim, out_dim)

    def run(m):
        X = datagen.inputs_uniform(3, m, in_dim)
        T = datagen.targets_uniform(3, m, out_dim)
        t0 = time.perf_counter()
        net.forward(W, X)
        net.train_step(W, X, T)
        return time.perf_counter() - t0

    m, dt = 4096, run(4096)
    while dt < 0.8 * target_s and m < (1 << 22):
        m = int(min(max(m * target_s / max(dt, 1e-3), 2 * m), 1 << 22))
        dt = run(m)
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or os.cpu_count()
    # the same on one core, on a smaller sample (about 3 s)
    net1 = oracle.Net(width, depth, in_dim, out_dim, acts[act], acts[out_act], threads=1)
    m1 = max(256, int(m / dt / threads * 3.0))
    X1 = datagen.inputs_uniform(3, m1, in_dim)
    T1 = datagen.targets_uniform(3, m1, out_dim)
    t0 = time.perf_counter()
    net1.forward(W, X1)
    net1.train_step(W, X1, T1)
    dt1 = time.perf_counter() - t0
    return {"value": m / dt, "unit": "samples/s", "cores": threads, "kind": "oracle",
            "sample": f"{m} rows of the same net and input recipe, inference forward + training "
                      f"step, fp64, {dt:.1f} s",
            "value_1core": m1 / dt1, "sample_1core": f"{m1} rows, {dt1:.1f} s"}


def measure(width, depth, in_dim, out_dim, M, act, out_act, K, Wm, R=1, inputs="default"):
    """Time K steps (after Wm warm-up steps) R times with HIP events on the
    launch stream; returns the repeat with the median time per step, plus
    the spread over the repeats."""
    import statistics

    import torch
    import datagen
    import paper_2403_17607_amd as ffmlp

    dev = torch.device("cuda:0")
    net = ffmlp.FusedMLP(width, depth, in_dim, out_dim, act, out_act)
    W = datagen.xavier_weights(2, width, depth, in_dim, out_dim, device=dev)
    # Input buffers used in turn.  By default two, so inference at large
    # batches does not run out of the 256 MiB last-level cache; "cold"
    # rotates X and T over at least 512 MiB whatever the batch, "hot" reuses
    # one of each.
    if inputs == "cold":
        nbuf = max(2, -(-(512 << 20) // max(1, M * (2 * in_dim + 4 * out_dim))))
    else:
        nbuf = 1 if inputs == "hot" else 2
    Xs = [datagen.inputs_uniform(2 + i, M, in_dim, device=dev) for i in range(nbuf)]
    Ts = [datagen.targets_uniform(2 + i, M, out_dim, device=dev)
          for i in range(nbuf if inputs == "cold" else 1)]
    packed = net.pack(W)
    ws = net.workspace(M, dev)
    Y = torch.empty(M, out_dim, dtype=torch.bfloat16, device=dev)
    G = torch.empty(net.param_count(), dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]

    def step(i, events=None):
        if events:
            events[0].record(stream)
        net.pack(W, out=packed)
        if events:
            events[1].record(stream)
        x = Xs[i % len(Xs)]
        net.forward(packed, x, Y=Y)
        if events:
            events[2].record(stream)
        net.train_step(packed, x, Ts[i % len(Ts)], ws, G=G, loss=loss)
        if events:
            events[3].record(stream)

    for i in range(Wm):
        step(i)
    # Untimed device-to-device copy of a known size (the first input
    # buffer): a reference for calibrating hardware byte counters.
    ref_copy = torch.empty_like(Xs[0])
    ref_copy.copy_(Xs[0])
    del ref_copy
    reps = []
    for r in range(R):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(K):
            step(i, ev[i])
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        reps.append({
            "ms_per_step": wall * 1e3 / K,
            "event_ms_per_step": sum(e[0].elapsed_time(e[3]) for e in ev) / K,
            "infer_ms": sum(e[1].elapsed_time(e[2]) for e in ev) / K,
            "train_ms": sum(e[2].elapsed_time(e[3]) for e in ev) / K,
            "pack_ms": sum(e[0].elapsed_time(e[1]) for e in ev) / K,
            "infer_ms_median_launch": statistics.median(e[1].elapsed_time(e[2]) for e in ev),
        })
    del ws
    torch.cuda.empty_cache()
    order = sorted(range(R), key=lambda r: reps[r]["ms_per_step"])
    res = dict(reps[order[R // 2]])
    res["repeats"] = R
    if R > 1:
        res["spread"] = {k: [min(x[k] for x in reps), max(x[k] for x in reps)]
                         for k in ("ms_per_step", "infer_ms", "train_ms")}
    res["nbuf"] = nbuf
    return res


def summarize(width, depth, in_dim, out_dim, M, act, out_act, m):
    """Derived rates of one measurement: samples/s, algorithmic TFLOP/s and
    HBM GB/s of the inference launch and of the training step."""
    fl_inf, fl_train = flops_per_row(width, depth, in_dim, out_dim)
    t_inf, t_train = m["infer_ms"], m["train_ms"]
    bytes_inf = 2 * in_dim + 2 * out_dim
    bytes_train = train_bytes_per_row(width, depth, in_dim, out_dim, act)
    return {
        "infer": {"ms": t_inf, "samples_per_s": M / (t_inf * 1e-3),
                  "tflops": fl_inf * M / (t_inf * 1e-3) / 1e12,
                  "pct_bf16_peak": 100 * fl_inf * M / (t_inf * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                  "hbm_gbs_algorithmic": bytes_inf * M / (t_inf * 1e-3) / 1e9,
                  "flop_per_byte": fl_inf / bytes_inf},
        "train": {"ms": t_train, "samples_per_s": M / (t_train * 1e-3),
                  "tflops": fl_train * M / (t_train * 1e-3) / 1e12,
                  "pct_bf16_peak": 100 * fl_train * M / (t_train * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                  "hbm_gbs_algorithmic": bytes_train * M / (t_train * 1e-3) / 1e9,
                  "flop_per_byte": fl_train / bytes_train, "bytes_per_row": bytes_train},
    }


def roofline_plot(path, points, batch):
    """Arithmetic intensity against achieved TFLOP/s, with the HBM and MFMA
    roofs, one point per width for inference and for the training step."""
    import matplotlib
    matplotlib.use("Agg")
    matplotlib.rcParams["svg.fonttype"] = "none"  # text as text: a small SVG
    import matplotlib.pyplot as plt
    ai = [2 ** (k / 8) for k in range(0, 8 * 12 + 1)]  # 1 .. 4096 flop/B
    fig, ax = plt.subplots(figsize=(7.5, 5))
    ax.plot(ai, [min(PEAK_BF16_TFLOPS, PEAK_HBM_GBS * a / 1e3) for a in ai], "k-", lw=1.5,
            label="MI355X roofline (8 TB/s HBM, 2.5 PFLOP/s dense bf16)")
    for kind, marker in (("infer", "o"), ("train", "s")):
        xs = [p[kind]["flop_per_byte"] for p in points]
        ys = [p[kind]["tflops"] for p in points]
        ax.plot(xs, ys, marker, ms=7, label={"infer": "inference (Algorithm 1)",
                                             "train": "training step (Algorithm 2)"}[kind])
        for p, x, y in zip(points, xs, ys):
            ax.annotate(f"w{p['width']}", (x, y), textcoords="offset points", xytext=(5, -10),
                        fontsize=8)
    ax.set_xscale("log", base=2)
    ax.set_yscale("log", base=10)
    ax.set_xlabel("algorithmic arithmetic intensity (flop / HBM byte)")
    ax.set_ylabel("achieved TFLOP/s (algorithmic flops)")
    ax.set_title(f"Fused MLP, 4 hidden layers, in = width, out 16, ReLU, batch {batch}")
    ax.grid(True, which="both", lw=0.3)
    ax.legend(fontsize=8, loc="lower right")
    fig.tight_layout()
    fig.savefig(path, metadata={"Date": None})
    plt.close(fig)


def default_steps(M):
    """Timed steps per repeat in the paper's protocol (section IV-A):
    max(1000 * 2^18 / M, 250)."""
    return max(1000 * (1 << 18) // max(M, 1), 250)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps K per repeat (default: the paper's protocol, "
                         "max(1000 * 2^18 / batch, 250))")
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--repeats", type=int, default=5,
                    help="time the K steps this many times and report the median repeat "
                         "(with the min-max spread)")
    ap.add_argument("--width", type=int, default=128)
    ap.add_argument("--depth", type=int, default=4)
    ap.add_argument("--in-dim", type=int, default=None)
    ap.add_argument("--out-dim", type=int, default=16)
    ap.add_argument("--batch", type=int, default=1 << 20)
    ap.add_argument("--act", default="relu")
    ap.add_argument("--out-act", default="linear")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle timing")
    ap.add_argument("--inputs", choices=["default", "cold", "hot"], default="default",
                    help="default: X alternates between two buffers; cold: X and T rotate "
                         "over at least 512 MiB of buffers (beyond the 256 MiB last-level "
                         "cache); hot: one X and T buffer every step")
    ap.add_argument("--roofline-plot", metavar="SVG",
                    help="instead of the bench line: measure widths 16, 32, 64, 128 (in = "
                         "width, out 16, 4 hidden layers, ReLU) at --batch and draw arithmetic "
                         "intensity against achieved TFLOP/s under the roofs")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(inference would shard rows with no communication; training would add "
              "one all-reduce of the gradients).", file=sys.stderr)
        sys.exit(2)

    M = args.batch
    K = args.steps if args.steps is not None else default_steps(M)
    Wm, R = args.warmup, args.repeats
    if args.roofline_plot:
        points = []
        for w in (16, 32, 64, 128):
            m = measure(w, 4, w, 16, M, "relu", "linear", K, Wm, R)
            p = summarize(w, 4, w, 16, M, "relu", "linear", m)
            p["width"] = w
            points.append(p)
            print(json.dumps({"width": w, "batch": M, **p}), flush=True)
        roofline_plot(args.roofline_plot, points, M)
        return

    width, depth = args.width, args.depth
    in_dim = args.in_dim or width
    out_dim = args.out_dim
    m = measure(width, depth, in_dim, out_dim, M, args.act, args.out_act, K, Wm, R, args.inputs)
    d = summarize(width, depth, in_dim, out_dim, M, args.act, args.out_act, m)
    fused = fused_backward(width, depth, in_dim, out_dim, args.act)
    fl_inf, _ = flops_per_row(width, depth, in_dim, out_dim)
    inf_tflops, train_gbs = d["infer"]["tflops"], d["train"]["hbm_gbs_algorithmic"]
    ms_per_step = m["ms_per_step"]
    out = {
        "metric": METRIC,
        "value": M / (ms_per_step * 1e-3),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wm,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"fused MLP width {width}, {depth} hidden layers, in {in_dim}, "
                               f"out {out_dim}, {args.act} hidden, {args.out_act} output, "
                               f"batch {M}: weight pack + inference + training step",
                   "width": width, "depth": depth, "in_dim": in_dim, "out_dim": out_dim,
                   "batch": M, "activation": args.act, "output_activation": args.out_act,
                   "inputs": {"default": "X alternates between 2 buffers",
                              "cold": f"X and T rotate over {m['nbuf']} buffers (>= 512 MiB)",
                              "hot": "one X and T buffer"}[args.inputs]},
        **d,
        "pack_ms": m["pack_ms"],
        "event_ms_per_step": m["event_ms_per_step"],
        "repeats": R,
        "roofline": {"kernel": "fwd_kernel (inference)", "bound": "mfma",
                     "achieved": inf_tflops, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": inf_tflops / PEAK_BF16_TFLOPS,
                     "launch_us": m["infer_ms"] * 1e3,
                     "launch_us_median": m["infer_ms_median_launch"] * 1e3,
                     "traffic": measured_traffic(
                         f"fwd_infer_w{width}_d{depth}_in{in_dim}_out{out_dim}_{args.act}_b{M}")
                     if args.out_act == "linear" else None,
                     "traffic_unit": "HBM bytes per launch: a committed rocprofv3 "
                                     "FETCH_SIZE + WRITE_SIZE measurement of this kernel and "
                                     "workload (profiles/traffic.json, scaled by a reference "
                                     "copy), null once the kernel's sources have changed",
                     "flops_per_row": fl_inf, "rows_per_launch": M},
        "roofline_train": {"kernels": (("trainw_kernel" if width == 64 else "trainf_kernel") +
                                       " (the whole step) + reduce_kernel"
                                       if fused_step(width, depth) else
                                       ("fwd_kernel (train) + " +
                                        ("bwdn_kernel" if width <= 32 else "bwdg_kernel") +
                                        " (fused backward and weight gradients) + reduce_kernel")
                                       if fused else
                                       ("fwd_kernel (train) + bwd_kernel + wgrad_kernel + "
                                        "reduce_kernel")),
                           "bound": "hbm", "achieved": train_gbs,
                           "peak": PEAK_HBM_GBS, "unit": "GB/s",
                           "frac": train_gbs / PEAK_HBM_GBS,
                           "bytes_per_row": train_bytes_per_row(width, depth, in_dim, out_dim,
                                                                args.act),
                           "bytes_per_row_three_kernels": train_bytes_per_row(
                               width, depth, in_dim, out_dim, args.act, fused=False),
                           "bytes_per_row_three_kernels_no_masks": train_bytes_per_row(
                               width, depth, in_dim, out_dim, args.act, fused=False,
                               masks=False)},
    }
    if R > 1:
        out["spread"] = m["spread"]
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(width, depth, in_dim, out_dim, args.act, args.out_act)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
