"""Throughput of the local-SGD hot path on one MI355X.

One step = one local-SGD round: H local steps on every one of the K replicas
(sample, gather, forward, loss, backward, fused update) followed by the K-way
average. Default workload: the ResNet-20-shaped CNN of the paper's CIFAR
experiments (3x3 convolutions as implicit GEMMs, 16/32/64 channels, three
basic blocks per stage, per-worker batch normalisation, global average
pooling, 10-way classifier), fp32, K=16, B_loc=128, H=16, heavy-ball momentum
0.9, weight decay 1e-4, synthetic 32x32x3 / 10-class Gaussian images (32,768
samples per round). ``--workload`` selects the other workloads.

Prints one JSON line: samples/s, the roofline position of the dominant kernel
(timed with HIP events on the library's stream) and the CPU oracle timed on a
bounded sample of the same workload on the host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_TFLOPS = {"fp32": 157.3, "bf16": 2500.0}
METRIC = "aggregate samples/s per local-SGD round at 1 GPU"
EVENT_GAP_MS = 0.4      # timed rounds between two HIP events: at least this long
MAX_AUTO_STEPS = 20000
PROFILES = os.path.join(ROOT, "profiles")


def traffic_file(workload: str) -> str:
    return os.path.join(PROFILES, f"traffic_counters_{workload}.json")


def parse():
    p = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=None,
                   help="timed rounds (default 20; rounds shorter than 1 ms: "
                        "as many as fill about 100 ms)")
    p.add_argument("--warmup", type=int, default=3, help="untimed rounds")
    p.add_argument("--workload", default="resnet20")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--lazy-average", action="store_true",
                   help="the lazy form of the plain average (the mean written "
                        "once, read by the next local step; MLP workloads)")
    p.add_argument("--no-kernel-timing", action="store_true")
    p.add_argument("--sweep", action="store_true",
                   help="HBM sweep of the K-way average and the fused update "
                        "from 64 MB to 4 GB working sets (one JSON line per size)")
    p.add_argument("--traffic-from", metavar="DIR",
                   help="no GPU run: turn the rocprofv3 FETCH_SIZE / "
                        "WRITE_SIZE passes under DIR (fetch/, write/) into "
                        "profiles/traffic_counters_<workload>.json")
    p.add_argument("--traffic-tag", default=None,
                   help="with --traffic-from: the launch tag to account "
                        "(default: the workload's dominant one)")
    return p.parse_args()


def kernel_cost(tag: str, w) -> tuple:
    """Algorithmic (flops, bytes) of one launch of the kernel at `tag`.

    Bytes count each operand once: read inputs, read+write of what the
    kernel updates; weights W and momentum U are fp32 (4 B) masters, GEMM
    operands 4 B (fp32) or 2 B (bf16)."""
    K, B = w.K, w.B_loc
    d = w.widths
    L = len(d) - 1
    e = 2 if w.dtype == "bf16" else 4
    P = sum(a * b + b for a, b in zip(d[:-1], d[1:]))
    if tag == "sample":
        return 0, K * B * 4
    if w.model == "resnet20":
        if tag in ("average", "average_bn_running"):
            n = resnet_param_count(d[-1]) if tag == "average" else RESNET20_RUNNING
            return K * n, K * n * 8
        costs = resnet_step_costs(w)
        if tag not in costs:
            return None, None
        launches, flops, nbytes = costs[tag]
        return flops / launches, nbytes / launches
    if w.model != "mlp":
        return None, None
    if tag == "xent":
        return 0, K * B * d[L] * (4 + e) + K * B * 8
    if tag == "average" and getattr(w, "lazy_average", False):
        # the mean written once (and its bf16 copy)
        return K * P, K * P * 4 + P * 4 + (P * 2 if e == 2 else 0)
    if tag in ("average", "average_blocks"):   # same traffic per launch
        gm = 16 * P if w.global_momentum else 0  # w_sync and u read + written
        return K * P, K * P * 8 + (K * P * 2 if e == 2 else 0) + gm
    if tag == "sign_sync":   # two passes: l1 + packed signs, then apply
        if w.scheme == "ef_sign":   # W, e read twice, written once
            return 0, 24 * K * P + 8 * P
        return 0, 8 * K * P + K * P // 2 + 8 * P
    if tag in ("tiny_round", "tiny_round_wide") and L == 1:   # a round in one workgroup
        H = w.H * w.Hb
        D, C = d
        flops = H * K * (2 * B * D * C + 2 * B * (D + 1) * C)   # logits + gradient
        # batch rows + labels per step, replicas and buffers read and written
        # once, the losses
        return flops, H * K * B * (D * 4 + 4) + 16 * K * P + 4 * H * K
    if tag == "wgrad_update":   # one launch over every generic layer
        Lg = L - 1 if d[L] <= 32 else L   # the top layer has its own kernels
        costs = [kernel_cost(f"wgrad_update{l}", w) for l in range(1, Lg + 1)]
        return sum(c[0] for c in costs), sum(c[1] for c in costs)
    if w.model != "mlp" or not tag[-1:].isdigit():
        return None, None        # no per-kernel accounting for this kernel
    name, l = tag.rstrip("0123456789"), int(tag[len(tag.rstrip("0123456789")):])
    din, dout = d[l - 1], d[l]
    mn = din * dout
    if name == "fwd":
        out = e if l < L else 4
        return (2 * K * B * mn,
                K * (B * din * e + mn * e + dout * 4 + B * dout * out))
    if name == "dgrad":
        return 2 * K * B * mn, K * (B * dout * e + mn * e + 2 * B * din * e)
    if name == "wgrad_update":   # includes the fused bias gradient + update
        upd = 16 + (2 if e == 2 else 0)
        return (2 * K * B * mn + K * B * dout,
                K * (B * din * e + B * dout * e + (mn + dout) * upd))
    if name == "bias_update":
        return K * B * dout, K * (B * dout * e + dout * 16)
    raise ValueError(tag)


# ResNet-20 multiply-adds per image: forward 40,551,040 (Table 5's 0.041 G);
# the weight gradient repeats them; the input gradient skips the stem.
RESNET20_MACS, RESNET20_STEM_MACS = 40551040, 32 * 32 * 27 * 16
RESNET20_RUNNING = 2 * (16 * 7 + 32 * 6 + 64 * 6)   # BN running means + variances


def resnet20_convs():
    """(c_in, c_out, stride, input side, output side) of the 19 3x3
    convolutions: the stem, then per stage three blocks of two."""
    out, c, side = [(3, 16, 1, 32, 32)], 16, 32
    for st, co in enumerate((16, 32, 64)):
        for b in range(3):
            stride = 2 if (st > 0 and b == 0) else 1
            so = side // stride
            out += [(c, co, stride, side, so), (co, co, 1, so, so)]
            c, side = co, so
    return out


def resnet_param_count(classes: int) -> int:
    return sum(9 * ci * co + 2 * co for ci, co, *_ in resnet20_convs()) + 64 * classes + classes


def resnet_step_costs(w) -> dict:
    """{launch tag: (launches, algorithmic flops, algorithmic bytes)} of one
    ResNet-20 local step over all K replicas. Flops: 2 per multiply-add of
    each convolution (forward, input gradient except the stem's, weight
    gradient). Bytes: every tensor a kernel family must read or write, once
    (fp32): activations, output gradients, weights; BN's forward apply reads
    the pre-BN output (and the shortcut input of a block's second
    convolution) and writes the activation; BN's backward reads the pre-BN
    output and the upstream gradient twice (sums, then apply; plus the block
    output for the ReLU mask after a shortcut add) and writes the input
    gradient; the weight update reads the gradient once and reads and writes
    the weights and momentum (20 B per weight)."""
    K, B, C = w.K, w.B_loc, w.widths[-1]
    convs = resnet20_convs()
    t = {}

    def add(tag, fl, by):
        n, f0, b0 = t.get(tag, (0, 0, 0))
        t[tag] = (n + 1, f0 + fl, b0 + by)
    for i, (ci, co, st, si, so) in enumerate(convs):
        x = K * B * si * si * ci * 4          # conv input
        y = K * B * so * so * co * 4          # conv output / BN tensor
        wt = K * 9 * ci * co * 4
        fl = 2 * K * B * so * so * 9 * ci * co
        add("conv_fwd", fl, x + y + wt)
        add("bn_stats", 0, K * (B * so * so // 256) * co * 16 + K * co * 24)
        second = i > 0 and i % 2 == 0         # second convolution of a block
        sc = 0
        if second:
            cin_blk = convs[i - 1][0]
            sc = y if (convs[i - 1][2] == 1 and cin_blk == co) else K * B * so * so * cin_blk * 4
        if i % 2 == 0:   # a block's first BN-ReLU is formed by its consumers
            add("bn_apply", 0, 2 * y + sc)
        add("bn_bwd", 0, (7 if second else 5) * y)
        if i > 0:
            add("conv_dgrad", fl, y + x + wt)
        add("conv_wgrad", fl, x + y + wt)
        add("conv_wupdate", 0, 5 * wt)
        if second:
            cin_blk, _, st_a, si_a, _ = convs[i - 1]
            if st_a == 1 and cin_blk == co:
                add("shortcut_bwd", 0, 4 * y)
            else:
                add("shortcut_bwd", 0, 4 * K * B * so * so * cin_blk * 4)
    last = K * B * 8 * 8 * 64 * 4
    add("gap", 0, last + K * B * 64 * 4)
    add("gap_bwd", 0, last + K * B * 64 * 4)
    add("head_fwd", 2 * K * B * 64 * C, K * B * (64 + 2 * C) * 4 + K * 65 * C * 4)
    add("head_wgrad", 2 * K * B * 64 * C, K * B * (64 + C) * 4 + K * 65 * C * 16)
    return t


def gemm_flops_per_local_step(w) -> int:
    if w.model == "resnet20":
        return 2 * (3 * RESNET20_MACS - RESNET20_STEM_MACS) * w.B_loc * w.K
    d = w.widths
    f = 0
    for l in range(1, len(d)):
        mn = d[l - 1] * d[l]
        f += 2 * 2 * w.B_loc * mn                   # forward + weight grad
        if l > 1:
            f += 2 * w.B_loc * mn                   # input gradient
    return f * w.K


def source_digest(w) -> str:
    """Digest of the kernel sources a workload's dominant kernels come from."""
    files = (("kernels.h", "resnet.hip", "elementwise.hip") if w.model == "resnet20"
             else ("kernels.h", "gemm.hip", "elementwise.hip"))
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_1808_07217_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_for(tag: str, w):
    """HBM bytes per launch of the dominant kernel from the committed PMC
    summary, if it was taken on this workload, this tag and the current
    kernel sources."""
    try:
        with open(traffic_file(w.name)) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_digest") != source_digest(w) or t.get("tag") != tag:
        return None
    return t.get("bytes_per_launch")


# Kernels (as rocprofv3 names them, by name prefix) behind a launch tag: the
# MLP's persistent fused weight-gradient + update kernel, the ResNet's
# convolution families, and the K-way average, the copy-like kernel used to
# scale the counters.
TAG_KERNELS = {
    "wgrad_update": ("gemm_f32_sgd_ws<",),
    "average": ("k_average4<",),
    "conv_fwd": ("k_conv_stem_fwd", "k_conv_halo16<0>", "k_conv_rows<0,"),
    "conv_dgrad": ("k_conv_halo16<1>", "k_conv_rows<1,", "k_conv_dgrad_s2<"),
    "conv_wgrad": ("k_conv_wgrad_stem", "k_conv_wgrad_halo16", "k_conv_wgrad_band<"),
    "bn_bwd": ("k_bn_partial4", "k_bn_finalize_wg", "k_bn_bwd_apply4"),
    "bn_apply": ("k_bn_apply4<",),
}


def _counter_rows(path: str, counter: str) -> list:
    """[(kernel name, grid size, counter value in KiB)] per dispatch from
    one rocprofv3 --pmc pass (its *_counter_collection.csv)."""
    import csv
    import glob
    files = glob.glob(os.path.join(path, "**", "*counter_collection.csv"),
                      recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {path}")
    rows = []
    for f in files:
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] == counter:
                    rows.append((r["Kernel_Name"], int(r["Grid_Size"]),
                                 float(r["Counter_Value"])))
    return rows


def _short(name: str) -> str:
    """A kernel's name without its namespaces and parameter list."""
    name = name.replace("lsgd::(anonymous namespace)::", "").replace("lsgd::", "")
    if name.startswith("void "):
        name = name[5:]
    return name.split("(")[0]


def _family_bytes(rows, prefixes) -> tuple:
    """(dispatches, mean bytes per dispatch) over the kernels whose short
    name starts with one of the prefixes."""
    vals = [v for k, _, v in rows if any(_short(k).replace(" ", "").startswith(
        p.replace(" ", "")) for p in prefixes)]
    if not vals:
        raise SystemExit(f"no dispatch of {prefixes}")
    return len(vals), 1024.0 * sum(vals) / len(vals)


def write_traffic(pmc_dir: str, w, tag: str) -> dict:
    """HBM bytes per launch of a tag's kernels from two counter passes, each
    scaled by what the same counter reads for the K-way average of the
    replicas (the launch with the largest grid), whose traffic is known
    exactly (K Ps fp32 words read and written)."""
    fetch = _counter_rows(os.path.join(pmc_dir, "fetch"), "FETCH_SIZE")
    write = _counter_rows(os.path.join(pmc_dir, "write"), "WRITE_SIZE")

    def calib(rows):
        avg = [(g, v) for k, g, v in rows if _short(k).startswith("k_average4<")]
        gmax = max(g for g, _ in avg)
        vals = [v for g, v in avg if g == gmax]
        return 1024.0 * sum(vals) / len(vals)
    if w.model == "resnet20":
        P = resnet_param_count(w.widths[-1])
    else:
        P = sum(a * b + b for a, b in zip(w.widths[:-1], w.widths[1:]))
    Ps = (P + 63) // 64 * 64
    avg_bytes = 4.0 * w.K * Ps
    f_scale = avg_bytes / calib(fetch)
    w_scale = avg_bytes / calib(write)
    n_f, rd = _family_bytes(fetch, TAG_KERNELS[tag])
    n_w, wr = _family_bytes(write, TAG_KERNELS[tag])
    rd, wr = rd * f_scale, wr * w_scale
    out = {"tag": tag, "kernels": list(TAG_KERNELS[tag]), "workload": w.name,
           "source_digest": source_digest(w),
           "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4),
           "dispatches": n_f, "read_bytes_per_launch": round(rd),
           "write_bytes_per_launch": round(wr), "bytes_per_launch": round(rd + wr),
           "algorithmic_bytes_per_launch": round(kernel_cost(tag, w)[1])}
    with open(traffic_file(w.name), "w") as f:
        json.dump(out, f, indent=1)
    return out


def sweep():
    """Achieved bandwidth of the two HBM-bound building blocks against the
    working-set size. Sets up to ~256 MB can stay in the 256 MB Infinity
    Cache between repetitions, so only the larger sizes measure HBM itself.
    For reference, the same working sets through kernels this library did
    not write: torch's copy_ (read and write n floats) and add (two reads,
    one write), timed the same way."""
    import torch
    from paper_1808_07217_amd import lsgd as L
    dev = torch.device("cuda", 0)
    K = 16
    for mb in (64, 128, 256, 512, 1024, 2048, 4096):
        nbytes = mb << 20
        P = nbytes // (4 * K) // 64 * 64
        W = torch.randn(K, P, device=dev)
        reps = 20 if mb <= 1024 else 8
        L.replica_average(W)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            L.replica_average(W)
        e1.record()
        torch.cuda.synchronize()
        t_avg = e0.elapsed_time(e1) / reps / 1e3
        avg_bytes = 2 * K * P * 4                # read and write [K][P]
        del W
        n = nbytes // (3 * 4) // 64 * 64          # W, U, G of n floats
        Wt = torch.randn(n, device=dev)
        Ut = torch.zeros(n, device=dev)
        Gt = torch.randn(n, device=dev)
        L.sgd_update(Wt, Ut, Gt, 1e-3, 0.9, 1e-4)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            L.sgd_update(Wt, Ut, Gt, 1e-3, 0.9, 1e-4)
        e1.record()
        torch.cuda.synchronize()
        t_upd = e0.elapsed_time(e1) / reps / 1e3
        upd_bytes = 20 * n                        # read W, U, G; write W, U

        def ref(fn, nb):
            fn()
            torch.cuda.synchronize()
            e0.record()
            for _ in range(reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            t = e0.elapsed_time(e1) / reps / 1e3
            return {"us": round(t * 1e6, 2), "GB/s": round(nb / t / 1e9, 1),
                    "frac_hbm": round(nb / t / 1e9 / PEAK_HBM_GBS, 4)}
        torch_add = ref(lambda: torch.add(Wt, Gt, out=Ut), 12 * n)
        del Wt, Ut, Gt
        torch.cuda.empty_cache()
        nc = nbytes // (2 * 4) // 64 * 64          # source and copy of nc floats
        src = torch.randn(nc, device=dev)
        dst = torch.empty_like(src)
        torch_copy = ref(lambda: dst.copy_(src), 8 * nc)
        del src, dst
        torch.cuda.empty_cache()
        print(json.dumps({
            "working_set_MB": mb,
            "average": {"K": K, "P": P, "us": round(t_avg * 1e6, 2),
                        "GB/s": round(avg_bytes / t_avg / 1e9, 1),
                        "frac_hbm": round(avg_bytes / t_avg / 1e9 / PEAK_HBM_GBS, 4)},
            "sgd_update": {"n": n, "us": round(t_upd * 1e6, 2),
                           "GB/s": round(upd_bytes / t_upd / 1e9, 1),
                           "frac_hbm": round(upd_bytes / t_upd / 1e9 / PEAK_HBM_GBS, 4)},
            "torch_copy": torch_copy, "torch_add": torch_add,
        }), flush=True)


def cpu_baseline(w, X, y, w0, min_seconds: float = 10.0):
    """The CPU oracle (as it is) on a bounded sample of the workload, repeated
    until about `min_seconds` of CPU work: whole rounds (H local steps on all
    K replicas plus the synchronisation) where one takes a few seconds; one
    local step of replica 0 where a round would take minutes (ResNet-20, the
    2048-wide MLP). Timed with the host BLAS's own thread count, then again
    with one thread."""
    from oracle import lsgd_oracle as O
    try:
        import threadpoolctl
    except ImportError:
        threadpoolctl = None
    threads = None
    if threadpoolctl is not None:
        info = threadpoolctl.threadpool_info()
        threads = max((i.get("num_threads") or 1) for i in info) if info else 1
    per_step = w.model == "resnet20" or w.dtype == "bf16"
    if per_step:
        what = f"one local step of replica 0 ({w.B_loc} samples)"
        unit = w.B_loc
    elif w.Kb > 0:
        what = (f"one round: H^b={w.Hb} x (H={w.H} local steps on all K={w.K} replicas "
                f"+ block average over K'={w.Kb}) + global average")
        unit = w.K * w.H * w.Hb * w.B_loc
    else:
        what = (f"one round: H={w.H} local steps on all K={w.K} replicas + "
                + ("synchronisation with global momentum" if w.global_momentum
                   else f"{w.scheme} synchronisation" if w.scheme != "local"
                   else "average"))
        unit = w.K * w.H * w.Hb * w.B_loc

    def timed():
        st = O.State(w0, w.K)
        n = 0
        t0 = time.perf_counter()
        while True:
            if per_step:
                O.local_step(st, w, X, y, w.lr, replicas=[0])
            elif w.Kb > 0:
                O.run_hierarchical_round(st, w, X, y, w.H, w.Hb, w.Kb, w.lr)
            else:
                O.run_round(st, w, X, y, w.H, w.lr)
            n += 1
            dt = time.perf_counter() - t0
            if dt >= min_seconds:
                return n, dt

    n, dt = timed()
    out = {"value": n * unit / dt, "unit": "samples/s", "cores": threads,
           "host_cores": os.cpu_count(), "kind": "oracle",
           "sample": f"{n} x {what} of {w.name}: {n * unit} samples in {dt:.2f} s; "
                     f"fp64 numpy, BLAS threads={threads}, host cores={os.cpu_count()}"}
    if threadpoolctl is not None:
        with threadpoolctl.threadpool_limits(1):
            n1, dt1 = timed()
        out["single_thread"] = {"value": n1 * unit / dt1, "unit": "samples/s",
                                "cores": 1,
                                "sample": f"{n1} x {what}: {n1 * unit} samples in "
                                          f"{dt1:.2f} s on one BLAS thread"}
    return out


def main():
    args = parse()
    if args.sweep:
        sweep()
        return
    if args.traffic_from:
        import workloads as wk
        w = wk.get(args.workload)
        tag = args.traffic_tag or ("conv_wgrad" if w.model == "resnet20" else "wgrad_update")
        print(json.dumps(write_traffic(args.traffic_from, w, tag)))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU "
              "path (the K workers are replicas on one device)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import workloads as wk
    from paper_1808_07217_amd import lsgd as L

    w = wk.get(args.workload)
    X, y = wk.dataset(w)
    w0 = wk.initial_weights(w)
    dev = torch.device("cuda", 0)
    cfg = L.make_config(w.widths, w.K, w.B_loc, w.N, dtype=w.dtype,
                        momentum=w.momentum, weight_decay=w.weight_decay,
                        nesterov=w.nesterov, seed=w.sample_seed, model=w.model,
                        global_momentum=w.global_momentum, scheme=w.scheme,
                        sampler=w.sampler)
    Xd = torch.from_numpy(np.array(X)).to(dev)
    yd = torch.from_numpy(np.array(y)).to(dev)
    reps = L.Replicas(cfg, Xd, yd, torch.from_numpy(w0).to(dev))
    if args.lazy_average:
        reps.set_lazy_average(True)
        import dataclasses
        w = dataclasses.replace(w)
        object.__setattr__(w, "lazy_average", True)
    stream = reps.stream
    hier = w.Kb > 0
    H = w.H * w.Hb            # local steps per (outer) round
    lrs = [w.lr] * H
    max_steps = args.steps if args.steps is not None else MAX_AUTO_STEPS
    loss = torch.empty((args.warmup + max_steps + 8) * H, w.K, device=dev)

    def rnd(i):
        if hier:   # H^b x (H local steps, block average), global average
            reps.run_hierarchical_round(w.H, w.Hb, w.Kb, lrs,
                                        loss[i * H:(i + 1) * H])
        else:
            reps.run_round(lrs, loss[i * H:(i + 1) * H])

    # Warmup. The rounds after the first bracket every launch with HIP events
    # (per-kernel breakdown, and the dominant kernel); the timed rounds then
    # bracket a sample of the dominant kernel's launches (two per round for a
    # kernel launched once per step, every (n + 1)-th for a family of n
    # launches per step; each bracket costs the stream some microseconds), on
    # the stream it is launched on.
    timing = not args.no_kernel_timing and args.warmup >= 1
    prof_rounds = 0
    w0_ev, w1_ev = (torch.cuda.Event(enable_timing=True) for _ in range(2))
    for i in range(args.warmup):
        if timing and (i >= 1 or args.warmup == 1):
            reps.profile(True)
            prof_rounds += 1
        if i == args.warmup - 1:
            w0_ev.record(stream)
        rnd(i)
    w1_ev.record(stream)
    torch.cuda.synchronize()
    # one warmup round's time: the number of timed rounds (when not given)
    # and how sparsely events may sample them. An event record costs the
    # stream a few microseconds, so short rounds are bracketed only every
    # few rounds (events cost at most about 2% of the timed region).
    est_ms = max(w0_ev.elapsed_time(w1_ev), 1e-3) if args.warmup >= 1 else 1.0
    sparse = max(1, math.ceil(EVENT_GAP_MS / est_ms))
    steps = args.steps
    if steps is None:
        steps = 20 if est_ms >= 1.0 else min(MAX_AUTO_STEPS, max(20, math.ceil(100.0 / est_ms)))
    dom = None
    if timing:
        rep = reps.profile_report()
        reps.profile(False)
        per_round = {t: ms / prof_rounds for t, (n, ms) in rep.items()}
        dom = max(per_round, key=per_round.get)
        per_round_launches = rep[dom][0] // prof_rounds
        per_step = max(1, per_round_launches // H)
        if sparse > 1:
            every = per_round_launches * sparse
        elif per_step > 1:
            # a family of launches per local step (one per layer): every
            # (n + 1)-th cycles through all of them, so the sampled average
            # is the family's
            every = per_step + 1
        else:
            every = max(1, per_round_launches // 2)
        reps.profile_select(dom, every=every)
        reps.profile(True)
    torch.cuda.synchronize()
    # an event every `sparse` round boundaries: the total and the per-round
    # spread (blocks of `sparse` rounds)
    bounds = sorted(set(range(0, steps, sparse)) | {steps})
    evs = {b: torch.cuda.Event(enable_timing=True) for b in bounds}
    with torch.cuda.stream(stream):
        evs[0].record(stream)
        t0 = time.perf_counter()
        for i in range(steps):
            rnd(args.warmup + i)
            if i + 1 in evs:
                evs[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = evs[0].elapsed_time(evs[steps])
    round_ms = sorted(evs[a].elapsed_time(evs[b]) / (b - a)
                      for a, b in zip(bounds[:-1], bounds[1:]))
    phases = None
    if w.warm_rounds > 0:
        # post-local SGD: the H = 1 warm phase (one average per local step)
        # timed on its own; the headline above is the H-step phase
        nw = min(w.warm_rounds, 100)
        reps.profile(False)
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            p0 = torch.cuda.Event(enable_timing=True)
            p1 = torch.cuda.Event(enable_timing=True)
            p0.record(stream)
            tw = time.perf_counter()
            for _ in range(nw):
                reps.run_round([w.lr], loss[:1])
            p1.record(stream)
        torch.cuda.synchronize()
        ms_h1 = max(p0.elapsed_time(p1), (time.perf_counter() - tw) * 1e3) / nw
        phases = {"H1": {"rounds_timed": nw, "samples_per_round": w.K * w.B_loc,
                         "ms_per_round": round(ms_h1, 4),
                         "samples_per_s": round(w.K * w.B_loc / (ms_h1 / 1e3), 1)}}
    if timing:
        n, ms = reps.profile_report()[dom]
        reps.profile(False)
        reps.profile_select(None)
        avg_s = ms / n / 1e3
        flops, nbytes = kernel_cost(dom, w)
        if w.model == "resnet20" and flops is not None:
            # the step's algorithmic totals over the launches the library
            # makes per local step (it may split a layer's work, e.g. the
            # forward pass over two halves of the replicas)
            _, f_step, b_step = resnet_step_costs(w)[dom]
            lps = per_round_launches / H
            flops, nbytes = f_step / lps, b_step / lps
    ms_per_step = max(gpu_ms, wall * 1e3) / steps
    samples = w.K * H * w.B_loc
    value = samples / (ms_per_step / 1e3)
    l_all = loss[:(args.warmup + steps) * H].float().cpu().numpy()
    if not np.all(np.isfinite(l_all)):
        raise RuntimeError("non-finite loss in the benchmark run")

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "samples/s",
        "n_gpus": 1, "steps": steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": (f"{w.name}: MLP {'-'.join(map(str, w.widths))} "
                                if w.model == "mlp" else f"{w.name}: ResNet-20 ")
                               + f"{w.dtype}, K={w.K}, B_loc={w.B_loc}, "
                               + (f"K'={w.Kb}, H={w.H}, H^b={w.Hb}" if hier
                                  else f"H={H}"),
                   "K": w.K, "B_loc": w.B_loc, "H": H,
                   **({"K_block": w.Kb, "H_block": w.Hb} if hier else {}),
                   "samples_per_step": samples,
                   **({"average_form": "lazy"} if args.lazy_average else {}),
                   "momentum": w.momentum, "nesterov": w.nesterov,
                   "weight_decay": w.weight_decay,
                   **({"scheme": w.scheme} if w.scheme != "local" else {}),
                   **({"sampler": w.sampler} if w.sampler != "iid" else {}),
                   **({"global_momentum": w.global_momentum}
                      if w.global_momentum else {})},
    }
    if phases is not None:
        phases[f"H{H}"] = {"samples_per_round": samples,
                           "ms_per_round": round(ms_per_step, 4),
                           "samples_per_s": round(value, 1)}
        out["phases"] = phases
    out["round_ms"] = {"median": round(float(np.median(round_ms)), 4),
                       "min": round(round_ms[0], 4), "max": round(round_ms[-1], 4)}
    gemm_flops = gemm_flops_per_local_step(w) * H
    out["e2e_mfma_frac"] = round(gemm_flops / (ms_per_step / 1e3) /
                                 (PEAK_TFLOPS[w.dtype] * 1e12), 4)

    if timing and flops is not None:
        ridge = PEAK_TFLOPS[w.dtype] * 1e12 / (PEAK_HBM_GBS * 1e9)
        if nbytes and flops / nbytes < ridge:
            roof = {"bound": "hbm", "achieved": round(nbytes / avg_s / 1e9, 1),
                    "peak": PEAK_HBM_GBS, "unit": "GB/s"}
        else:
            roof = {"bound": "mfma",
                    "achieved": round(flops / avg_s / 1e12, 2),
                    "peak": PEAK_TFLOPS[w.dtype], "unit": "TFLOP/s"}
        roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
        roof["traffic"] = traffic_for(dom, w)
        roof["kernel"] = dom
        roof["avg_launch_us"] = round(avg_s * 1e6, 2)
        roof["launches_timed"] = n
        roof["algorithmic_bytes_per_launch"] = nbytes
        roof["algorithmic_flops_per_launch"] = flops
        out["roofline"] = roof
    if timing:
        # from the event-bracketed warmup rounds
        out["kernel_ms_per_step"] = {t: round(v, 4) for t, v in
                                     sorted(per_round.items(),
                                            key=lambda kv: -kv[1])}
        # matrix-core fraction of each GEMM-carrying launch tag (algorithmic
        # flops over its bracketed time, against the dtype's dense peak)
        mf = {}
        for t, ms in per_round.items():
            try:
                f, _ = kernel_cost(t, w)
            except ValueError:
                f = None
            if f and ms > 0:
                if w.model == "resnet20" and t in resnet_step_costs(w):
                    # the round's flops, however many launches carry them
                    f_round = resnet_step_costs(w)[t][1] * H
                else:
                    f_round = f * rep[t][0] / prof_rounds
                mf[t] = round(f_round / (ms / 1e3) / (PEAK_TFLOPS[w.dtype] * 1e12), 4)
        if mf:
            out["kernel_mfma_frac"] = mf
        if "average" in rep:   # the synchronisation kernel's own rate
            n_avg, ms_avg = rep["average"]
            _, by = kernel_cost("average", w)
            t_avg = ms_avg / n_avg / 1e3
            out["average_kernel"] = {
                "form": "lazy" if getattr(w, "lazy_average", False) else "broadcast",
                "avg_launch_us": round(t_avg * 1e6, 2),
                "algorithmic_bytes_per_launch": by,
                "GB/s": round(by / t_avg / 1e9, 1),
                "frac_hbm": round(by / t_avg / 1e9 / PEAK_HBM_GBS, 4)}
    reps.close()

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, X, y, w0)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
