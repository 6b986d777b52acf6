#!/usr/bin/env python
"""Group-attention forward throughput on one MI355X.

One step = one whole group-attention forward (grouping rounds, aggregation,
group softmax + combine) over one batch of synthetic input already resident in
HBM.  Two input sets alternate so consecutive steps do not hit in the 256 MB
last-level cache.  Prints one JSON line: throughput, the roofline of the dominant
kernel, the CPU oracle timed on a sample, per-kernel times, and the merge plan
and backward pass of the same grouping timed on their own.
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

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
MFMA_BF16_PEAK_TFS = 2500.0  # MI355X dense bf16 MFMA
METRIC = "group-attention queries/sec (B·H·n) at n=8000,N=128; % HBM roofline"


def kernel_work(name, w, N, BH, iters=None):
    """(bound, algorithmic work per launch, unit, peak) of each kernel, or None.

    Bytes count only what the method itself reads and writes (no |k| bounds,
    previous groups or other state of this implementation):

    lloyd:     the persistent grouping launch (every Lloyd round, the update
               and the value sums): per key T reads of its row of K (one per
               round: a slice's keys do not fit on chip across rounds), one
               read of its row of V and one write of its group,
               (T + 1) d*es + 4 bytes.  The per-group outputs (centroids,
               counts, value means: N (6 d + 8) bytes per slice, under 0.5 %)
               are left out.  Each round's 2 N d flop per d*es bytes of K
               (128 flop/B at N = 128) is below MI355X's ridge (2.5 PF / 8 TB/s
               = 312 flop/B), so the roofline that bounds it is HBM.
    assign, assign_first: one round of the launch-per-round path: per key its
               row of K (read) and its group (written), d*es + 4 bytes.
    attend:    Q read + O write, 2 n d storage elements per slice (4 N d flop
               per query is below the ridge too).
    sums_full, valuesum: one pass over K (or V) and the groups, n (d*es + 4).
    """
    es = 2 if w.dtype == "bf16" else 4
    n, d = w.n, w.d
    T = w.iters if iters is None else iters
    if name == "lloyd":
        return "hbm", ((T + 1) * d * es + 4) * n * BH / 1e9, "GB/s", HBM_PEAK_GBS
    if name in ("assign", "assign_first"):
        return "hbm", (d * es + 4) * n * BH / 1e9, "GB/s", HBM_PEAK_GBS
    if name == "attend":
        return "hbm", 2.0 * n * d * es * BH / 1e9, "GB/s", HBM_PEAK_GBS
    if name in ("sums_full", "valuesum", "update"):
        return "hbm", 1.0 * n * (d * es + 4) * BH / 1e9, "GB/s", HBM_PEAK_GBS
    if name in ("proj_qkv", "proj_out"):
        # dense contractions over D = 64 H: 2 M Dout D flop, M = B n tokens
        H = BH // w.B
        D = 64 * H
        dout = 3 * D if name == "proj_qkv" else D
        return "mfma", 2.0 * w.B * n * dout * D / 1e12, "TFLOP/s", MFMA_BF16_PEAK_TFS
    return None


# the sources a kernel is built from (its recorded counter traffic holds while they are unchanged)
KERNEL_SOURCES = {"lloyd": ("ga_lloyd.hip", "ga_device.h")}
DEFAULT_SOURCES = ("ga_kernels.hip", "ga_device.h")


def kernel_source_digest(kernel):
    h = hashlib.sha256()
    for f in KERNEL_SOURCES.get(kernel, DEFAULT_SOURCES):
        with open(os.path.join(ROOT, "paper_2306_01926_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def traffic_for(kernel, workload):
    """Measured HBM bytes per launch from a committed rocprofv3 counter summary,
    or None if there is none or the kernel's sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_sha256") != kernel_source_digest(kernel):
        return None
    return rec.get("hbm_bytes_per_launch")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    # the GPU's clocks take some 10-40 ms of sustained load to settle: the
    # default warm-up covers that for the forward (about 12 ms)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="n8000_N128_bf16")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--N", type=int, default=None,
                    help="group count (default: the workload's, or its draw for call 0 when it varies)")
    ap.add_argument("--cpu-slices", type=int, default=256, help="(b,h) slices the oracle times (both input sets)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run an elementwise copy of this many MiB (a known-size kernel for HBM counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU: group attention runs here on a single MI355X "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE={world}); every (batch, head) slice is independent, "
              f"so batches and heads shard across GPUs without communication.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2306_01926_amd import ga, inputs

    if args.workload in inputs.BLOCK_WORKLOADS:
        return bench_block(args)
    dev = torch.device("cuda:0")
    w = inputs.WORKLOADS[args.workload]
    N = args.N if args.N is not None else inputs.draw_group_count(w, args.seed, 0)
    if w.N is not None and N != w.N:
        print(f"bench.py: workload {w.name} has N={w.N}; --N {N} applies only to a workload whose N varies",
              file=sys.stderr)
        sys.exit(2)
    if w.N is None and N not in w.N_choices:
        print(f"bench.py: N={N} is not one of {w.name}'s group counts {w.N_choices}", file=sys.stderr)
        sys.exit(2)
    BH = w.B * w.H
    scale = 1.0 / math.sqrt(w.d)
    print(f"bench: workload {w.name} B={w.B} H={w.H} n={w.n} d={w.d} N={N} iters={w.iters} {w.dtype}",
          file=sys.stderr, flush=True)
    host_sets = [inputs.workload_inputs(w, args.seed + k) for k in range(2)]
    digests = [{name: inputs.sha256(t) for name, t in zip("QKV", hs)} for hs in host_sets]
    sets = [tuple(t.to(dev) for t in s) for s in host_sets]
    outs = [torch.empty_like(s[0]) for s in sets]
    ws = ga.workspace(ga.shape_of(sets[0][0]), N, dev)[0]

    def step(k):
        Q, K, V = sets[k % 2]
        ga.forward(Q, K, V, N, w.iters, scale, out=outs[k % 2], ws=ws)

    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()

    # timed region: K whole-forward steps, events on the launch stream
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for k in range(args.steps):
        step(k)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / args.steps

    # same steps again with every kernel launch bracketed by hipEvents
    ga.timing_enable(True)
    t0.record()
    for k in range(args.steps):
        step(k)
    t1.record()
    torch.cuda.synchronize()
    ga.timing_enable(False)
    per_kernel = ga.timing_collect()
    ms_timed = t0.elapsed_time(t1) / args.steps

    # the adaptive scheduler's merge plan of the same grouping (run once per
    # training step, outside the forward): timed on its own
    sched = None
    if w.dtype == "bf16" and N <= 256:
        Q0, K0, V0 = sets[0]
        _, bel0, cnt0, cen0 = ga.forward(Q0, K0, V0, N, w.iters, scale, return_groups=True, ws=ws)
        for _ in range(2):
            ga.merge_plan(Q0, K0, bel0, cen0, cnt0, N, scale, 2.0)
        torch.cuda.synchronize()
        ga.timing_enable(True)
        for _ in range(args.steps):
            plan = ga.merge_plan(Q0, K0, bel0, cen0, cnt0, N, scale, 2.0)
        torch.cuda.synchronize()
        ga.timing_enable(False)
        tk = ga.timing_collect()  # merge_zero, merge_norms, merge_pairs per call
        avg = sum(t for _, t in tk.values()) / args.steps
        # algorithmic bytes: Q and K rows, the groups, the centroids and counts read once
        mbytes = BH * (w.n * (2 * w.d * 2 + 4) + N * (w.d * 4 + 4))
        sched = dict(kernel="merge_plan", launches={k: t / l for k, (l, t) in tk.items()}, eps=2.0, avg_ms=avg,
                     bound="hbm", achieved=mbytes / (avg / 1e3) / 1e9,
                     peak=HBM_PEAK_GBS, unit="GB/s", frac=mbytes / (avg / 1e3) / 1e9 / HBM_PEAK_GBS,
                     merges_min=int(plan["merges"].min()), next_N=ga.next_group_count(N, plan["merges"], 0.5))

    # the backward pass (gradient with the grouping fixed) of the same forward
    bwd = None
    if w.dtype == "bf16" and N <= 128:
        Q0, K0, V0 = sets[0]
        _, bel0, cnt0, cen0 = ga.forward(Q0, K0, V0, N, w.iters, scale, return_groups=True, ws=ws)
        vs0 = ga.aggregate(V0, bel0, N, ws=ws)
        dO = torch.randn(Q0.shape, device=dev).to(torch.bfloat16)
        bws = torch.empty(ga.backward_workspace_bytes(ga.shape_of(Q0), N), dtype=torch.uint8, device=dev)
        for _ in range(250):  # untimed: about 50 ms for the clocks to settle on the backward's launches
            ga.backward(Q0, dO, bel0, cen0, cnt0, vs0, N, scale, ws=bws)
        torch.cuda.synchronize()
        t0.record()
        for _ in range(args.steps):
            ga.backward(Q0, dO, bel0, cen0, cnt0, vs0, N, scale, ws=bws)
        t1.record()
        torch.cuda.synchronize()
        bms = t0.elapsed_time(t1) / args.steps
        ga.timing_enable(True)
        for _ in range(args.steps):
            ga.backward(Q0, dO, bel0, cen0, cnt0, vs0, N, scale, ws=bws)
        torch.cuda.synchronize()
        ga.timing_enable(False)
        tk = ga.timing_collect()
        # algorithmic bytes: read q and dO, write dQ (3 rows per query); read
        # the group and write dK and dV (4 B + 2 rows per key)
        bbytes = BH * w.n * (3 * w.d * 2 + 4 + 2 * w.d * 2)
        bwd = dict(ms=bms, launches={k: t / l for k, (l, t) in tk.items()}, bound="hbm",
                   achieved=bbytes / (bms / 1e3) / 1e9, peak=HBM_PEAK_GBS, unit="GB/s",
                   frac=bbytes / (bms / 1e3) / 1e9 / HBM_PEAK_GBS, queries_per_s=BH * w.n / (bms / 1e3))

    queries = BH * w.n
    es = 2 if w.dtype == "bf16" else 4
    compulsory = 4.0 * queries * w.d * es  # read Q, K, V once, write O once
    value = queries / (ms / 1e3)
    pct_hbm = compulsory / (ms / 1e3) / (HBM_PEAK_GBS * 1e9)

    kernels = {}
    for name, (launches, tot) in per_kernel.items():
        avg = tot / launches
        kernels[name] = dict(launches_per_step=launches / args.steps, avg_ms=avg)
        kw = kernel_work(name, w, N, BH)
        if kw:
            bound, work, unit, peak = kw
            ach = work / (avg / 1e3)
            kernels[name].update(bound=bound, achieved=ach, unit=unit, frac=ach / peak)
    # the dominant kernel: most time per step among those with a defined roofline
    dom = max((k for k in per_kernel if "frac" in kernels[k]), key=lambda k: per_kernel[k][1])
    kd = kernels[dom]
    _, work, _, peak = kernel_work(dom, w, N, BH)
    roofline = dict(scope="dominant kernel of the step", kernel=dom, bound=kd["bound"],
                    achieved=round(kd["achieved"], 3), peak=peak, unit=kd["unit"],
                    frac=round(kd["frac"], 4), traffic=traffic_for(dom, w.name),
                    avg_launch_ms=round(kd["avg_ms"], 5))

    if args.copy_calibration_mib:
        # int32 x + 0: one elementwise kernel that reads and writes exactly this many bytes
        nel = args.copy_calibration_mib * (1 << 20) // 4
        src = torch.arange(nel, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.add(src, 0, out=dst)
        torch.cuda.synchronize()
        del src, dst

    # parity spot-check and CPU baseline on a bounded sample of slices (oracle)
    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        import oracle

        # the first --cpu-slices (b,h) slices, input set 0 first, then set 1
        S = max(1, min(args.cpu_slices, 2 * BH))
        take = [min(S, BH), S - min(S, BH)]
        threads = oracle.threads()
        flat = lambda t, s: t.reshape(1, BH, w.n, w.d)[:, :s]
        cpu_s, mism, cen_ok, num, den = 0.0, 0, True, 0.0, 0.0
        for k, s in enumerate(take):
            if s == 0:
                continue
            Qs, Ks, Vs = (inputs.as_float64(flat(t, s)) for t in host_sets[k])
            c0 = time.perf_counter()
            ref = oracle.forward(Qs, Ks, Vs, N, w.iters, scale, w.dtype)
            cpu_s += time.perf_counter() - c0
            O, bel, cnt, cen = ga.forward(*sets[k], N, w.iters, scale, return_groups=True, ws=ws)
            torch.cuda.synchronize()
            bel = bel.reshape(1, BH, w.n)[:, :s].cpu().numpy()
            Og = O.reshape(1, BH, w.n, w.d)[:, :s].float().cpu().numpy().astype(np.float64)
            mism += int((bel != ref["belong"]).sum())
            cen_ok &= bool(np.array_equal(cen.reshape(1, BH, N, w.d)[:, :s].cpu().numpy(), ref["centroid"]))
            num, den = max(num, float(np.abs(Og - ref["O"]).max())), max(den, float(np.abs(ref["O"]).max()))
            del Qs, Ks, Vs, ref, O, bel, cnt, cen, Og
        cpu = dict(value=S * w.n / cpu_s, unit="queries/s", cores=threads, kind="oracle",
                   sample=f"{take[0]} + {take[1]} (b,h) slices of input sets 0 + 1 (of {BH} each) at full n={w.n}, "
                          f"all {w.iters} grouping rounds + aggregation + attention, fp64, {cpu_s:.1f} s wall on "
                          f"{threads} threads")
        parity = dict(slices=S, assign_mismatches=mism, centroid_bit_exact=cen_ok, out_max_rel_err=num / den)

    line = {
        "metric": METRIC, "value": value, "unit": "queries/s",
        # the headline: the whole forward against the HBM roofline of its compulsory bytes
        # (read Q, K, V once, write O once), target 0.5; "roofline" below is one kernel's
        "pct_hbm_roofline": pct_hbm, "target_pct_hbm_roofline": 0.5, "compulsory_bytes": compulsory,
        "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "n": w.n, "d": w.d, "N": N, "iters": w.iters,
                   "input_sets": 2},
        "input_sha256": digests,
        # every contraction of the forward (T assign rounds, scores, combine): 2 N d (T + 2) flop per query
        "mfma_frac_of_step": 2.0 * N * w.d * (w.iters + 2) * queries / (ms / 1e3) / (MFMA_BF16_PEAK_TFS * 1e12),
        "roofline": roofline, "cpu_baseline": cpu,
        "kernels": kernels, "ms_per_step_with_kernel_events": ms_timed, "parity_sample": parity,
        "scheduler": sched, "backward": bwd,
    }
    print(json.dumps(line), flush=True)


def per_kernel_report(per_kernel, steps, w, N, BH):
    kernels = {}
    for name, (launches, tot) in per_kernel.items():
        avg = tot / launches
        kernels[name] = dict(launches_per_step=launches / steps, avg_ms=avg)
        kw = kernel_work(name, w, N, BH)
        if kw:
            bound, work, unit, peak = kw
            ach = work / (avg / 1e3)
            kernels[name].update(bound=bound, achieved=ach, unit=unit, frac=ach / peak)
    return kernels


def bench_block(args):
    """Attention block (projections, group attention, output projection) on
    token embeddings X [B, n, 64 H]: one step = one ga_attention_block."""
    import types

    import numpy as np
    import torch

    from paper_2306_01926_amd import ga, inputs

    dev = torch.device("cuda:0")
    bw = inputs.BLOCK_WORKLOADS[args.workload]
    w = types.SimpleNamespace(B=bw.B, n=bw.n, d=64, dtype="bf16", iters=bw.iters)
    BH = bw.B * bw.H
    print(f"bench: attention block {bw.name} B={bw.B} n={bw.n} H={bw.H} D={bw.D} N={bw.N} iters={bw.iters} bf16",
          file=sys.stderr, flush=True)
    host = [inputs.block_inputs(bw.B, bw.n, bw.H, args.seed + k) for k in range(2)]
    sets = [tuple(t.to(dev) for t in s) for s in host]
    outs = [torch.empty_like(s[0]) for s in sets]
    ws = torch.empty(ga.block_workspace_bytes(ga.block_shape(sets[0][0], bw.H), bw.N), dtype=torch.uint8,
                     device=dev)

    def step(k):
        X, Wqkv, Wo = sets[k % 2]
        ga.attention_block(X, Wqkv, Wo, bw.H, bw.N, bw.iters, 0.125, out=outs[k % 2], ws=ws)

    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for k in range(args.steps):
        step(k)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / args.steps
    ga.timing_enable(True)
    for k in range(args.steps):
        step(k)
    torch.cuda.synchronize()
    ga.timing_enable(False)
    per_kernel = ga.timing_collect()
    kernels = per_kernel_report(per_kernel, args.steps, w, bw.N, BH)
    dom = max((k for k in per_kernel if "frac" in kernels[k]), key=lambda k: per_kernel[k][1])
    kd = kernels[dom]
    roofline = dict(scope="dominant kernel of the step", kernel=dom, bound=kd["bound"],
                    achieved=round(kd["achieved"], 3), peak=kernel_work(dom, w, bw.N, BH)[3], unit=kd["unit"],
                    frac=round(kd["frac"], 4),
                    traffic=traffic_for(dom, bw.name), avg_launch_ms=round(kd["avg_ms"], 5))
    tokens = bw.B * bw.n
    flops = 2.0 * tokens * 4 * bw.D * bw.D + 2.0 * BH * bw.n * bw.N * 64 * (bw.iters + 2)

    cpu = parity = None
    if not args.no_cpu_baseline:
        import oracle

        X0, W0, O0 = (inputs.as_float64(t) for t in host[0])
        threads = oracle.threads()
        nb = bw.B  # every batch of input set 0
        c0 = time.perf_counter()
        ref = oracle.attention_block(X0[:nb], W0, O0, bw.H, bw.N, bw.iters, 0.125)
        cpu_s = time.perf_counter() - c0
        cpu = dict(value=nb * bw.n / cpu_s, unit="tokens/s", cores=threads, kind="oracle",
                   sample=f"batches 0..{nb - 1} of {bw.B} ({nb * bw.n} tokens, {bw.H} heads each): fp64 projections, "
                          f"all {bw.iters} grouping rounds, aggregation, attention, output projection; {cpu_s:.1f} s "
                          f"wall on {threads} threads")
        step(0)
        torch.cuda.synchronize()
        Yg = outs[0][:nb].float().cpu().numpy().astype(np.float64)
        parity = dict(batches=nb, out_max_rel_err=float(np.abs(Yg - ref["Y"]).max() / np.abs(ref["Y"]).max()))

    line = {
        "metric": "attention-block tokens/sec (B·n) at n=4000, d_model=512, H=8, N=128", "value": tokens / (ms / 1e3),
        "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": bw.name, "B": bw.B, "n": bw.n, "H": bw.H, "d_model": bw.D, "N": bw.N,
                   "iters": bw.iters, "input_sets": 2},
        "mfma_frac_of_step": flops / (ms / 1e3) / (MFMA_BF16_PEAK_TFS * 1e12),
        "roofline": roofline, "cpu_baseline": cpu, "kernels": kernels, "parity_sample": parity,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
