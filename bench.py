"""Benchmark of the MI355X Range-Arithmetic prover.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config C] [--no-cpu-baseline]

One step proves every layer of a synthetic fixed-point workload (matrix
sum-check, rescale/ReLU witness, concatenated range sum-check, ReLU
zero-check) with its inputs already resident in HBM.  Prints one JSON line:
prover field elements folded per second (whole job), ms per step and per
layer, the roofline of the dominant kernel group (measured with HIP events on
the library's stream over the timed region) and the CPU oracle's rate on a
bounded sample of the same workload.

Elements folded: each sum-check round binds one variable of every witness
table of its instance (matrix: the two bound vectors of length m; range: the
bit table of P N entries; ReLU: R and Y of length N); a round over a table of
2^v entries consumes all of them, so one instance consumes 2^(v+1) - 2
entries per table over its v rounds.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# 32x32->64-bit integer multiply-adds (v_mad_u64_u32 / v_mad_i64_i32): one per
# lane per clock, 256 CUs x 64 lanes x 2.4 GHz ("ALU peak")
IMUL_PEAK_G = 256 * 64 * 2.4


def layer_shapes(wl):
    """(n, m, k, a_bytes, s, relu) per layer."""
    out = []
    n = wl.X.shape[0]
    for li, L in enumerate(wl.layers):
        m, k = L.B.shape
        if li > 0:
            link = wl.links[li]
            n = n if link is None else link.rows
        out.append((n, m, k, 2 if li == 0 else 4, L.s, int(L.relu)))
    return out


def elements_folded(shapes, planes):
    tot = 0
    for (n, m, k, _, _, relu), P in zip(shapes, planes):
        N = n * k
        tot += 2 * (2 * m - 2)            # matrix instance: a and b
        tot += 2 * P * N - 2              # range instance: the bit table
        if relu:
            tot += 2 * (2 * N - 2)        # ReLU instance: R and Y
    return tot


def add_instance(w, group, v, ntab, cmax, lt=10):
    """Global (multi-block) launches of one sum-check instance: each fused
    launch of C rounds reads the 2^lS-entry tables and writes 2^(lS-C)."""
    lS = v
    while lS > lt:
        C = min(cmax, lS - lt)
        b, a, u = w.get(group, ("hbm", 0, "GB"))
        w[group] = ("hbm", a + 8 * ntab * ((1 << lS) + (1 << (lS - C))), "GB")
        lS -= C


def add_xrounds(w, v, relu, lt=11, cmax=3):
    """Global launches of the rounds over x (range instance, and the ReLU
    zero-check in the same threads): the first launch reads Bx and the integer
    R, Y; every launch writes the bound tables (Bx, and D, S with ReLU) at
    2^-C of the size it read."""
    lS, first = v, True
    b, a, u = w.get("range_rounds", ("hbm", 0, "GB"))
    while lS > lt:
        C = min(cmax, lS - lt)
        rd = (8 + 8 * relu) if first else (8 + 16 * relu)
        a += rd * (1 << lS) + (8 + 16 * relu) * (1 << (lS - C))
        lS -= C
        first = False
    w["range_rounds"] = ("hbm", a, "GB")


def group_work(shapes, planes):
    """Algorithmic work per step of each kernel group: (bound, amount, unit)."""
    w = {}

    def add(g, bound, amt, unit):
        b, a, u = w.get(g, (bound, 0, unit))
        w[g] = (bound, a + amt, u)

    for (n, m, k, ab, _, relu), P in zip(shapes, planes):
        N = n * k
        add("gemm_mfma", "mfma", 2 * n * m * k, "GOP")                # 2 n m k integer ops (algorithmic)
        add("bind_rows", "hbm", n * m * ab + 8 * m, "GB")
        add("bind_cols", "hbm", m * k * 2 + 8 * m, "GB")
        add("witness_minmax", "hbm", 8 * N, "GB")
        add("witness_rescale", "hbm", N * (8 + 4 + 2 + 4 + 4 + 8), "GB")  # C in; R, Rm, Y, Z, bits out
        add("range_plane", "hbm", N * (8 + 8), "GB")                    # bits in; Bx out
        add_xrounds(w, N.bit_length() - 1, relu)
        add_instance(w, "matmul_rounds", m.bit_length() - 1, 2, 2)
    return w


def cpu_baseline(cfg):
    """The oracle (single thread) on a bounded sample of the same workload."""
    from oracle import oracle as orc
    from paper_2505_17623_amd import inputs
    if cfg == 3:
        wl, sample = inputs.cfg3(n=512), "one 512x512x512 layer of the same distribution (s=12, ReLU)"
    elif cfg == 5:
        wl, sample = inputs.cfg5(batch=64, d=1024), "MLP 1024-1024-1024 at batch 64, same distribution (s=12)"
    elif cfg == 4:
        wl, sample = inputs.cfg4(batch=4, H=32), "the same CNN at batch 4"
    else:
        wl, sample = inputs.workload(cfg, "full"), "the full workload"
    orc.build(force=False)
    t0 = time.perf_counter()
    res = orc.prove_network(wl)
    dt = time.perf_counter() - t0
    shapes = layer_shapes(wl)
    el = elements_folded(shapes, [r["P"] for r in res])
    return dict(value=el / dt, unit="field elements folded/s", cores=1, kind="oracle",
                sample=f"{sample}; {el} elements in {dt:.2f} s")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=3, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after the timed region, copy a MIB-sized device buffer once (a plain copy kernel "
                         "of known size, to scale hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this prover runs on one GPU; --gpus {args.gpus} is not supported "
              f"(sharding is described in DESIGN.md but not built)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2505_17623_amd import inputs, ra

    torch.cuda.set_device(0)
    wl = inputs.workload(args.config, "full")
    L = len(wl.layers)
    steps_total = max(args.warmup, 1) + 2 * args.steps + 2
    chal = inputs.xorshift64_stream(inputs.CHALLENGE_SEED_BASE + args.config,
                                    inputs.CHALLENGES_PER_LAYER * L * steps_total)
    dev = torch.device("cuda:0")
    X = ra.to_device(wl.X, dev)
    Bs = [ra.to_device(Ly.B, dev) for Ly in wl.layers]
    torch.cuda.synchronize()
    ctx = ra.Context(chal)
    shapes = layer_shapes(wl)
    print(f"# workload: {wl.name}; layers {shapes}", file=sys.stderr, flush=True)

    # warmup: synchronous calls; the first step fixes each layer's range
    # parameter t, which the later steps pass in so that no call has to wait
    # for the device before the whole step is enqueued (deferred outputs)
    first = None
    for i in range(max(args.warmup, 1)):
        out = ra.prove_network(ctx, wl, dev, X=X, Bs=Bs)
        if first is None:
            first = [o["transcript"] for o in out]
        print(f"# warmup step {i} done", file=sys.stderr, flush=True)
    planes = [tr["P"] for tr in first]
    ts = [tr["t"] for tr in first]
    ctx.set_deferred(True)
    out = ra.prove_network(ctx, wl, dev, X=X, Bs=Bs, ts=ts)
    ctx.sync()
    assert [o["transcript"]["P"] for o in out] == planes

    # timed region: K steps, each enqueued whole and completed by one sync
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        out = ra.prove_network(ctx, wl, dev, X=X, Bs=Bs, ts=ts)
        ctx.sync()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    elapsed = t1 - t0
    # the same K steps again with HIP events around every kernel group (recording
    # events adds host work between launches, so this pass is not the one timed)
    ctx.set_profiling(True)
    torch.cuda.synchronize()
    for i in range(args.steps):
        ra.prove_network(ctx, wl, dev, X=X, Bs=Bs, ts=ts)
        ctx.sync()
    torch.cuda.synchronize()
    prof = ctx.profile()
    ctx.set_profiling(False)
    ms_step = 1e3 * elapsed / args.steps
    el = elements_folded(shapes, planes)
    value = el * args.steps / elapsed

    # roofline of the dominant kernel group
    work = group_work(shapes, planes)
    dom = max((g for g in prof if g in work), key=lambda g: prof[g][0])
    bound, amount, unit = work[dom]
    dom_ms, dom_launches = prof[dom]
    dom_s_per_step = dom_ms / 1e3 / args.steps
    if bound == "hbm":
        achieved, peak, runit = amount / dom_s_per_step / 1e9, HBM_PEAK_GBS, "GB/s"
    else:
        achieved, peak, runit = amount / dom_s_per_step / 1e9, IMUL_PEAK_G, "Gimul/s"
    roofline = dict(kernel=dom, bound=bound, achieved=round(achieved, 2), peak=peak, unit=runit,
                    frac=round(achieved / peak, 4), traffic=None,
                    launches_per_step=dom_launches / args.steps, ms_per_step=round(dom_ms / args.steps, 4))
    groups = {g: dict(ms_per_step=round(v[0] / args.steps, 4), launches_per_step=v[1] / args.steps)
              for g, v in sorted(prof.items(), key=lambda kv: -kv[1][0]) if v[1]}
    for g, d in groups.items():
        if g in work:
            b, a, u = work[g]
            s_per = d["ms_per_step"] / 1e3
            if s_per > 0:
                d["achieved"] = round(a / s_per / 1e9, 2)
                d["unit"] = "GB/s" if b == "hbm" else "Gimul/s"
                d["frac"] = round(d["achieved"] / (HBM_PEAK_GBS if b == "hbm" else IMUL_PEAK_G), 4)

    if args.copy_calibration:
        src = torch.empty(args.copy_calibration << 20, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args.config)
        cpu["value"] = round(cpu["value"], 1)

    rec = dict(metric="prover field-elements folded/sec (HBM GB/s vs peak) + ms per layer proof",
               value=round(value, 1), unit="field elements folded/s", n_gpus=1, steps=args.steps,
               warmup=args.warmup, ms_per_step=round(ms_step, 4), ms_per_layer=round(ms_step / L, 4),
               higher_is_better=True, scaling="weak", vs_baseline=None, dtype="u64 (F_p, p=2^61-1)",
               data="synthetic",
               config=dict(workload=f"config {args.config}: {wl.name}", layers=L,
                           shapes=[list(s[:3]) for s in shapes], planes=planes,
                           elements_folded_per_step=el),
               roofline=roofline, cpu_baseline=cpu, kernel_groups=groups)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
