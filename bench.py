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

# Peaks (MI355X, published / derived from unit counts, "Roofline"):
#   hbm   8 TB/s HBM3E
#   mfma  5.0 POP/s dense int8 matrix-core operations
#   alu   32-bit integer multiplies (v_mad_u64_u32 partial products), one per
#         lane per clock: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
PEAKS = {"hbm": (8000.0, "GB/s", 1e9), "mfma": (5000.0, "TOP/s", 1e12),
         "alu": (256 * 4 * 16 * 2.4, "Gmul/s", 1e9)}
MULS_PER_FIELD_MUL = 4      # 32x32 -> 64 partial products of a product in F_p, p = 2^61 - 1
X_TAIL_LOG, X_BLOCK_MAX, X_FUSE_MAX, MM_TAIL_LOG, MM_FUSE = 8, 10, 4, 10, 2


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


def x_schedule(lN):
    """Rounds over x per launch, as the library runs them: register passes of
    X_FUSE_MAX rounds, one pass of B rounds per workgroup in LDS (B = 0: none),
    and the last pass of v rounds."""
    v = min(lN, X_TAIL_LOG)
    rem, reg = lN - v, 0
    while rem - reg > X_BLOCK_MAX:
        reg += X_FUSE_MAX
    return [X_FUSE_MAX] * (reg // X_FUSE_MAX), rem - reg, v


def group_work(shapes, planes):
    """Algorithmic work per step of each kernel group: {group: (bound, amount)}
    with amount in bytes (hbm), int8 operations (mfma) or 32-bit multiplies
    (alu, 4 per field multiplication), plus the fold groups' HBM bytes."""
    w, hbm2 = {}, {}

    def add(g, bound, amt, d=w):
        b, a = d.get(g, (bound, 0))
        d[g] = (bound, a + amt)

    for (n, m, k, ab, _, relu), P in zip(shapes, planes):
        N = n * k
        # exact product on the matrix cores: LA x 2 int8 limb products of 2 n m k
        # operations.  int32 activations are the previous layer's ReLU outputs,
        # in [0, 2^24): their top limb plane is zero and the product skips it,
        # so three limbs are counted (a tile that needs the fourth does more
        # work than is counted here)
        LA = 2 if ab == 2 else 3
        add("gemm_mfma", "mfma", 2 * n * m * k * LA * 2)
        add("bind_rows", "hbm", n * m * ab + 8 * m)
        add("bind_cols", "hbm", m * k * 2 + 8 * m)
        # the fused front: both bindings read A and B once and write the eq
        # tables (its limb split reads them again; that is the product's work)
        add("matmul_front", "hbm", n * m * ab + m * k * 2 + 8 * (n + k))
        add("witness_minmax", "hbm", 8 * N)
        add("witness_rescale", "hbm", N * (8 + 4 + 2 + 4 + 4 + 8))  # C in; R, Rm, Y, Z, bits out
        # Gram matrix of the plane rounds: per output, tile pairs x 32 x 32 x 2 x 8 digits
        TP = 3 if P > 32 else 1
        add("range_plane", "mfma", N * TP * 1024 * 2 * 8)
        # rounds over x: per pair, 6 field products (range) and 7 (ReLU)
        lN = N.bit_length() - 1
        per_pair = 6 + 7 * relu
        regs, B, v = x_schedule(lN)
        j = 0
        for C in regs + ([B] if B else []):
            lS = lN - j
            for c in range(C):
                add("range_rounds", "alu", MULS_PER_FIELD_MUL * per_pair * (1 << (lS - c - 1)))
            rd = (8 + 8 * relu) if j == 0 else (8 + 16 * relu)
            add("range_rounds", "hbm", rd * (1 << lS) + (8 + 16 * relu) * (1 << (lS - C)), hbm2)
            j += C
        for jj in range(lN - j):
            add("range_tail", "alu", MULS_PER_FIELD_MUL * per_pair * (1 << (lN - j - jj - 1)))
        # matrix sum-check: per pair 3 products (X = 0, 1, 2) and 2 folds
        lm = m.bit_length() - 1
        for jj in range(lm):
            add("matmul_rounds" if lm - jj > MM_TAIL_LOG else "matmul_tail", "alu",
                MULS_PER_FIELD_MUL * 5 * (1 << (lm - jj - 1)))
    return w, hbm2


# Kernel -> group, for hardware-counter summaries (rocprofv3 kernel names).
KERNEL_GROUP = [("k_front", "matmul_front"), ("k_gemm_mfma", "gemm_mfma"), ("k_split", "gemm_mfma"),
                ("k_zero_i64", "gemm_mfma"),
                ("k_bind_rows", "bind_rows"), ("k_sum_chunks", "bind_rows"), ("k_bind_cols", "bind_cols"),
                ("k_minmax", "witness_minmax"), ("k_wit_params", "witness_minmax"),
                ("k_rescale", "witness_rescale"), ("k_claims_final", "witness_rescale"),
                ("k_plane_gram", "range_plane"), ("k_gram_reduce", "range_setup"),
                ("k_xrounds", "range_rounds"), ("k_xblock", "range_rounds"), ("k_range_setup", "range_setup"),
                ("k_rounds", "matmul_rounds"), ("k_tail", "matmul_tail"), ("k_eq_table", "eq_table"),
                ("k_assemble", "assemble")]
def traffic_file(cfg):
    return os.path.join(ROOT, "profiles", f"traffic_config{cfg}.json")


def sources_digest():
    """SHA-256 over the library sources: counters taken on other sources are stale."""
    import hashlib
    h = hashlib.sha256()
    for d in ("paper_2505_17623_amd/csrc", "include"):
        for f in sorted(os.listdir(os.path.join(ROOT, d))):
            with open(os.path.join(ROOT, d, f), "rb") as fh:
                h.update(f.encode() + fh.read())
    return h.hexdigest()


def traffic_of(group, cfg):
    """Measured HBM bytes per step of a kernel group (profiles/traffic_config<cfg>.json), or
    None when they were taken on other sources or another workload."""
    try:
        with open(traffic_file(cfg)) as fh:
            t = json.load(fh)
    except OSError:
        return None
    if t.get("sources_sha256") != sources_digest() or t.get("config") != cfg:
        return None
    return t["groups"].get(group)


def pmc_summary(fetch_csv, write_csv, cfg, steps_run, calib_mib):
    """HBM bytes per step and kernel group from two rocprofv3 --pmc runs
    (FETCH_SIZE, WRITE_SIZE; KiB per dispatch), each scaled by what the same
    counter reads for the plain copy of calib_mib MiB that bench.py makes with
    --copy-calibration."""
    import csv
    import collections
    out = {}
    for name, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        per_kernel = collections.defaultdict(list)
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] == name:
                per_kernel[r["Kernel_Name"]].append(float(r["Counter_Value"]))
        copies = [max(v) for k, v in per_kernel.items() if "copyBuffer" in k]
        factor = max(copies) / (calib_mib * 1024.0)
        groups = collections.defaultdict(float)
        for k, v in per_kernel.items():
            g = next((grp for pre, grp in KERNEL_GROUP if pre in k), None)
            if g:
                groups[g] += sum(v) / steps_run / factor * 1024.0  # bytes per step
        out[name] = (factor, dict(groups))
    groups = {g: round(out["FETCH_SIZE"][1].get(g, 0) + out["WRITE_SIZE"][1].get(g, 0))
              for g in set(out["FETCH_SIZE"][1]) | set(out["WRITE_SIZE"][1])}
    return dict(config=cfg, sources_sha256=sources_digest(), calibration_mib=calib_mib,
                fetch_factor=round(out["FETCH_SIZE"][0], 4), write_factor=round(out["WRITE_SIZE"][0], 4),
                groups=groups, fetch=out["FETCH_SIZE"][1], write=out["WRITE_SIZE"][1])


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
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=3, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after the timed region, copy a MIB-sized device buffer once (a plain copy kernel "
                         "of known size, to scale hardware byte counters)")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="summarise two rocprofv3 --pmc runs of this bench (FETCH_SIZE, WRITE_SIZE) into "
                         "profiles/traffic_config<C>.json and print it; no GPU work")
    args = ap.parse_args()
    if args.pmc_summary:
        steps_run = max(args.warmup, 1) + 4 * args.steps  # warmup, two sizing passes, timed, event-timed
        t = pmc_summary(args.pmc_summary[0], args.pmc_summary[1], args.config, steps_run,
                        args.copy_calibration or 256)
        with open(traffic_file(args.config), "w") as fh:
            json.dump(t, fh, indent=1)
        print(json.dumps(t, indent=1))
        return
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
    dev = torch.device("cuda:0")
    X = ra.to_device(wl.X, dev)
    Bs = [ra.to_device(Ly.B, dev) for Ly in wl.layers]
    torch.cuda.synchronize()
    ctx = ra.Context(seed=wl.challenge_seed)
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
    # Deferred outputs: a step is enqueued whole, and K steps are enqueued back
    # to back (each writes its own transcript words), so the host prepares the
    # next step while the device proves the current one.  Every layer keeps
    # its device outputs in `bufs` across steps.  Two untimed passes of K
    # steps size the pinned transcript area and the buffers.
    ctx.set_deferred(True)
    bufs = []
    for _ in range(2):
        outs = [ra.prove_network(ctx, wl, dev, X=X, Bs=Bs, ts=ts, bufs=bufs) for _ in range(args.steps)]
        ctx.sync()
        assert all([o["transcript"]["P"] for o in out] == planes for out in outs)

    # timed region: K steps enqueued back to back, completed by one sync
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    outs = [ra.prove_network(ctx, wl, dev, X=X, Bs=Bs, ts=ts, bufs=bufs) for _ in range(args.steps)]
    ctx.sync()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    elapsed = t1 - t0
    assert all(len(out[-1]["transcript"]["rs_evals"]) > 0 for out in outs)
    # the same K steps again with HIP events around every kernel group (recording
    # events adds host work between launches, so this pass is not the one timed)
    ctx.set_profiling(True)
    torch.cuda.synchronize()
    for i in range(args.steps):
        ra.prove_network(ctx, wl, dev, X=X, Bs=Bs, ts=ts, bufs=bufs)
    ctx.sync()
    torch.cuda.synchronize()
    prof = ctx.profile()
    ctx.set_profiling(False)
    ms_step = 1e3 * elapsed / args.steps
    el = elements_folded(shapes, planes)
    value = el * args.steps / elapsed

    # roofline of the dominant kernel group
    work, fold_bytes = group_work(shapes, planes)
    dom = max((g for g in prof if g in work), key=lambda g: prof[g][0])
    bound, amount = work[dom]
    peak, runit, scale = PEAKS[bound]
    dom_ms, dom_launches = prof[dom]
    dom_s_per_step = dom_ms / 1e3 / args.steps
    achieved = amount / dom_s_per_step / scale
    roofline = dict(kernel=dom, bound=bound, achieved=round(achieved, 2), peak=peak, unit=runit,
                    frac=round(achieved / peak, 4), traffic=traffic_of(dom, args.config),
                    launches_per_step=dom_launches / args.steps, ms_per_step=round(dom_ms / args.steps, 4))
    groups = {g: dict(ms_per_step=round(v[0] / args.steps, 4), launches_per_step=v[1] / args.steps)
              for g, v in sorted(prof.items(), key=lambda kv: -kv[1][0]) if v[1]}
    for g, d in groups.items():
        s_per = d["ms_per_step"] / 1e3
        if g in work and s_per > 0:
            b, a = work[g]
            pk, u, sc = PEAKS[b]
            d.update(bound=b, achieved=round(a / s_per / sc, 2), unit=u, frac=round(a / s_per / sc / pk, 4))
        if g in fold_bytes and s_per > 0:
            d["hbm_frac"] = round(fold_bytes[g][1] / s_per / 1e9 / PEAKS["hbm"][0], 4)

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
