"""Benchmark of the MI355X Range-Arithmetic prover.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config C] [--no-cpu-baseline]

Default workload: config 5, two 512x4096x4096 layers (the transformer-block
MLP at batch 512, s = 12, ReLU after the first), the largest configuration
and the one the headline is quoted on.

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
import gc
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
    """Algorithmic work per step of each kernel group, as the method defines
    it (not the dense work an implementation does instead):
    {group: {"bound": b, "amount": a, "secondary": (b2, a2) or None}}.
      gemm_mfma      the exact product C = A B: 2 n m k integer operations,
                     priced at the dense int8 MFMA peak it runs on
                     (secondary: the int8 limb products it actually issues);
      matmul_front   HBM bytes: A and B read once (2 or 4 B per entry), the
                     eq tables written;
      range_plane    HBM bytes of the plane rounds: the packed bit table in
                     (P N / 8 B) and the plane-bound table Bx out (8 N B)
                     (secondary: the int8 MFMA operations of the Gram matrix's
                     16 x 16 tiles on and above the diagonal);
      range_rounds   HBM bytes of the register/LDS passes over x: each pass
                     reads its input tables and writes the folded ones
                     (secondary: 32-bit multiplies, 4 per field product);
      range_tail, matmul_rounds, matmul_tail  32-bit multiplies (latency-bound
                     passes over small tables);
      witness_*      HBM bytes (only when the witness is not fused)."""
    w = {}

    def add(g, bound, amt, sec=None):
        d = w.setdefault(g, {"bound": bound, "amount": 0, "secondary": None})
        d["amount"] += amt
        if sec:
            b2, a2 = d["secondary"] or (sec[0], 0)
            d["secondary"] = (b2, a2 + sec[1])

    for (n, m, k, ab, _, relu), P in zip(shapes, planes):
        N = n * k
        # int32 activations are the previous layer's ReLU outputs, in [0, 2^24):
        # their top limb plane is zero and the product skips it (three limbs)
        LA = 2 if ab == 2 else 3
        add("gemm_mfma", "mfma", 2 * n * m * k, ("mfma", 2 * n * m * k * LA * 2))
        add("bind_rows", "hbm", n * m * ab + 8 * m)
        add("bind_cols", "hbm", m * k * 2 + 8 * m)
        add("matmul_front", "hbm", n * m * ab + m * k * 2 + 8 * (n + k))
        add("witness_minmax", "hbm", 8 * N)
        add("witness_rescale", "hbm", N * (8 + 4 + 2 + 4 + 4 + 8))  # C in; R, Rm, Y, Z, bits out
        tiles = 10 if P > 32 else 3  # 16 x 16 tiles on and above the Gram matrix's diagonal
        add("range_plane", "hbm", P * N // 8 + 8 * N, ("mfma", N * tiles * 256 * 2 * 8))
        # rounds over x: per pair, 6 field products (range) and 7 (ReLU); each
        # pass reads Bx (and R, Y as int32 in the first, D and S after) and
        # writes them folded to 2^-C of their size
        lN = N.bit_length() - 1
        per_pair = 6 + 7 * relu
        regs, B, v = x_schedule(lN)
        j = 0
        for C in regs + ([B] if B else []):
            lS = lN - j
            muls = sum(MULS_PER_FIELD_MUL * per_pair * (1 << (lS - c - 1)) for c in range(C))
            rd = (8 + 8 * relu) if j == 0 else (8 + 16 * relu)
            add("range_rounds", "hbm", rd * (1 << lS) + (8 + 16 * relu) * (1 << (lS - C)), ("alu", muls))
            j += C
        for jj in range(lN - j):
            add("range_tail", "alu", MULS_PER_FIELD_MUL * per_pair * (1 << (lN - j - jj - 1)))
        # matrix sum-check: per pair 3 products (X = 0, 1, 2) and 2 folds
        lm = m.bit_length() - 1
        for jj in range(lm):
            add("matmul_rounds" if lm - jj > MM_TAIL_LOG else "matmul_tail", "alu",
                MULS_PER_FIELD_MUL * 5 * (1 << (lm - jj - 1)))
    return w


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


# the sources of the kernels a headline step launches (the F_p path) and of
# their launchers: counters taken on other versions of these are stale
HEADLINE_SOURCES = ["witness.hip", "gemm.hip", "sumcheck.hip", "planes.hip", "xrounds.hip", "m61.hpp",
                    "common.hpp", "gram_reduce.hpp", "plane_round.hpp", "xsetup.hpp", "assemble.hpp", "claims.hpp",
                    "tail.hpp", "rsetup.hpp"]


def sources_digest():
    """SHA-256 over the headline path's kernel sources."""
    import hashlib
    h = hashlib.sha256()
    for f in HEADLINE_SOURCES:
        with open(os.path.join(ROOT, "paper_2505_17623_amd", "csrc", f), "rb") as fh:
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


def _oracle_sample(cfg):
    """A bounded sample of workload cfg for the oracle, with the workload's
    ratio of product work (n m k) to folded elements (about 2 P n k): that
    ratio is m / (2 P) per layer, so the samples keep every layer's inner
    dimension m and shrink the batch."""
    from paper_2505_17623_amd import inputs
    if cfg == 3:
        return inputs.cfg3(n=1024), "the full 1024^3 layer"
    if cfg == 5:
        return inputs.cfg5(batch=128, d=4096), "MLP 4096-4096-4096 at batch 128 (same m and distribution, s=12)"
    if cfg == 4:
        return inputs.cfg4(batch=4, H=32), "the same CNN at batch 4"
    return inputs.workload(cfg, "full"), "the full workload"


def _oracle_worker(cfg):
    """One oracle run of the sample (child process): (seconds, transcript digest)."""
    import hashlib
    from oracle import oracle as orc
    wl, _ = _oracle_sample(cfg)
    t0 = time.perf_counter()
    res = orc.prove_network(wl)
    dt = time.perf_counter() - t0
    keys = ["t", "P", "c0", "mm_evals", "a_star", "b_star", "r_claim", "rm_claim", "y_claim", "z_claim",
            "range_sum", "rs_evals", "bits_claim", "zc_evals", "r_at", "y_at"]
    h = hashlib.sha256(json.dumps([[r[k] for k in keys] for r in res]).encode()).hexdigest()
    return dt, h, [r["P"] for r in res]


def host_cores():
    """Host threads this process may use: the affinity set, at most the
    16 a one-GPU machine gives a job."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, all_cores=True):
    """The oracle as it stands (plain C, one thread per process) on a bounded
    sample of the workload: once alone, then (all_cores) as one copy per host
    thread in child processes, each checked to give the single run's
    transcript.  The all-cores rate is copies x elements / wall time."""
    import multiprocessing as mp
    from oracle import oracle as orc
    wl, sample = _oracle_sample(cfg)
    orc.build(force=False)
    dt, digest, planes = _oracle_worker(cfg)
    el = elements_folded(layer_shapes(wl), planes)
    out = dict(value=el / dt, unit="field elements folded/s", cores=1, kind="oracle",
               sample=f"{sample}; {el} elements in {dt:.2f} s on one thread",
               host=dict(cpu_model=cpu_model(), nproc=os.cpu_count(), usable_threads=host_cores()))
    ncores = host_cores()
    if all_cores and ncores > 1:
        ctx = mp.get_context("spawn")  # fresh interpreters: nothing of this process's GPU state
        t0 = time.perf_counter()
        with ctx.Pool(ncores) as pool:
            res = pool.map(_oracle_worker, [cfg] * ncores)
        wall = time.perf_counter() - t0
        assert all(h == digest for _, h, _ in res), "oracle copies disagree with the single run"
        out.update(value=ncores * el / wall, cores=ncores,
                   sample=out["sample"] + f"; all cores: {ncores} copies in {wall:.2f} s wall, transcripts "
                   f"identical to the single run",
                   single_thread_value=round(el / dt, 1))
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=5, choices=[1, 2, 3, 4, 5],
                    help="workload (default 5: two 512x4096x4096 layers, the largest that fits one GPU)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--links", action="store_true",
                    help="also prove the workload's gather links (config 4: im2col and flatten) in every step; "
                         "each link call waits for the device")
    ap.add_argument("--fp2-steps", type=int, default=10,
                    help="after the timed region, time this many steps of the same workload proven with "
                         "challenges in F_{p^2} (reported beside the headline; 0 skips it)")
    ap.add_argument("--commit-steps", type=int, default=2,
                    help="then this many steps of Pedersen commitments (secp256k1) to every layer's witness "
                         "tables R, Rm, Y, Z and the bit words (reported beside the headline; 0 skips it)")
    ap.add_argument("--fs-steps", type=int, default=10,
                    help="then this many steps of the non-interactive proof (Fiat-Shamir over F_{p^2}, the "
                         "transcript hashed on the device; reported beside the headline; 0 skips it)")
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
        out = ra.prove_network(ctx, wl, dev, X=X, Bs=Bs, links=args.links)
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
        outs = [ra.prove_network(ctx, wl, dev, X=X, Bs=Bs, ts=ts, bufs=bufs, links=args.links) for _ in range(args.steps)]
        ctx.sync()
        assert all([o["transcript"]["P"] for o in out] == planes for out in outs)

    # timed region: K steps enqueued back to back, completed by one sync.
    # The heap built so far (transcripts of the untimed passes) is collected
    # and frozen first, so that a full garbage collection over it cannot
    # stall the host inside the timed steps.
    gc.collect()
    gc.freeze()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    outs = [ra.prove_network(ctx, wl, dev, X=X, Bs=Bs, ts=ts, bufs=bufs, links=args.links) for _ in range(args.steps)]
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
        ra.prove_network(ctx, wl, dev, X=X, Bs=Bs, ts=ts, bufs=bufs, links=args.links)
    ctx.sync()
    torch.cuda.synchronize()
    prof = ctx.profile()
    ctx.set_profiling(False)
    ms_step = 1e3 * elapsed / args.steps
    el = elements_folded(shapes, planes)
    value = el * args.steps / elapsed

    # roofline of the dominant kernel group: its algorithmic work per launch
    # (group_work) over its average launch time, measured with HIP events
    # on the library's stream
    work = group_work(shapes, planes)

    def rate(bound, amount, s_per_step):
        peak, unit, scale = PEAKS[bound]
        a = amount / s_per_step / scale
        return dict(bound=bound, achieved=round(a, 2), peak=peak, unit=unit, frac=round(a / peak, 4))

    dom = max((g for g in prof if g in work), key=lambda g: prof[g][0])
    dom_ms, dom_launches = prof[dom]
    per_step_s = dom_ms / 1e3 / args.steps
    launches = dom_launches / args.steps
    wd = work[dom]
    traffic = traffic_of(dom, args.config)
    roofline = dict(kernel=dom, **rate(wd["bound"], wd["amount"], per_step_s),
                    traffic=None if traffic is None else round(traffic / launches),
                    algorithmic_per_launch=round(wd["amount"] / launches), launches_per_step=launches,
                    ms_per_launch=round(dom_ms / dom_launches, 5))
    if wd["secondary"]:
        roofline["secondary"] = rate(wd["secondary"][0], wd["secondary"][1], per_step_s)
    groups = {g: dict(ms_per_step=round(v[0] / args.steps, 4), launches_per_step=v[1] / args.steps)
              for g, v in sorted(prof.items(), key=lambda kv: -kv[1][0]) if v[1]}
    for g, d in groups.items():
        s_per = d["ms_per_step"] / 1e3
        if g in work and s_per > 0:
            d.update(rate(work[g]["bound"], work[g]["amount"], s_per))
            if work[g]["secondary"]:
                d["secondary"] = rate(work[g]["secondary"][0], work[g]["secondary"][1], s_per)

    # the same workload with challenges in F_{p^2} (soundness error squared):
    # each layer call waits for its work, t given, buffers kept across steps
    fp2 = None
    if args.fp2_steps > 0:
        ctx2 = ra.Context(seed=wl.challenge_seed)
        bufs2 = []
        for _ in range(2):
            ra.prove_network_fp2(ctx2, wl, dev, X=X, Bs=Bs, ts=ts, bufs=bufs2)
        gc.collect()
        gc.freeze()
        torch.cuda.synchronize()
        u0 = time.perf_counter()
        outs2 = [ra.prove_network_fp2(ctx2, wl, dev, X=X, Bs=Bs, ts=ts, bufs=bufs2) for _ in range(args.fp2_steps)]
        torch.cuda.synchronize()
        el2 = time.perf_counter() - u0
        assert all([o["transcript"]["P"] for o in out] == planes for out in outs2)
        ms2 = 1e3 * el2 / args.fp2_steps
        fp2 = dict(field="F_p[i]/(i^2+1)", steps=args.fp2_steps, ms_per_step=round(ms2, 4),
                   ms_per_layer=round(ms2 / L, 4), value=round(el * args.fp2_steps / el2, 1),
                   unit="field elements folded/s", vs_fp_ms=round(ms2 / ms_step, 3),
                   note="synchronous per layer (each call waits); not the headline")
        del outs2, bufs2, ctx2
        print(f"# F_p^2 leg: {ms2:.3f} ms per step", file=sys.stderr, flush=True)

    # the non-interactive proof: every challenge hashed from the transcript on
    # the device (witness Merkle root first), one transcript across the steps
    fsl = None
    if args.fs_steps > 0:
        domain, pubs = wl.fs_inputs()
        ctx3 = ra.Context(fs_domain=domain)
        bufs3 = []
        for _ in range(2):
            ra.prove_network_fp2(ctx3, wl, dev, X=X, Bs=Bs, ts=ts, bufs=bufs3, pubs=pubs)
        gc.collect()
        gc.freeze()
        torch.cuda.synchronize()
        u0 = time.perf_counter()
        outs3 = [ra.prove_network_fp2(ctx3, wl, dev, X=X, Bs=Bs, ts=ts, bufs=bufs3, pubs=pubs)
                 for _ in range(args.fs_steps)]
        torch.cuda.synchronize()
        el3 = time.perf_counter() - u0
        assert all([o["transcript"]["P"] for o in out] == planes for out in outs3)
        ms3 = 1e3 * el3 / args.fs_steps
        fsl = dict(field="F_p[i]/(i^2+1)", transform="Fiat-Shamir, SHA-256 on the device", steps=args.fs_steps,
                   ms_per_step=round(ms3, 4), ms_per_layer=round(ms3 / L, 4),
                   value=round(el * args.fs_steps / el3, 1), unit="field elements folded/s",
                   vs_fp_ms=round(ms3 / ms_step, 3), note="synchronous per layer; not the headline")
        del outs3, bufs3, ctx3
        print(f"# non-interactive leg: {ms3:.3f} ms per step", file=sys.stderr, flush=True)

    # commitments to the witness tables of every layer (the tables of the last
    # headline step, left in `bufs`)
    com = None
    if args.commit_steps > 0:
        import hashlib
        cctx = ra.Context(seed=wl.challenge_seed)
        nmax = max(int(b["C"].numel()) for b in bufs)
        gens = ra.commit_generators(cctx, hashlib.sha256(b"range-arithmetic bench generators").digest(), nmax)
        tables = []
        for b in bufs:
            R, Rm, Y, Z, bits = b["wit"]
            tables += [(R, None), (Rm, ra.RA_U16), (Y, None), (Z, None), (bits, ra.RA_U64)]
        # one call per table (ra_commit), then all tables in one call
        # (ra_commit_batch), which must give the same points
        single = [ra.commit(cctx, T, gens, d) for T, d in tables]  # warm-up
        assert ra.commit_batch(cctx, tables, gens) == single
        torch.cuda.synchronize()
        c0 = time.perf_counter()
        for _ in range(args.commit_steps):
            pts = [ra.commit(cctx, T, gens, d) for T, d in tables]
        torch.cuda.synchronize()
        ms_single = 1e3 * (time.perf_counter() - c0) / args.commit_steps
        c0 = time.perf_counter()
        for _ in range(args.commit_steps):
            pts = ra.commit_batch(cctx, tables, gens)
        torch.cuda.synchronize()
        msc = 1e3 * (time.perf_counter() - c0) / args.commit_steps
        entries = sum(int(T.numel()) for T, _ in tables)
        com = dict(curve="secp256k1", tables=len(tables), entries_per_step=entries, steps=args.commit_steps,
                   ms_per_step=round(msc, 3), ms_per_table=round(msc / len(tables), 3),
                   ms_per_step_one_call_per_table=round(ms_single, 3),
                   note="Pedersen vector commitments to the witness tables (one batched call per step); "
                        "not the headline")
        assert pts == single
        del gens, cctx
        print(f"# commitments: {msc:.2f} ms per step ({len(tables)} tables)", file=sys.stderr, flush=True)

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
               config=dict(workload=f"config {args.config}: {wl.name}" + (" with gather links" if args.links else ""),
                           layers=L,
                           shapes=[list(s[:3]) for s in shapes], planes=planes,
                           elements_folded_per_step=el),
               roofline=roofline, cpu_baseline=cpu, kernel_groups=groups, field_fp2=fp2,
               non_interactive=fsl, commitments=com)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
