"""Writes tests/golden/full_cfg<N>.json: the CPU oracle's transcript of every
layer of workload N at full size, with SHA-256 digests of the inputs and of
every output table.  Calls only the oracle and the seeded input generator.

    python tests/golden/make_golden.py [cfg ...]          (default: 1 2 3 4 5)
    python tests/golden/make_golden.py --fp2 [cfg ...]    -> full_fp2_cfg<N>.json
    python tests/golden/make_golden.py --links [cfg ...]  -> full_links_cfg<N>.json
    python tests/golden/make_golden.py --fs [cfg ...]     -> full_fs_cfg<N>.json

With --fp2 the oracle proves the workload with challenges in F_{p^2} (the
seed's stream read in pairs); the witness tables are those of the F_p proof,
so only the transcript words (pairs re, im) and the digests of Z are kept.
With --fs the oracle proves the workload non-interactively (Fiat-Shamir over
F_{p^2}, the workload's fs_inputs()): the transcripts, each layer's witness
root and the digests of Z are kept.
With --links every gather link of the workload is proven after its layer
(the later layers then read later challenges): the transcripts, each link's
words and the digests of Z are kept.

Digest formats: C, R, Rm, Y, Z as little-endian int64 arrays in row-major
order; the bit table as P x N bytes (0/1), plane-major; A and B as int64.
"""
import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import oracle as orc  # noqa: E402
from paper_2505_17623_amd import inputs  # noqa: E402

TRANSCRIPT = ["t", "P", "c0", "mm_evals", "a_star", "b_star", "r_claim", "rm_claim", "y_claim", "z_claim",
              "range_sum", "rs_evals", "bits_claim", "zc_evals", "r_at", "y_at", "challenges_used"]


def digest(a) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def digest_i64(a) -> str:
    return digest(np.asarray(a).astype("<i8"))


def main_fp2(cfgs):
    orc.build(force=False)
    for cfg in cfgs:
        wl = inputs.workload(cfg, "full")
        t0 = time.time()
        res = orc.prove_network_fp2(wl)
        layers = [dict(shape=[r["n"], r["m"], r["k"]], s=r["s"], relu=r["relu"], mode=r["mode"],
                       transcript={k: r[k] for k in TRANSCRIPT}, digests=dict(Z=digest_i64(r["Z"])))
                  for r in res]
        out = dict(workload=wl.name, config=cfg, field="F_p[i]/(i^2+1)",
                   oracle_seconds=round(time.time() - t0, 1), layers=layers,
                   source="oracle/ra_oracle_fp2.c via tests/golden/make_golden.py --fp2")
        path = os.path.join(HERE, f"full_fp2_cfg{cfg}.json")
        with open(path, "w") as f:
            json.dump(out, f, indent=1)
        print(f"config {cfg} over F_p^2: {len(layers)} layers, oracle {out['oracle_seconds']} s -> {path}",
              flush=True)


def main_fs(cfgs):
    orc.build(force=False)
    for cfg in cfgs:
        wl = inputs.workload(cfg, "full")
        domain, pubs = wl.fs_inputs()
        t0 = time.time()
        res = orc.prove_network_fs(wl, domain, pubs)
        layers = []
        for r in res:
            root = orc.witness_root(r["R"], r["Rm"], r["Y"], r["Z"], orc.pack_words(r["bits"]))
            layers.append(dict(shape=[r["n"], r["m"], r["k"]], transcript={k: r[k] for k in TRANSCRIPT},
                               root=root.hex(), digests=dict(Z=digest_i64(r["Z"]))))
        out = dict(workload=wl.name, config=cfg, field="F_p[i]/(i^2+1)", transform="Fiat-Shamir, SHA-256",
                   oracle_seconds=round(time.time() - t0, 1), layers=layers,
                   source="oracle/ra_oracle_fp2.c, oracle/ra_oracle_fs.c via tests/golden/make_golden.py --fs")
        path = os.path.join(HERE, f"full_fs_cfg{cfg}.json")
        with open(path, "w") as f:
            json.dump(out, f, indent=1)
        print(f"config {cfg} non-interactive: {len(layers)} layers, oracle {out['oracle_seconds']} s -> {path}",
              flush=True)


def main_links(cfgs):
    orc.build(force=False)
    for cfg in cfgs:
        wl = inputs.workload(cfg, "full")
        t0 = time.time()
        res = orc.prove_network(wl, links=True)
        layers = [dict(shape=[r["n"], r["m"], r["k"]], transcript={k: r[k] for k in TRANSCRIPT},
                       link=r.get("link"), digests=dict(Z=digest_i64(r["Z"]))) for r in res]
        out = dict(workload=wl.name, config=cfg, oracle_seconds=round(time.time() - t0, 1), layers=layers,
                   cursor=res[-1]["cursor"], source="oracle/ra_oracle.c via tests/golden/make_golden.py --links")
        path = os.path.join(HERE, f"full_links_cfg{cfg}.json")
        with open(path, "w") as f:
            json.dump(out, f, indent=1)
        print(f"config {cfg} with links: {len(layers)} layers, oracle {out['oracle_seconds']} s -> {path}",
              flush=True)


def main(cfgs):
    orc.build(force=False)
    for cfg in cfgs:
        wl = inputs.workload(cfg, "full")
        t0 = time.time()
        res = orc.prove_network(wl)
        layers = []
        for li, r in enumerate(res):
            layers.append(dict(
                shape=[r["n"], r["m"], r["k"]], s=r["s"], relu=r["relu"], mode=r["mode"],
                transcript={k: r[k] for k in TRANSCRIPT},
                digests=dict(A=digest_i64(r["A"]), B=digest_i64(wl.layers[li].B), C=digest_i64(r["C"]),
                             R=digest_i64(r["R"]), Rm=digest_i64(r["Rm"]), Y=digest_i64(r["Y"]),
                             Z=digest_i64(r["Z"]), bits=digest(r["bits"].astype(np.uint8)))))
        out = dict(workload=wl.name, config=cfg, oracle_seconds=round(time.time() - t0, 1), layers=layers,
                   source="oracle/ra_oracle.c via tests/golden/make_golden.py")
        path = os.path.join(HERE, f"full_cfg{cfg}.json")
        with open(path, "w") as f:
            json.dump(out, f, indent=1)
        print(f"config {cfg}: {len(layers)} layers, oracle {out['oracle_seconds']} s -> {path}", flush=True)


if __name__ == "__main__":
    args = sys.argv[1:]
    if args and args[0] == "--fp2":
        main_fp2([int(a) for a in args[1:]] or [1, 2, 3, 4, 5])
    elif args and args[0] == "--fs":
        main_fs([int(a) for a in args[1:]] or [1, 2, 3, 4, 5])
    elif args and args[0] == "--links":
        main_links([int(a) for a in args[1:]] or [4])
    else:
        main([int(a) for a in args] or [1, 2, 3, 4, 5])
