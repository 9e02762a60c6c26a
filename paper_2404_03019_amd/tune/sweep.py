"""Offline performance database for the kernel selector (Section III-C, "data-aware config rules").

For every instance of a seeded synthetic family (length distribution, nnz,
mean segment length, F, op, plain or fused gather, with or without edge
weights) this times every
candidate kernel choice through the library's forced-choice entry points and
appends one JSON line per (instance, candidate) to a performance database.
Already-measured keys are skipped, so an interrupted sweep resumes.

The values of the inputs do not affect the timing; they are drawn on the GPU
with a seeded torch generator. Segment lengths come from numpy with the
instance seed.

Usage (on the GPU):
  python -m paper_2404_03019_amd.tune.sweep --out paper_2404_03019_amd/tune/perfdb.jsonl
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

DISTS = ("fixed", "poisson", "uniform", "zipf", "lognormal_narrow", "lognormal_wide", "one_heavy")
FS = (1, 2, 3, 4, 8, 16, 32, 64, 128, 256)
EP_ROWS = (4, 8, 16, 32, 64, 128, 256)
TILE_ROWS = (16, 32, 64, 128)  # row runs also timed over 2 and 4 column tiles in sequence (fused form)


def draw_lengths(rng, dist: str, S: int, nnz: int) -> np.ndarray:
    from workloads import lr_rescale

    if dist == "fixed":
        w = np.ones(S)
    elif dist == "poisson":
        w = rng.poisson(max(1.0, nnz / S), S).astype(np.float64) + 1e-3
    elif dist == "uniform":
        w = rng.random(S) + 0.05
    elif dist == "zipf":
        w = rng.zipf(rng.uniform(1.6, 2.4), S).astype(np.float64)
    elif dist == "lognormal_narrow":
        w = rng.lognormal(0.0, 0.5, S)
    elif dist == "lognormal_wide":
        w = rng.lognormal(0.0, 1.5, S)
    elif dist == "one_heavy":
        w = rng.random(S) + 0.05
        w[rng.integers(0, S)] = 0.2 * w.sum()
    else:
        raise ValueError(dist)
    return lr_rescale(w, nnz)


def instances(n: int, seed: int):
    """A seeded list of (id, dist, nnz, mean, F, op, gather) instances."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        dist = DISTS[rng.integers(len(DISTS))]
        F = int(FS[rng.integers(len(FS))])
        gather = int(rng.random() < 0.35)
        op = "max" if rng.random() < 0.3 else "sum"
        mean = float(2.0 ** rng.uniform(0.5, 10.0))
        # keep each input below ~3 GB of streamed data
        max_nnz = min(1.2e8, 3e9 / (4 * F + 20))
        nnz = int(min(max_nnz, 10 ** rng.uniform(4.0, 8.1)))
        S = max(1, int(round(nnz / mean)))
        out.append(dict(id=i, dist=dist, nnz=nnz, S=S, F=F, op=op, gather=gather, seed=seed * 100003 + i))
    return out


def gather_instances(n: int, seed: int):
    """A seeded list of fused-form instances, half of them without edge weights
    (the unweighted index_segment_reduce and the weighted SpMM form)."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        dist = DISTS[rng.integers(len(DISTS))]
        F = int(FS[rng.integers(len(FS))])
        weighted = int(rng.random() < 0.5)
        u = rng.random()
        op = "max" if u < 0.3 else ("mean" if u < 0.45 else "sum")
        mean = float(2.0 ** rng.uniform(0.5, 10.0))
        max_nnz = min(1.2e8, 3e9 / (4 * F + 20))
        nnz = int(min(max_nnz, 10 ** rng.uniform(4.0, 8.1)))
        S = max(1, int(round(nnz / mean)))
        out.append(dict(id=20000 + i, dist=dist, nnz=nnz, S=S, F=F, op=op, gather=1, weighted=weighted,
                        seed=seed * 100003 + i))
    return out


def paired_instances(n: int, seed: int):
    """Pairs of segment reductions with the same nnz, num_segments, F and op (so the same O(1)
    features) and opposite length spreads: one with even lengths (fixed or Poisson), one with
    heavy-tailed ones (Zipf or wide lognormal). Only the length statistics tell the two apart,
    which is what the tree with statistics is for."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        F = int(FS[rng.integers(len(FS))])
        op = "max" if rng.random() < 0.3 else "sum"
        mean = float(2.0 ** rng.uniform(0.5, 8.0))
        max_nnz = min(1.2e8, 3e9 / (4 * F + 20))
        nnz = int(min(max_nnz, 10 ** rng.uniform(4.5, 8.0)))
        S = max(1, int(round(nnz / mean)))
        even = ("fixed", "poisson")[rng.integers(2)]
        heavy = ("zipf", "lognormal_wide")[rng.integers(2)]
        for j, dist in enumerate((even, heavy)):
            out.append(dict(id=30000 + 2 * i + j, dist=dist, nnz=nnz, S=S, F=F, op=op, gather=0,
                            seed=seed * 100003 + 2 * i + j))
    return out


def named_instances():
    """The five named workloads (lengths from their recipes), each op they are run with,
    and the SpMM workload without weights and with max."""
    from workloads.generators import C2_FEATURES

    out = []
    specs = [("c1_zipf_small", 32, "sum", 0), ("c3_powerlaw_graph", 32, "sum", 0),
             ("c4_spmm", 128, "sum", 1), ("c5_pointcloud_knn", 64, "mean", 0),
             ("c5_pointcloud_knn", 64, "max", 0)]
    specs += [("c2_poisson_fsweep", F, op, 0) for F in C2_FEATURES for op in ("sum", "max")]
    specs += [("c4_spmm", 128, "sum", 1, 0), ("c4_spmm", 128, "max", 1, 1)]
    for i, spec in enumerate(specs):
        name, F, op, gather = spec[:4]
        weighted = spec[4] if len(spec) > 4 else gather
        out.append(dict(id=10000 + i, dist=name, nnz=0, S=0, F=F, op=op, gather=gather, weighted=weighted,
                        seed=i))
    return out


def lanes_for(F: int) -> int:
    """Lanes of a row group for fp32 rows of F columns: 4-float vectors from F = 4 on (the last
    one overlapping when 4 does not divide F), one 3-float vector for F = 3, else F floats."""
    V = 4 if F >= 4 else F
    vecs = -(-F // V)
    L = 1
    while L < vecs and L < 64:
        L <<= 1
    return L


def candidates(F: int, allow_sp: bool, gather: bool = False):
    c = [dict(family=1, rows=0)] + [dict(family=1, rows=k) for k in EP_ROWS]
    if gather and F >= 64 and F % 4 == 0:  # column tiles in sequence (tile-major blocks)
        c += [dict(family=1, rows=k, lanes=lanes_for(F) // t, flags=4, tiles=t) for t in (2, 4) for k in TILE_ROWS]
    if allow_sp:
        L = lanes_for(F)
        g = 1
        while g <= 64 // L:
            c.append(dict(family=2, groups=g))
            g <<= 1
    return c


def ckey(c: dict) -> str:
    t = c.get("tiles", 1)
    return f"f{c['family']}_r{c.get('rows', 0)}_g{c.get('groups', 0)}" + (f"_t{t}" if t > 1 else "")


def as_choice(c: dict) -> dict:
    """The library's choice for candidate c (its `tiles` is a database label only)."""
    return {k: v for k, v in c.items() if k != "tiles"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=os.path.join(HERE, "perfdb.jsonl"))
    ap.add_argument("--n", type=int, default=240)
    ap.add_argument("--seed", type=int, default=2024)
    ap.add_argument("--gather-n", type=int, default=120)
    ap.add_argument("--gather-seed", type=int, default=4048)
    ap.add_argument("--paired-n", type=int, default=40)
    ap.add_argument("--paired-seed", type=int, default=6072)
    ap.add_argument("--reps", type=int, default=5)
    ap.add_argument("--budget-s", type=float, default=900.0, help="stop after this many seconds")
    args = ap.parse_args()

    import torch

    import paper_2404_03019_amd as geot

    done = set()
    if os.path.exists(args.out):
        for line in open(args.out):
            try:
                r = json.loads(line)
                done.add((r["instance"]["id"], r["instance"]["seed"], r["cand"]))
            except (ValueError, KeyError):
                pass
    done_inst = {(i, s) for (i, s, _) in done}
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    t_start = time.time()
    with open(args.out, "a") as fout:
        for inst in named_instances() + instances(args.n, args.seed) + \
                gather_instances(args.gather_n, args.gather_seed) + paired_instances(args.paired_n, args.paired_seed):
            if time.time() - t_start > args.budget_s:
                print("budget reached", flush=True)
                break
            weighted = inst.get("weighted", inst["gather"])
            if (inst["id"], inst["seed"]) in done_inst and all(
                    (inst["id"], inst["seed"], ckey(c)) in done
                    for c in candidates(inst["F"], False, bool(inst["gather"]))):
                continue  # every candidate but possibly SP done (SP is skipped on heavy tails)
            if 10000 <= inst["id"] < 20000:  # a named workload: lengths from its recipe
                from workloads import config_lengths

                _, L = config_lengths(inst["dist"])
                inst["S"], inst["nnz"] = int(L.size), int(L.sum())
            else:
                rng = np.random.default_rng(inst["seed"])
                L = draw_lengths(rng, inst["dist"], inst["S"], inst["nnz"])
            S, nnz, F = inst["S"], inst["nnz"], inst["F"]
            idx = torch.repeat_interleave(torch.arange(S, device=dev), torch.from_numpy(L).to(dev))
            gen.manual_seed(inst["seed"])
            if inst["gather"]:
                nx = max(1, S)
                X = torch.randn(nx, F, device=dev, generator=gen)
                col = torch.randint(0, nx, (nnz,), device=dev, generator=gen)
                w = torch.rand(nnz, device=dev, generator=gen) if weighted else None
                out = torch.empty(S, F, device=dev)
                nbytes = nnz * (16 + 4 * weighted + 4 * F) + S * F * 4

                def call(c):
                    geot.gather_scatter(X, col, w, idx, S, inst["op"], out=out, choice=as_choice(c))
            else:
                src = torch.randn(nnz, F, device=dev, generator=gen)
                out = torch.empty(S, F, device=dev)
                nbytes = nnz * (8 + 4 * F) + S * F * 4

                def call(c):
                    geot.segment_reduce(src, idx, S, inst["op"], out=out, choice=as_choice(c))
            st = geot.index_stats(idx, S)
            mean = nnz / S
            feats = dict(nnz=nnz, S=S, F=F, mean=mean, op=inst["op"], gather=inst["gather"], weighted=weighted,
                         cv=math.sqrt(st["var_len"]) / mean if mean > 0 else 0.0,
                         max_rel=st["max_len"] / mean if mean > 0 else 0.0)
            best = math.inf
            # a segment-parallel team owns a whole segment: hopeless on very heavy tails
            for c in candidates(F, feats["max_rel"] <= 256.0, bool(inst["gather"])):
                key = (inst["id"], inst["seed"], ckey(c))
                if key in done:
                    continue
                call(c)  # warm-up (and first-touch of the pool)
                torch.cuda.synchronize()
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                call(c)
                e1.record()
                e1.synchronize()
                first = e0.elapsed_time(e1)
                ts = [first]
                if first < 20 * best and first < 250.0:
                    for _ in range(args.reps - 1):
                        e0.record()
                        call(c)
                        e1.record()
                        e1.synchronize()
                        ts.append(e0.elapsed_time(e1))
                ms = float(np.median(ts))
                best = min(best, ms)
                rec = dict(instance=inst, features=feats, cand=ckey(c), choice=c,
                           used=geot.last_choice(), ms=ms, gbs=nbytes / (ms * 1e-3) / 1e9)
                fout.write(json.dumps(rec) + "\n")
            fout.flush()
            print(f"instance {inst['id']} {inst['dist']} nnz={nnz} S={S} F={F} {inst['op']} "
                  f"gather={inst['gather']} best={best:.3f} ms", flush=True)
            del idx, out
            if inst["gather"]:
                del X, col, w
            else:
                del src
            torch.cuda.empty_cache()


if __name__ == "__main__":
    main()
