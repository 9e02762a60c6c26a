"""Fit the selector's decision trees to the performance database and emit them as C++ if/else.

Follows Section III-C of the GeoT paper: a decision tree of depth at most 5
over cheap input features, whose leaves hold a whole kernel configuration
(chosen jointly, not parameter by parameter), emitted as nested if/else in
``csrc/selector_generated.h`` and compiled into the library.

Leaves and splits are fitted to the measured times directly: each leaf takes
the candidate with the least total log-slowdown (log of time over the best
measured time of the same input) over the inputs that reach it, and each
split is the feature threshold that most reduces that total. The paper's own
recipe (Top-1 labels and a scikit-learn multi-output regressor of depth 5,
leaves rounded to valid parameters) is fitted too and reported as an
ablation, beside the hand-written rule.

Two trees per operation, as the paper keeps two, and one pair for each of the
two operations (segment reduction, and the fused gather form, whose inputs
also say whether edges carry weights), since their best configurations
differ:
  * ``nostats``: O(1) features only (log2 nnz, log2 num_segments, F,
    log2 mean length, op; for the fused form also weighted); chooses among
    element-parallel row runs;
  * ``stats``: adds the length cv and log2(longest / mean) from
    geot_index_stats; chooses the family and its parameters.
A single pair over both operations (with gather and weighted as features) is
fitted too and reported as an ablation.

Usage: python -m paper_2404_03019_amd.tune.fit [--db perfdb.jsonl] [--out ../csrc/selector_generated.h]
"""
from __future__ import annotations

import argparse
import collections
import json
import math
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
DEFAULT_DB = os.path.join(HERE, "perfdb.jsonl")
DEFAULT_OUT = os.path.join(os.path.dirname(HERE), "csrc", "selector_generated.h")
MAX_DEPTH = 5


def load(db: str):
    inst = collections.OrderedDict()
    for line in open(db):
        r = json.loads(line)
        k = (r["instance"]["id"], r["instance"]["seed"])
        e = inst.setdefault(k, dict(instance=r["instance"], features=r["features"], times={}, choices={}))
        e["times"][r["cand"]] = r["ms"]
        e["choices"][r["cand"]] = r["choice"]
    return list(inst.values())


KINDS = ("segment", "gather")


def kind_of(e) -> str:
    return "gather" if e["instance"]["gather"] else "segment"


def weighted_of(e) -> int:
    """Fused-form inputs of the first sweeps carry no flag: they all had weights."""
    inst = e["instance"]
    return int(inst.get("weighted", inst["gather"])) if inst["gather"] else 0


def feature_row(e, stats: bool, kind: str | None = None):
    """Features of input e for the trees of `kind` (None: the single-tree ablation)."""
    f = e["features"]
    row = [math.log2(max(f["nnz"], 1)), math.log2(max(f["S"], 1)), float(f["F"]),
           math.log2(max(f["mean"], 1e-9)), 1.0 if f["op"] == "max" else 0.0]
    if kind is None:
        row += [float(f["gather"]), float(weighted_of(e))]
    elif kind == "gather":
        row += [float(weighted_of(e))]
    if stats:
        row += [float(f["cv"]), math.log2(max(f["max_rel"], 1e-9))]
    return row


def feature_names(stats: bool, kind: str | None = None):
    names = ["lnnz", "lS", "F", "lmean", "opmax"]
    if kind is None:
        names += ["isgather", "weighted"]
    elif kind == "gather":
        names += ["weighted"]
    return names + (["cv", "lmaxrel"] if stats else [])


def best_of(e, fam=None):
    items = [(t, c) for c, t in e["times"].items()
             if (fam is None or e["choices"][c]["family"] == fam) and e["choices"][c].get("rows", 1) != 0]
    return min(items) if items else (math.inf, None)


def targets(e):
    t_all, c_all = best_of(e)
    _, c_ep = best_of(e, 1)
    _, c_sp = best_of(e, 2)
    fam = e["choices"][c_all]["family"]
    k = e["choices"][c_ep]["rows"]
    g = e["choices"][c_sp]["groups"] if c_sp else 1
    return fam, math.log2(k), math.log2(g)


def fit_tree(X, Y):
    from sklearn.tree import DecisionTreeRegressor

    t = DecisionTreeRegressor(max_depth=MAX_DEPTH, min_samples_leaf=2, random_state=0)
    t.fit(np.asarray(X), np.asarray(Y))
    return t


def round_leaf(v, with_family: bool):
    if with_family:
        fam = 2 if v[0] >= 1.5 else 1
        k = int(2 ** min(8, max(2, round(v[1]))))
        g = int(2 ** min(6, max(0, round(v[2]))))
        return fam, k, g
    k = int(2 ** min(8, max(2, round(v[0]))))
    return 1, k, 1


def emit(tree, names, with_family, indent):
    t = tree.tree_
    lines = []

    def rec(node, depth):
        pad = " " * (indent + 4 * depth)
        if t.children_left[node] == t.children_right[node]:
            fam, k, g = round_leaf(t.value[node][:, 0], with_family)
            lines.append(f"{pad}out[0] = {fam}; out[3] = {k}; out[4] = {g};")
            return
        f = names[t.feature[node]]
        thr = t.threshold[node]
        lines.append(f"{pad}if ({f} <= {thr:.6g}) {{")
        rec(t.children_left[node], depth + 1)
        lines.append(f"{pad}}} else {{")
        rec(t.children_right[node], depth + 1)
        lines.append(f"{pad}}}")

    rec(0, 0)
    return lines


def predict_cand(tree, row, with_family, e):
    v = tree.predict(np.asarray([row]))[0]
    fam, k, g = round_leaf(np.atleast_1d(v), with_family)
    c = f"f1_r{k}_g0" if fam == 1 else f"f2_r0_g{g}"
    if c not in e["times"]:  # SP not measured for this input: fall back to the element-parallel leaf
        c = f"f1_r{k}_g0"
    return c


EP_ROWS = (4, 8, 16, 32, 64, 128, 256)
TILE_ROWS = (16, 32, 64, 128)  # row runs timed with the columns in 2 or 4 tiles, one after another
MISSING_COST = math.log(50.0)  # a candidate that was not measured (or too slow to finish)
NAMED_WEIGHT = 16.0            # the named benchmark workloads count this many times


def lanes_for(F: int) -> int:
    """Lanes of a row group for fp32 rows of F columns: 4-float vectors from F = 4 on (the last
    one overlapping when 4 does not divide F), one 3-float vector for F = 3, else F floats."""
    V = 4 if F >= 4 else F
    vecs = -(-F // V)
    L = 1
    while L < vecs and L < 64:
        L <<= 1
    return L


INHERIT = (0, 0, 0, 0)  # a leaf of the statistics tree that keeps the O(1) tree's choice


def candidate_space(stats: bool, kind: str | None = None):
    """(family, rows, groups, tiles): tiles > 1 runs the element-parallel kernel over that many
    column tiles in sequence (tile-major blocks; fused form only). The statistics trees also
    have INHERIT: the O(1) tree's choice for the same input."""
    c = [INHERIT] if stats and kind is not None else []
    c += [(1, k, 1, 1) for k in EP_ROWS]
    if kind != "segment":
        c += [(1, k, 1, t) for t in (2, 4) for k in TILE_ROWS]
    if stats:
        c += [(2, 0, g, 1) for g in (1, 2, 4, 8, 16, 32, 64)]
    return c


def cand_key(cand, F: int) -> str:
    """The database key of a candidate for an input with F columns."""
    fam, k, g, t = cand
    if fam == 1:
        return f"f1_r{k}_g0" + (f"_t{t}" if t > 1 else "")
    return f"f2_r0_g{min(g, 64 // lanes_for(F))}"


def cost_matrix(data, cands, inherit=None):
    """C[i, j] = w_i * log(time of candidate j / best measured time of input i); the named
    workloads get weight NAMED_WEIGHT, every other input weight 1. `inherit(e)` gives the
    candidate an INHERIT leaf stands for on input e."""
    C = np.full((len(data), len(cands)), MISSING_COST)
    for i, e in enumerate(data):
        tb, _ = best_of(e)
        for j, cand in enumerate(cands):
            if cand == INHERIT:
                cand = inherit(e)
            t = e["times"].get(cand_key(cand, e["instance"]["F"]))
            if t is not None and t > 0 and tb > 0:
                C[i, j] = min(MISSING_COST, math.log(t / tb))
        if 10000 <= e["instance"]["id"] < 20000:
            C[i] *= NAMED_WEIGHT
    return C


class CostTree:
    """Greedy tree minimising the total cost of one candidate per leaf."""

    def __init__(self, max_depth=MAX_DEPTH, min_leaf=2):
        self.max_depth, self.min_leaf = max_depth, min_leaf

    def fit(self, X, C):
        self.X, self.C = np.asarray(X, dtype=np.float64), np.asarray(C, dtype=np.float64)
        self.root = self._grow(np.arange(len(self.X)), 0)
        return self

    def _leaf(self, rows):
        tot = self.C[rows].sum(axis=0)
        return dict(leaf=int(np.argmin(tot)), cost=float(tot.min()))

    def _grow(self, rows, depth):
        node = self._leaf(rows)
        if depth >= self.max_depth or len(rows) < 2 * self.min_leaf:
            return node
        best = (node["cost"] - 1e-9, None)
        for f in range(self.X.shape[1]):
            order = rows[np.argsort(self.X[rows, f], kind="stable")]
            vals = self.X[order, f]
            pre = np.cumsum(self.C[order], axis=0)
            total = pre[-1]
            for i in range(self.min_leaf - 1, len(order) - self.min_leaf):
                if vals[i] == vals[i + 1]:
                    continue
                c = pre[i].min() + (total - pre[i]).min()
                if c < best[0]:
                    best = (c, (f, 0.5 * (vals[i] + vals[i + 1])))
        if best[1] is None:
            return node
        f, thr = best[1]
        left = rows[self.X[rows, f] <= thr]
        right = rows[self.X[rows, f] > thr]
        return dict(feature=f, threshold=thr, left=self._grow(left, depth + 1),
                    right=self._grow(right, depth + 1))

    def predict_one(self, x):
        n = self.root
        while "leaf" not in n:
            n = n["left"] if x[n["feature"]] <= n["threshold"] else n["right"]
        return n["leaf"]


def emit_cost_tree(tree, names, cands, indent, final=True):
    """if/else of a tree. With final False (a statistics tree), a leaf returns its choice, and
    an INHERIT leaf falls through to the O(1) tree that follows."""
    lines = []

    def rec(n, depth):
        pad = " " * (indent + 4 * depth)
        if "leaf" in n:
            if cands[n["leaf"]] == INHERIT:
                lines.append(f"{pad}// the O(1) tree's choice (below)")
                return
            fam, k, g, t = cands[n["leaf"]]
            lines.append(f"{pad}out[0] = {fam}; out[3] = {k}; out[4] = {g};" + (f" out[5] = {t};" if t > 1 else "") +
                         ("" if final else " return;"))
            return
        lines.append(f"{pad}if ({names[n['feature']]} <= {n['threshold']:.9g}) {{")
        rec(n["left"], depth + 1)
        lines.append(f"{pad}}} else {{")
        rec(n["right"], depth + 1)
        lines.append(f"{pad}}}")

    rec(tree.root, 0)
    return lines


class Fitted:
    """The four trees (kind x stats) fitted on the database, and the single-pair ablation.

    The statistics tree of each operation refines its O(1) tree: it is fitted after it, with
    one more candidate, INHERIT, whose cost on an input is that of the O(1) tree's choice. A
    leaf therefore names another kernel only where that is measured better on the inputs that
    reach it, and the tree as a whole never costs more than the O(1) tree on the database."""

    def __init__(self, data):
        self.data = data
        self.trees, self.single = {}, {}
        for stats in (False, True):
            for kind in KINDS:
                sub = [e for e in data if kind_of(e) == kind]
                X = [feature_row(e, stats, kind) for e in sub]
                C = cost_matrix(sub, candidate_space(stats, kind), inherit=lambda e: self.choose(e, False))
                self.trees[(kind, stats)] = CostTree().fit(X, C)
            self.single[stats] = CostTree().fit([feature_row(e, stats) for e in data],
                                                cost_matrix(data, candidate_space(stats)))

    def choose(self, e, stats: bool):
        """(family, rows, groups, tiles) the emitted selector gives input e."""
        kind = kind_of(e)
        c = candidate_space(stats, kind)[self.trees[(kind, stats)].predict_one(feature_row(e, stats, kind))]
        return self.choose(e, False) if c == INHERIT else c

    def choose_as_library(self, e, stats: bool):
        """What geot_select returns: the tree's choice, except that the segment-parallel
        family is never used where the longest segment exceeds 256x the mean."""
        c = self.choose(e, stats)
        if stats and c[0] == 2 and e["features"]["max_rel"] > 256.0:
            c = self.choose(e, False)
        return c

    def choose_single(self, e, stats: bool):
        return candidate_space(stats)[self.single[stats].predict_one(feature_row(e, stats))]


def build(db: str) -> Fitted:
    """Load the database (inputs with at least one measured element-parallel row run) and fit."""
    data = load(db)
    data = [e for e in data if any(e["choices"][c]["family"] == 1 and e["choices"][c].get("rows", 0) > 0
                                   for c in e["times"])]
    return Fitted(data)


def render(fitted: Fitted) -> str:
    """The C++ header text of the four trees."""
    n_seg = sum(1 for e in fitted.data if kind_of(e) == "segment")
    n_gat = len(fitted.data) - n_seg
    body = ["// Kernel selection rules compiled into libgeot_hip (Section III-C: a decision tree",
            "// over cheap input features, emitted as if/else). GENERATED by",
            "// paper_2404_03019_amd/tune/fit.py from the MI355X performance database",
            "// paper_2404_03019_amd/tune/perfdb.jsonl; do not edit by hand.",
            "//",
            f"// Training inputs: {n_seg} segment reductions, {n_gat} fused gather forms. One pair of",
            f"// trees per operation, depth <= {MAX_DEPTH}. Each leaf is the candidate with the least",
            "// total log-slowdown over the inputs reaching it; the tree with statistics refines the",
            "// O(1) one (its leaves that keep the O(1) choice fall through to it). out[0] family (1 element-parallel,",
            "// 2 segment-parallel), out[3] rows per row group, out[4] row groups per segment",
            "// (clamped to the wave); out[1] vec, out[2] lanes: 0 = from the shape; out[5] column",
            "// tiles run one after another (1: the columns' own tiling, in adjacent blocks).",
            "// gather: 0 segment reduction, 1 fused form with edge weights, 2 without.",
            "#pragma once", "", "#include <cmath>", "#include <cstdint>", "", "namespace geot {", "",
            "static inline void tree_select(double nnz, double num_segments, double F, int op, int gather,",
            "                               int has_stats, double cv, double max_rel, int32_t out[6]) {",
            "    const double lnnz = std::log2(nnz > 1.0 ? nnz : 1.0);",
            "    const double lS = std::log2(num_segments > 1.0 ? num_segments : 1.0);",
            "    const double mean = num_segments > 0.0 ? nnz / num_segments : 0.0;",
            "    const double lmean = std::log2(mean > 1e-9 ? mean : 1e-9);",
            "    const double opmax = op == 2 ? 1.0 : 0.0;",
            "    const double weighted = gather == 1 ? 1.0 : 0.0;",
            "    const double lmaxrel = std::log2(max_rel > 1e-9 ? max_rel : 1e-9);",
            "    (void)lnnz; (void)lS; (void)F; (void)lmean; (void)opmax; (void)weighted; (void)cv; (void)lmaxrel;",
            "    out[0] = 1; out[1] = 0; out[2] = 0; out[3] = 0; out[4] = 0; out[5] = 1;"]
    for kind, cond, close in (("segment", "    if (gather == 0) {", None), ("gather", "    } else {", "    }")):
        body += [cond, "        if (has_stats) {  // refines the O(1) tree below: a leaf that keeps its choice falls through"]
        body += emit_cost_tree(fitted.trees[(kind, True)], feature_names(True, kind), candidate_space(True, kind), 12,
                               final=False)
        body += ["        }"]
        body += emit_cost_tree(fitted.trees[(kind, False)], feature_names(False, kind),
                               candidate_space(False, kind), 8)
    body += ["    }", "}", "", "}  // namespace geot", ""]
    return "\n".join(body)


def _time_of(e, cand):
    return e["times"].get(cand_key(cand, e["instance"]["F"]), math.nan)


def evaluate(fitted: Fitted):
    """Per input: chosen time / best measured time over every candidate (the segment-parallel
    ones included), for the per-operation trees, the single pair (ablation), the paper's recipe
    (per operation, ablation) and the hand rule; `nostats_ep` is the O(1) tree against the best
    element-parallel candidate, the only family it chooses from."""
    cn, cs = candidate_space(False), candidate_space(True)
    # the paper's recipe: Top-1 labels, multi-output regressor, rounded leaves
    paper = {}
    for kind in KINDS:
        sub = [e for e in fitted.data if kind_of(e) == kind]
        paper[(kind, False)] = fit_tree([feature_row(e, False, kind) for e in sub], [[targets(e)[1]] for e in sub])
        paper[(kind, True)] = fit_tree([feature_row(e, True, kind) for e in sub], [list(targets(e)) for e in sub])
    rep = []
    for e in fitted.data:
        tb, _ = best_of(e)
        tbe, _ = best_of(e, 1)
        kind = kind_of(e)
        rep.append(dict(
            name=e["instance"]["dist"], id=e["instance"]["id"], F=e["instance"]["F"],
            op=e["instance"]["op"], gather=e["instance"]["gather"], weighted=weighted_of(e),
            nnz=e["features"]["nnz"], best=tb,
            nostats=_time_of(e, fitted.choose(e, False)) / tb,
            nostats_ep=_time_of(e, fitted.choose(e, False)) / tbe,
            stats=_time_of(e, fitted.choose_as_library(e, True)) / tb,
            single_nostats=_time_of(e, fitted.choose_single(e, False)) / tb,
            single_stats=_time_of(e, fitted.choose_single(e, True)) / tb,
            paper_nostats=e["times"].get(predict_cand(paper[(kind, False)], feature_row(e, False, kind), False, e),
                                         math.nan) / tb,
            paper_stats=e["times"].get(predict_cand(paper[(kind, True)], feature_row(e, True, kind), True, e),
                                       math.nan) / tb,
            hand=e["times"].get("f1_r0_g0", math.nan) / tb))
    return rep


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--db", default=DEFAULT_DB)
    ap.add_argument("--out", default=DEFAULT_OUT)
    args = ap.parse_args()
    fitted = build(args.db)
    open(args.out, "w").write(render(fitted))
    rep = evaluate(fitted)

    def gm(xs):
        xs = [x for x in xs if x == x and x > 0]
        return math.exp(sum(math.log(x) for x in xs) / len(xs)) if xs else math.nan

    print(f"inputs {len(fitted.data)}; wrote {args.out}")
    groups = [("all", lambda r: True), ("segment", lambda r: not r["gather"]),
              ("gather weighted", lambda r: r["gather"] and r["weighted"]),
              ("gather unweighted", lambda r: r["gather"] and not r["weighted"])]
    for gname, sel in groups:
        sub = [r for r in rep if sel(r)]
        print(f"-- {gname} ({len(sub)} inputs)")
        if not sub:
            continue
        for k in ("nostats", "nostats_ep", "stats", "single_nostats", "single_stats", "paper_nostats", "paper_stats",
                  "hand"):
            v = [r[k] for r in sub]
            w = sum(1 for x in v if x == x and x <= 1.10)
            print(f"   {k:15s} geomean slowdown vs best {gm(v):.3f}  max {np.nanmax(v):.3f}  within 10%: {w}/{len(v)}")
    print("named workloads:")
    for r in rep:
        if r["id"] >= 10000 and r["id"] < 20000:
            print(f"  {r['name']:20s} F={r['F']:3d} {r['op']:4s} w={r['weighted']} best {r['best']:.3f} ms  "
                  f"nostats x{r['nostats']:.3f}  stats x{r['stats']:.3f}  single x{r['single_nostats']:.3f}  "
                  f"paper x{r['paper_stats']:.3f}  hand x{r['hand']:.3f}")
    json.dump(rep, open(os.path.join(HERE, "fit_report.json"), "w"), indent=0)


if __name__ == "__main__":
    main()
