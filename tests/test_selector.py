"""The selector: the committed C++ if/else is exactly what fitting the committed MI355X
performance database produces, the compiled if/else agrees with the fitted trees on
every training input, and the library's geot_select returns the tree's choice.
CPU only (g++ compiles the generated header).
"""
import math
import os
import subprocess

import numpy as np
import pytest

from paper_2404_03019_amd.tune import fit

DB = fit.DEFAULT_DB
HEADER = fit.DEFAULT_OUT

pytestmark = pytest.mark.skipif(not os.path.exists(DB), reason="no performance database committed")

DRIVER = r"""
#include <cstdio>
#include "selector_generated.h"
int main() {
    double nnz, S, F, cv, mx; int op, gather, has;
    while (std::scanf("%lf %lf %lf %d %d %d %lf %lf", &nnz, &S, &F, &op, &gather, &has, &cv, &mx) == 8) {
        int32_t out[6];
        geot::tree_select(nnz, S, F, op, gather, has, cv, mx, out);
        std::printf("%d %d %d %d\n", out[0], out[3], out[4], out[5]);
    }
    return 0;
}
"""


@pytest.fixture(scope="module")
def fitted():
    return fit.build(DB)


def test_committed_header_is_reproducible(fitted):
    assert open(HEADER).read() == fit.render(fitted), \
        "selector_generated.h is stale: rerun python -m paper_2404_03019_amd.tune.fit"


def test_compiled_tree_matches_the_fitted_trees(fitted, tmp_path):
    drv = tmp_path / "drv.cpp"
    drv.write_text(DRIVER)
    exe = str(tmp_path / "drv")
    subprocess.run(["g++", "-O1", "-std=c++17", "-I", os.path.dirname(HEADER), str(drv), "-o", exe],
                   check=True)
    lines, want = [], []
    ops = {"sum": 0, "mean": 1, "max": 2}
    for e in fitted.data:
        f = e["features"]
        g = 0 if not f["gather"] else (1 if fit.weighted_of(e) else 2)
        for has in (0, 1):
            lines.append(f"{f['nnz']} {f['S']} {f['F']} {ops[f['op']]} {g} {has} "
                         f"{f['cv']!r} {f['max_rel']!r}")
            want.append(fitted.choose(e, bool(has)))
    got = subprocess.run([exe], input="\n".join(lines) + "\n", capture_output=True, text=True,
                         check=True).stdout.split("\n")
    mism = [(l, g, w) for l, g, w in zip(lines, got, want)
            if tuple(int(t) for t in g.split()) != tuple(w)]
    # a feature exactly on a threshold may round differently between the two evaluations
    assert len(mism) <= max(1, len(lines) // 200), mism[:5]


def test_library_select_follows_the_tree(fitted):
    import paper_2404_03019_amd as geot

    picks = [e for e in fitted.data if not e["features"]["gather"]][:40] + \
        [e for e in fitted.data if e["features"]["gather"]][:40]
    for e in picks:
        f = e["features"]
        fam, k, g, t = fitted.choose(e, False)
        c = geot.select(f["nnz"], f["S"], f["F"], f["op"], bool(f["gather"]), weighted=bool(fit.weighted_of(e)))
        assert c["family"] == fam and c["rows"] == k, (f, c, (fam, k))
        # column tiles in sequence: lanes of the 4-wide shape divided by the tiles, tile-major order
        tiled = t > 1 and f["F"] % 4 == 0
        assert bool(c["flags"] & 4) == (tiled and f["F"] > 4 * fit.lanes_for(f["F"]) // t), (f, c, t)
        if tiled:
            assert c["lanes"] == max(1, fit.lanes_for(f["F"]) // t), (f, c, t)


def test_selector_beats_the_hand_rule_and_the_paper_recipe(fitted):
    """Measured on MI355X: geometric-mean slowdown against the best measured candidate,
    over all inputs and over the fused-form inputs alone."""
    rep = fit.evaluate(fitted)

    def gm(k, sel=lambda r: True):
        v = [r[k] for r in rep if r[k] == r[k] and sel(r)]
        return math.exp(sum(math.log(x) for x in v) / len(v))

    assert gm("nostats") < gm("paper_nostats") < gm("hand")
    assert gm("stats") < gm("paper_stats")
    # the O(1) tree against the best element-parallel candidate (the family it chooses from)
    assert gm("nostats_ep") <= 1.05
    # the tree with statistics refines the O(1) one: never worse on the database, and within 5 %
    # of the best of every candidate (the segment-parallel family included)
    assert gm("stats") <= gm("nostats") + 1e-9
    assert gm("stats") <= 1.05
    fused = lambda r: r["gather"]
    assert gm("nostats", fused) <= gm("single_nostats", fused) + 1e-9
    assert gm("nostats_ep", fused) <= 1.05
    named = [r for r in rep if 10000 <= r["id"] < 20000]
    # the large named workloads (above 0.2 ms) are within 10% of the best candidate, with or
    # without statistics
    big = [r for r in named if r["best"] >= 0.2]
    assert big and all(r["nostats"] <= 1.10 and r["stats"] <= 1.10 for r in big), big
