"""Fits the library's default algorithm choice from measured timings.

The paper's comparison includes a heuristic pick ("guess": the algorithm a
vendor library predicts for a layer without timing it, Sec. V-B) next to
measured selection.  This script builds such a predictor for this library
from per-layer, per-algorithm timings taken with ``bench.py --sweep``:

* training set: ``tables/sweep_fit.jsonl`` -- the 20-layer random chains of
  the algorithm sweep at seeds 1..8 and seeded independent layers of mixed
  kind (dtype, depthwise / grouped, filter size, stride, dilation, batch,
  plane size); the five benchmark workloads are NOT in it;
* model: a depth-limited regression tree over shape features (the same
  features the library computes from a descriptor) whose targets are every
  algorithm's log2 slowdown on the layer (time / best time; an algorithm
  that does not support the layer counts as 10x slower); each leaf then
  ranks the algorithms by their summed slowdown over the training layers of
  the leaf, and the library takes the first algorithm of the ranking that
  supports the layer.  Depth and leaf size were chosen by leave-one-set-out
  cross-validation on the training set alone (``--cv`` prints the grid: the
  geometric mean over held-out sets of fitted network time / best network
  time);
* output: ``csrc/guess_tree.inc`` (node and ranking tables, C++), and a
  report of the held-out network times on ``tables/sweep_workloads.jsonl``
  (the five benchmark workloads).

Run from the repository root:  python -m paper_2410_08300_amd.fit_guess
Tests import it to check that the library walks the same tree.
"""
import json
import math
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
TRAIN = os.path.join(HERE, "tables", "sweep_fit.jsonl")
HELD_OUT = os.path.join(HERE, "tables", "sweep_workloads.jsonl")
OUT = os.path.join(HERE, "csrc", "guess_tree.inc")

# conv_algo_t values (include/convsel.h).
ALGO_IDS = {"direct": 1, "implicit_gemm": 2, "im2col_gemm": 3, "winograd": 4, "implicit_precomp_gemm": 5,
            "kn2row": 6, "smm": 7}
ALGOS = sorted(ALGO_IDS, key=ALGO_IDS.get)
FEATURES = ("bf16", "depthwise", "taps", "stride", "log2_cg", "log2_kg", "log2_npq", "log2_pq", "winograd_ok",
            "dilated", "grouped")
UNSUPPORTED_PENALTY = 10.0
MAX_DEPTH = 8
MIN_LEAF = 2


def out_size(h, pad, dil, r, stride):
    return (h + 2 * pad - dil * (r - 1) - 1) // stride + 1


def features(shape):
    """Feature vector of a layer given as the sweep's shape dict (the same
    quantities the library derives from a descriptor, in the same order)."""
    n, c, h, w, k = shape["n"], shape["c"], shape["h"], shape["w"], shape["k"]
    r, s, st, pad, dil, g = shape["r"], shape["s"], shape["stride"], shape["pad"], shape["dilation"], shape["groups"]
    p, q = out_size(h, pad, dil, r, st), out_size(w, pad, dil, s, st)
    cg, kg = c // g, k // g
    wino = int(r == 3 and s == 3 and st == 1 and dil == 1 and g == 1)
    return [float(shape["dtype"] == "bf16"), float(cg == 1), float(r * s), float(st), math.log2(cg), math.log2(kg),
            math.log2(n * p * q), math.log2(p * q), float(wino), float(dil > 1), float(g > 1 and cg > 1)]


def load(path):
    """{(set, layer): {"shape": dict, "count": int, "ms": {algo: ms}}}."""
    layers = {}
    with open(path) as f:
        for line in f:
            r = json.loads(line)
            e = layers.setdefault((r["workload"], r["layer"]), {"shape": r["shape"], "count": r["count"], "ms": {}})
            e["ms"][r["algo"]] = r["ms"]
    return layers


def slowdown(ms, a):
    return ms[a] / min(ms.values()) if a in ms else UNSUPPORTED_PENALTY


def fit(train, max_depth=MAX_DEPTH, min_leaf=MIN_LEAF):
    from sklearn.tree import DecisionTreeRegressor
    keys = sorted(train)
    X = np.array([features(train[k]["shape"]) for k in keys])
    Y = np.array([[math.log2(slowdown(train[k]["ms"], a)) for a in ALGOS] for k in keys])
    tree = DecisionTreeRegressor(max_depth=max_depth, min_samples_leaf=min_leaf, random_state=0)
    tree.fit(X, Y)
    t = tree.tree_
    leaf_of = tree.apply(X)
    leaves = sorted(set(leaf_of.tolist()))
    rank = {}
    for lf in leaves:
        members = [k for i, k in enumerate(keys) if leaf_of[i] == lf]
        cost = {a: sum(slowdown(train[k]["ms"], a) for k in members) for a in ALGOS}
        rank[lf] = sorted(ALGOS, key=lambda a: (cost[a], ALGO_IDS[a]))
    nodes = []
    for i in range(t.node_count):
        if t.children_left[i] < 0:
            nodes.append((-1, 0.0, -1, -1, leaves.index(i)))
        else:
            nodes.append((int(t.feature[i]), float(t.threshold[i]), int(t.children_left[i]),
                          int(t.children_right[i]), -1))
    return nodes, [rank[lf] for lf in leaves]


def predict_ranking(nodes, ranks, shape):
    f = features(shape)
    i = 0
    while nodes[i][0] >= 0:
        feat, thr, left, right, _ = nodes[i]
        i = left if f[feat] <= thr else right
    return ranks[nodes[i][4]]


def predict(nodes, ranks, shape, supported):
    """First algorithm of the leaf's ranking among `supported` (names)."""
    for a in predict_ranking(nodes, ranks, shape):
        if a in supported:
            return a
    return "direct"


def write_inc(nodes, ranks, path=OUT):
    L = ["// Decision tree of the default algorithm choice.  Generated by",
         "// paper_2410_08300_amd/fit_guess.py from tables/sweep_fit.jsonl; do not edit.",
         "// Features (in order): " + ", ".join(FEATURES) + ".",
         "// Node: {feature, threshold, left, right, leaf}; go left when feature <= threshold;",
         "// feature < 0 marks a leaf, whose ranking row lists conv_algo_t values, best first.",
         "static const GuessNode kGuessNodes[] = {"]
    for feat, thr, left, right, leaf in nodes:
        L.append("    {%d, %s, %d, %d, %d}," % (feat, repr(float(thr)), left, right, leaf))
    L.append("};")
    L.append("static const int kGuessRank[][%d] = {" % len(ALGOS))
    for r in ranks:
        L.append("    {%s}," % ", ".join(str(ALGO_IDS[a]) for a in r))
    L.append("};")
    with open(path, "w") as f:
        f.write("\n".join(L) + "\n")


def report(nodes, ranks, data):
    """Network time (sum of count x per-layer ms) per set: best per layer,
    the fitted pick, and each single algorithm."""
    sets = sorted({k[0] for k in data})
    rows = []
    for st in sets:
        ks = [k for k in data if k[0] == st]
        best = sum(min(data[k]["ms"].values()) * data[k]["count"] for k in ks)
        pick = 0.0
        for k in ks:
            a = predict(nodes, ranks, data[k]["shape"], list(data[k]["ms"]))
            pick += data[k]["ms"][a] * data[k]["count"]
        single = {a: sum(data[k]["ms"][a] * data[k]["count"] for k in ks) if all(a in data[k]["ms"] for k in ks)
                  else None for a in ALGOS}
        rows.append((st, best, pick, single))
    return rows


def cross_validate(train):
    """Leave-one-set-out geometric-mean network slowdown per (depth, leaf)."""
    sets = sorted({k[0] for k in train})
    for depth in (4, 5, 6, 8, 10):
        for leaf in (1, 2, 3, 5):
            logs = []
            for held in sets:
                nodes, ranks = fit({k: v for k, v in train.items() if k[0] != held}, depth, leaf)
                for _, best, pick, _ in report(nodes, ranks, {k: v for k, v in train.items() if k[0] == held}):
                    logs.append(math.log(pick / best))
            print("depth %2d min_leaf %d: cv slowdown %.3f" % (depth, leaf, math.exp(sum(logs) / len(logs))))


def main():
    import sys
    train = load(TRAIN)
    if "--cv" in sys.argv:
        cross_validate(train)
        return
    nodes, ranks = fit(train)
    write_inc(nodes, ranks)
    print("tree: %d nodes, %d leaves; written %s" % (len(nodes), len(ranks), OUT))
    for name, path in (("training", TRAIN), ("held out", HELD_OUT)):
        if not os.path.exists(path):
            continue
        print("== %s (%s)" % (name, os.path.basename(path)))
        for st, best, pick, single in report(nodes, ranks, load(path)):
            sing = " ".join("%s=%.3f" % (a, v) for a, v in single.items() if v is not None)
            print("%-14s best %.3f ms  fitted %.3f ms (%.3fx)  %s" % (st, best, pick, pick / best, sing))


if __name__ == "__main__":
    main()
