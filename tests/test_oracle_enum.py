"""Pins of the oracle's plan enumeration (Sec. 4.2, Alg. 1; Eq. 1).

Expected values come from outside the enumerator:

* the logical plans of the E->L model (two types: text through L, image
  through E -> L) listed by hand from the rules: three simple subplans
  ([L], [E][L], [E+L]), the two that cover both types alone, and the pairs
  with and without shared nodes;
* counts by stars and bars: with one GPU per executor, n_v >= 1 executors
  on V nodes within N GPUs can be chosen in C(N, V) ways, times |K|^V
  configurations and 9 routing weights per type with two alternatives;
* counts with several GPU options by brute force over itertools;
* the physical plans of one logical plan, in order, regenerated here by
  itertools in the stated lexicographic order, compared column by column;
* the fully colocated and fully disaggregated families of the plan
  generator (an independent implementation) as subsets;
* structural invariants on the omni graph (validity and budget by phase 1's
  flags, weights summing to ten, no repeated plan, simple-subplan counts of
  a tree of colocatable edges: 2^edges).
"""
import itertools
from math import comb

import numpy as np
import pytest

from oracle import oracle as O
from paper_2512_14098_amd.inputs import load_config, make_plans
from paper_2512_14098_amd.inputs.plans import PlanTable

KNOBS3 = [16, 64, 256]


def _c1_opts(N=8, share=True, k_s=2, gpus=None):
    cfg = load_config("c1")
    spec = {"k_s": k_s, "share": share, "batch": {"E": KNOBS3, "L": KNOBS3}}
    if gpus:
        spec["gpus"] = gpus
    return cfg, O.make_model(cfg["model"]), O.enum_opts(cfg["model"], spec, N)


def _as_tuple(L, T):
    nodes = tuple(L.node_comp[v] for v in range(L.n_nodes))
    alts = tuple(tuple(tuple(L.alt_node[t][a][c] for c in range(2)) for a in range(L.n_alt[t])) for t in range(T))
    return nodes, alts


X = 255  # off the path
# E = component 0 (mask 1), L = component 1 (mask 2), E+L = mask 3; types: text = [L], image = [E, L]
C1_LOGICAL = [
    ((1, 2), (((X, 1),), ((0, 1),))),                      # [E][L]
    ((3,), (((X, 0),), ((0, 0),))),                        # [E+L]
    ((2, 1, 2), (((X, 0), (X, 2)), ((1, 2),))),            # [L] + [E][L]
    ((2, 1), (((X, 0),), ((1, 0),))),                      # [L] + [E][L], L shared
    ((2, 3), (((X, 0), (X, 1)), ((1, 1),))),               # [L] + [E+L]
    ((1, 2, 1, 2), (((X, 1), (X, 3)), ((0, 1), (2, 3)))),  # [E][L] twice
    ((1, 2, 2), (((X, 1), (X, 2)), ((0, 1), (0, 2)))),     # [E][L] twice, E shared
    ((1, 2, 1), (((X, 1),), ((0, 1), (2, 1)))),            # [E][L] twice, L shared
    ((1, 2, 3), (((X, 1), (X, 2)), ((0, 1), (2, 2)))),     # [E][L] + [E+L]
    ((3, 3), (((X, 0), (X, 1)), ((0, 0), (1, 1)))),        # [E+L] twice
]


def test_logical_plans_of_the_two_type_graph_by_hand():
    cfg, m, o = _c1_opts()
    got = [_as_tuple(L, 2) for L in O.enum_logical(m, o)]
    assert got == C1_LOGICAL
    # without sharing: the shared variants go; with k_s = 1: only the two singles
    _, m, o = _c1_opts(share=False)
    assert [_as_tuple(L, 2) for L in O.enum_logical(m, o)] == [C1_LOGICAL[i] for i in (0, 1, 2, 4, 5, 8, 9)]
    _, m, o = _c1_opts(k_s=1)
    assert [_as_tuple(L, 2) for L in O.enum_logical(m, o)] == C1_LOGICAL[:2]


@pytest.mark.parametrize("N", [1, 2, 3, 8, 17, 64])
def test_counts_stars_and_bars(N):
    cfg, m, o = _c1_opts(N=N)
    for L in O.enum_logical(m, o):
        V = L.n_nodes
        a = sum(1 for t in range(2) if L.n_alt[t] == 2)
        assert O.enum_count(m, o, L) == (3 ** V) * comb(N, V) * 9 ** a


def test_counts_with_gpu_options_brute_force():
    N = 9
    gopt = {"E": [1, 2], "L": [1, 4]}
    cfg, m, o = _c1_opts(N=N, gpus=gopt)
    g_of = {1: [1, 2], 2: [1, 4], 3: [1, 2]}  # lowest component's options per node mask
    for L in O.enum_logical(m, o):
        nodes = [L.node_comp[v] for v in range(L.n_nodes)]
        n = 0
        for gs in itertools.product(*[g_of[mask] for mask in nodes]):
            for ns in itertools.product(range(1, N + 1), repeat=len(nodes)):
                if sum(g * k for g, k in zip(gs, ns)) <= N:
                    n += 3 ** len(nodes)
        a = sum(1 for t in range(2) if L.n_alt[t] == 2)
        assert O.enum_count(m, o, L) == n * 9 ** a


def _brute_plans(L, T, N, knobs, gopts):
    """Every physical plan of logical plan L in the stated order, as plan dicts."""
    V = L.n_nodes
    per_node = []
    for v in range(V):
        mask = L.node_comp[v]
        c0 = (mask & -mask).bit_length() - 1
        cfgs = [(g, b) for g in gopts[c0] for b in knobs[c0]]
        per_node.append(cfgs)

    def assignments(v, budget):
        if v == V:
            yield []
            return
        for (g, b) in per_node[v]:
            for n in range(1, budget // g + 1):
                for rest in assignments(v + 1, budget - g * n):
                    yield [(g, b, n)] + rest

    two = [t for t in range(T) if L.n_alt[t] == 2]
    out = []
    for asg in assignments(0, N):
        for ws in itertools.product(range(1, 10), repeat=len(two)):
            wt = dict(zip(two, ws))
            nodes = [(L.node_comp[v], asg[v][2], asg[v][1], asg[v][0]) for v in range(V)]
            routes = []
            for t in range(T):
                alts = []
                for a in range(L.n_alt[t]):
                    w = 10 if L.n_alt[t] == 1 else (wt[t] if a == 0 else 10 - wt[t])
                    alts.append((w, {c: L.alt_node[t][a][c] for c in range(8) if L.alt_node[t][a][c] != 255}))
                routes.append(alts)
            out.append(dict(nodes=nodes, routes=routes))
    return out


def _table_eq(tab, plans):
    from paper_2512_14098_amd.inputs import plan_table_from_list
    want = plan_table_from_list(plans)
    for f in PlanTable.FIELDS:
        assert np.array_equal(getattr(tab, f), getattr(want, f)), f


def test_physical_plans_in_order_against_itertools():
    N = 4
    gopt = {"E": [1, 2], "L": [1]}
    cfg, m, o = _c1_opts(N=N, gpus=gopt)
    Ls = O.enum_logical(m, o)
    knobs = {0: KNOBS3, 1: KNOBS3}
    gopts = {0: [1, 2], 1: [1]}
    allp = []
    for L in Ls:
        allp += _brute_plans(L, 2, N, knobs, gopts)
    total = sum(O.enum_count(m, o, L) for L in Ls)
    assert total == len(allp)
    # the whole sequence, and windows that start and end inside logical plans
    _table_eq(O.enum_plans(m, o, Ls, 0, total), allp)
    assert total > 5000
    for first, count in ((1, 7), (500, 1000), (total - 3, 3), (total // 2 + 1, 1)):
        _table_eq(O.enum_plans(m, o, Ls, first, count), allp[first:first + count])


def _canon_rows(tab):
    rows = set()
    for p in range(tab.P):
        pl = tab.plan(p)
        rows.add((tuple(tuple(sorted(n.items())) for n in pl["nodes"]),
                  tuple(tuple((a["w"], tuple(a["node"])) for a in r) for r in pl["routes"])))
    return rows


def test_generator_families_are_enumerated():
    cfg, m, o = _c1_opts(N=8)
    Ls = O.enum_logical(m, o)
    tab = O.enum_plans(m, o, Ls, 0, 252 + 24)   # the two singles come first
    got = _canon_rows(tab)
    fam = make_plans(dict(cfg, plans={"families": cfg["plans"]["families"]}), cache=False)
    assert fam.P == 276 and _canon_rows(fam) == got


def test_omni_graph_invariants():
    cfg = load_config("c2")
    mc = cfg["model"]
    m = O.make_model(mc)
    spec = {"k_s": 2, "share": True, "batch": {c["name"]: KNOBS3 for c in mc["components"]}}
    o = O.enum_opts(mc, spec, 16)
    Ls = O.enum_logical(m, o)
    # the colocatable edges of the full graph form a tree of 4 edges: 16 groupings, each a
    # single plan covering all four types
    singles = [L for L in Ls if all(L.n_alt[t] == 1 for t in range(4)) and L.n_nodes <= 5
               and sorted(L.node_comp[v] for v in range(L.n_nodes)) != []]
    full = [L for L in singles if sum(bin(L.node_comp[v]).count("1") for v in range(L.n_nodes)) == 5
            and len({L.node_comp[v] for v in range(L.n_nodes)}) == L.n_nodes]
    assert len(Ls) > 16 and len(full) >= 16
    assert len({(tuple(L.node_comp[:L.n_nodes]),
                 tuple(tuple(tuple(L.alt_node[t][a]) for a in range(L.n_alt[t])) for t in range(4)))
                for L in Ls}) == len(Ls)
    counts = [O.enum_count(m, o, L) for L in Ls]
    # a window of plans across the first logical plans and one deep inside the space
    for first in (0, sum(counts) // 2):
        tab = O.enum_plans(m, o, Ls, first, 3000)
        rd, bn, fl = O.eval_coarse(m, tab, np.array([[1, 400, 150, 600, 4000, 4000, 50, 50]] * 4, np.uint64), 16)
        assert not np.any(fl & 4), "invalid plan"
        assert not np.any(fl & 2), "over budget"
        w = tab.alt_w.reshape(8, 2, -1).astype(int)
        for t in range(4):
            assert np.all(w[t, 0] + w[t, 1] == 10)
        assert len(_canon_rows(tab)) == 3000


def _brute_plans_het(L, T, N, knobs, gopts):
    """As _brute_plans with nodes of two configurations allowed (Eq. 1's n_{v,k} for two k):
    after every one-configuration assignment of a node, its pairs of configurations k1 < k2
    with n1, n2 >= 1 executors and w = 1..9 tenths for the first, in that order."""
    V = L.n_nodes
    per_node = []
    for v in range(V):
        mask = L.node_comp[v]
        c0 = (mask & -mask).bit_length() - 1
        per_node.append([(g, b) for g in gopts[c0] for b in knobs[c0]])

    def node_options(v, budget):
        cf = per_node[v]
        for (g, b) in cf:
            for n in range(1, budget // g + 1):
                yield (n, b, g), g * n
        for i1, i2 in itertools.combinations(range(len(cf)), 2):
            (g1, b1), (g2, b2) = cf[i1], cf[i2]
            for n1 in range(1, budget + 1):
                for n2 in range(1, budget + 1):
                    if g1 * n1 + g2 * n2 > budget:
                        continue
                    for w in range(1, 10):
                        yield (n1, b1, g1, n2, b2, g2, w), g1 * n1 + g2 * n2

    def assignments(v, budget):
        if v == V:
            yield []
            return
        for opt, cost in node_options(v, budget):
            for rest in assignments(v + 1, budget - cost):
                yield [opt] + rest

    two = [t for t in range(T) if L.n_alt[t] == 2]
    out = []
    for asg in assignments(0, N):
        for ws in itertools.product(range(1, 10), repeat=len(two)):
            wt = dict(zip(two, ws))
            nodes = [(L.node_comp[v],) + asg[v] if len(asg[v]) == 7 else
                     (L.node_comp[v], asg[v][0], asg[v][1], asg[v][2]) for v in range(V)]
            routes = []
            for t in range(T):
                alts = []
                for a in range(L.n_alt[t]):
                    w = 10 if L.n_alt[t] == 1 else (wt[t] if a == 0 else 10 - wt[t])
                    alts.append((w, {c: L.alt_node[t][a][c] for c in range(8) if L.alt_node[t][a][c] != 255}))
                routes.append(alts)
            out.append(dict(nodes=nodes, routes=routes))
    return out


@pytest.mark.parametrize("N,gpus", [(3, {"E": [1, 2], "L": [1]}), (4, {"E": [1], "L": [1]})])
def test_two_configuration_nodes_in_order_against_itertools(N, gpus):
    cfg = load_config("c1")
    spec = {"k_s": 2, "share": True, "batch": {"E": [16, 64], "L": [16, 64, 256]}, "gpus": gpus, "het": True}
    m, o = O.make_model(cfg["model"]), O.enum_opts(cfg["model"], spec, N)
    Ls = O.enum_logical(m, o)
    knobs = {0: [16, 64], 1: [16, 64, 256]}
    gopts = {0: gpus["E"], 1: gpus["L"]}
    allp = []
    for L in Ls:
        plans = _brute_plans_het(L, 2, N, knobs, gopts)
        assert O.enum_count(m, o, L) == len(plans)
        allp += plans
    total = len(allp)
    assert total > 2000 and any(len(nd) == 8 for p in allp for nd in p["nodes"])
    tab = O.enum_plans(m, o, Ls, 0, total)
    _table_eq(tab, allp)
    for first, count in ((1, 7), (total // 3, 500), (total - 3, 3)):
        _table_eq(O.enum_plans(m, o, Ls, first, count), allp[first:first + count])
    # every plan is valid for phase 1 and within the budget of Eq. (1) over both configurations
    rd, bn, fl = O.eval_coarse(m, tab, O.trace_gen(m, [0], 2000)["moments"][0], N)
    assert np.all((fl & 6) == 0)
    # without the option the same space holds only the one-configuration plans, in order
    o1 = O.enum_opts(cfg["model"], dict(spec, het=False), N)
    one = [p for p in allp if all(len(nd) == 4 for nd in p["nodes"])]
    assert sum(O.enum_count(m, o1, L) for L in Ls) == len(one)
    _table_eq(O.enum_plans(m, o1, Ls, 0, len(one)), one)
