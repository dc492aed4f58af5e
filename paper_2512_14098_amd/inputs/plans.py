"""Physical-plan tables (Sec. 4.2, Alg. 1 and Eq. 1 of the paper).

A plan is a set of nodes, each hosting a set of model components (a
colocated group when more than one), with ``replicas`` executors of
``gpus`` GPUs each and a maximum batch, plus per request type at most two
alternative paths (parallel subplans, k_s = 2) with routing weights in
tenths (step 0.1).  Each alternative maps every component on the type's
path to the node that serves it.

Layout (structure of arrays, field slot major, plan index fastest, so that
one GPU thread per plan reads coalesced):

=============  =======  ===========  ==========================================
field          dtype    shape        meaning
=============  =======  ===========  ==========================================
n_nodes        uint8    [P]          nodes in the plan (<= 16)
node_comp      uint8    [16, P]      component bitmask hosted by node v
node_rep       uint8    [16, P]      executors (replicas) of node v
node_batch     uint16   [16, P]      max batch of node v (<= 256)
node_gpus      uint8    [16, P]      GPUs per executor of node v
node_rep2      uint8    [16, P]      executors of node v's second configuration (0: none)
node_batch2    uint16   [16, P]      max batch of that second configuration
node_gpus2     uint8    [16, P]      GPUs per executor of that second configuration
node_w         uint8    [16, P]      tenths of node v's requests to its first configuration
n_alt          uint8    [8, P]       alternatives of type t (1 or 2)
alt_w          uint8    [16, P]      slot 2t+a: weight of alternative a, tenths
alt_node       uint8    [128, P]     slot (2t+a)*8+c: node serving component c
=============  =======  ===========  ==========================================

Three families are produced: fully colocated (every component in one node),
fully disaggregated (one node per component; replicas by coin change,
Eq. 1), and seeded samples of mixed / compound plans: one or two subplans,
each covering a subset of the types, each edge of a subplan kept or merged,
optional node sharing between the two subplans, replicas drawn within the
GPU budget, batches from the knob set, routing weights in tenths, and (with the
sampler option ``het`` > 0, the probability per node of two or more executors)
a node's executors split between two batch configurations with the share of the
node's requests for the first drawn in tenths (Eq. 1's executors of several
configurations per node).
"""
import hashlib
import itertools
import os
import sys

import numpy as np

MAXV, MAXT, MAXC = 16, 8, 8


class PlanTable:
    FIELDS = ("n_nodes", "node_comp", "node_rep", "node_batch", "node_gpus", "n_alt", "alt_w",
              "alt_node", "node_rep2", "node_batch2", "node_gpus2", "node_w")

    def __init__(self, P):
        self.P = int(P)
        self.n_nodes = np.zeros(P, np.uint8)
        self.node_comp = np.zeros((MAXV, P), np.uint8)
        self.node_rep = np.zeros((MAXV, P), np.uint8)
        self.node_batch = np.zeros((MAXV, P), np.uint16)
        self.node_gpus = np.zeros((MAXV, P), np.uint8)
        self.n_alt = np.zeros((MAXT, P), np.uint8)
        self.alt_w = np.zeros((2 * MAXT, P), np.uint8)
        self.alt_node = np.full((2 * MAXT * MAXC, P), 255, np.uint8)
        # a node's second executor configuration (Eq. 1: executors of several configurations
        # per node): none by default, all of a node's requests to its first (10 tenths)
        self.node_rep2 = np.zeros((MAXV, P), np.uint8)
        self.node_batch2 = np.zeros((MAXV, P), np.uint16)
        self.node_gpus2 = np.zeros((MAXV, P), np.uint8)
        self.node_w = np.full((MAXV, P), 10, np.uint8)

    def subset(self, ids):
        ids = np.asarray(ids, dtype=np.int64)
        out = PlanTable(len(ids))
        for f in self.FIELDS:
            a = getattr(self, f)
            setattr(out, f, np.ascontiguousarray(a[..., ids]))
        return out

    def plan(self, p):
        """Readable dict of plan p (for reports and tests)."""
        nv = int(self.n_nodes[p])
        nodes = [dict(comp=int(self.node_comp[v, p]), rep=int(self.node_rep[v, p]),
                      batch=int(self.node_batch[v, p]), gpus=int(self.node_gpus[v, p]),
                      rep2=int(self.node_rep2[v, p]), batch2=int(self.node_batch2[v, p]),
                      gpus2=int(self.node_gpus2[v, p]), w=int(self.node_w[v, p]))
                 for v in range(nv)]
        routes = []
        for t in range(MAXT):
            na = int(self.n_alt[t, p])
            if na == 0:
                break
            routes.append([dict(w=int(self.alt_w[2 * t + a, p]),
                                node=[int(self.alt_node[(2 * t + a) * 8 + c, p]) for c in range(MAXC)])
                           for a in range(na)])
        return dict(nodes=nodes, routes=routes)


def _model_index(model):
    names = [c["name"] for c in model["components"]]
    idx = {n: i for i, n in enumerate(names)}
    paths = [sorted(idx[c] for c in t["comps"]) for t in model["types"]]
    edges = [sorted((idx[a], idx[b]) for a, b in t.get("edges", [])) for t in model["types"]]
    return names, idx, paths, edges


def plan_table_from_list(plans, P=None):
    """plans: list of dict(nodes=[(comp_mask, rep, batch, gpus[, rep2, batch2, gpus2, w])],
    routes=[[(w, {c: node})]]); the optional second executor configuration of a node: rep2
    executors of batch2 and gpus2, w tenths of the node's requests to the first."""
    P = len(plans) if P is None else P
    tab = PlanTable(P)
    for p, pl in enumerate(plans):
        tab.n_nodes[p] = len(pl["nodes"])
        for v, nd in enumerate(pl["nodes"]):
            cm, rep, b, g = nd[:4]
            tab.node_comp[v, p] = cm
            tab.node_rep[v, p] = rep
            tab.node_batch[v, p] = b
            tab.node_gpus[v, p] = g
            if len(nd) > 4:
                tab.node_rep2[v, p], tab.node_batch2[v, p], tab.node_gpus2[v, p], tab.node_w[v, p] = nd[4:8]
        for t, alts in enumerate(pl["routes"]):
            tab.n_alt[t, p] = len(alts)
            for a, (w, cmap) in enumerate(alts):
                tab.alt_w[2 * t + a, p] = w
                for c, v in cmap.items():
                    tab.alt_node[(2 * t + a) * 8 + c, p] = v
    return tab


def _single_route(paths, node_of):
    return [[(10, {c: node_of[c] for c in path})] for path in paths]


def _colocated(model, fam, gpus):
    names, idx, paths, _ = _model_index(model)
    mask = (1 << len(names)) - 1
    lo, hi = fam["replicas"]
    out = []
    for rep in range(lo, hi + 1):
        if rep > gpus:
            continue
        for b in fam["batch"]:
            out.append(dict(nodes=[(mask, rep, b, 1)],
                            routes=_single_route(paths, {c: 0 for c in range(len(names))})))
    return out


def _disaggregated(model, fam, gpus):
    names, idx, paths, _ = _model_index(model)
    C = len(names)
    maxt = min(int(fam.get("max_total", gpus)), gpus)
    out = []
    reps_all = [r for r in itertools.product(range(1, maxt + 1), repeat=C) if sum(r) <= maxt]
    for reps in reps_all:
        if fam.get("same_batch", False):
            bsets = [(b,) * C for b in fam["batch"]]
        else:
            bsets = list(itertools.product(fam["batch"], repeat=C))
        for bs in bsets:
            nodes = [(1 << c, reps[c], bs[c], 1) for c in range(C)]
            out.append(dict(nodes=nodes, routes=_single_route(paths, {c: c for c in range(C)})))
    return out


def _candidate(ctx, j):
    """Candidate plan j of the sampler (its own Philox stream, keyed by the config's seed
    with counter j), as its canonical encoding, or None if it does not fit the budget."""
    T, C, paths, edges, colocatable, knobs, gpus, seed, het = ctx
    rng = np.random.Generator(np.random.Philox(key=seed, counter=j))
    ns = 1 if rng.random() < 0.5 or T == 1 else 2
    if ns == 1:
        cover = [list(range(T))]
    else:
        while True:
            assign = rng.integers(0, 3, size=T)
            s0 = [t for t in range(T) if assign[t] in (0, 2)]
            s1 = [t for t in range(T) if assign[t] in (1, 2)]
            if s0 and s1:
                break
        cover = [s0, s1]
    nodes, node_of, sub_nodes = [], [], []
    for si, types_s in enumerate(cover):
        comps = sorted(set(c for t in types_s for c in paths[t]))
        es = sorted(set(e for t in types_s for e in edges[t]))
        par = {c: c for c in comps}

        def find(c):
            while par[c] != c:
                c = par[c]
            return c
        for (a, b) in es:
            if colocatable is not None and (a, b) not in colocatable:
                continue
            if rng.random() < 0.5:
                ra, rb = find(a), find(b)
                if ra != rb:
                    par[max(ra, rb)] = min(ra, rb)
        groups = {}
        for c in comps:
            groups.setdefault(find(c), 0)
            groups[find(c)] |= 1 << c
        nmap, mine = {}, []
        for root in sorted(groups):
            mask = groups[root]
            shared = None
            if si == 1 and rng.random() < 0.5:
                for v in sub_nodes[0]:
                    if nodes[v] == mask:
                        shared = v
                        break
            if shared is None:
                shared = len(nodes)
                nodes.append(mask)
            mine.append(shared)
            for c in range(C):
                if (mask >> c) & 1:
                    nmap[c] = shared
        node_of.append(nmap)
        sub_nodes.append(mine)
    V = len(nodes)
    if V > gpus or V > MAXV:
        return None
    reps = [1] * V
    extra = gpus - V
    k = int(rng.integers(0, extra + 1))
    if k:  # k draws of the node that gets one more replica
        for v, more in enumerate(np.bincount(rng.integers(0, V, size=k), minlength=V).tolist()):
            reps[v] += more
    batch = []
    for mask in nodes:
        first = (mask & -mask).bit_length() - 1
        batch.append(int(knobs[first][int(rng.integers(0, len(knobs[first])))]))
    second = [()] * V
    if het > 0:  # a node of 2+ executors may split them between two batch configurations
        for v, mask in enumerate(nodes):
            if reps[v] >= 2 and rng.random() < het:
                first = (mask & -mask).bit_length() - 1
                others = [int(b) for b in knobs[first] if int(b) != batch[v]]
                if others:
                    r2 = int(rng.integers(1, reps[v]))
                    b2 = others[int(rng.integers(0, len(others)))]
                    w = int(rng.integers(1, 10))
                    second[v] = (r2, b2, 1, w)
                    reps[v] -= r2
    routes = []
    for t in range(T):
        alts = [si for si in range(ns) if t in cover[si]]
        if len(alts) == 1:
            routes.append([(10, {c: node_of[alts[0]][c] for c in paths[t]})])
        else:
            w0 = int(rng.integers(1, 10))
            routes.append([(w0, {c: node_of[alts[0]][c] for c in paths[t]}),
                           (10 - w0, {c: node_of[alts[1]][c] for c in paths[t]})])
    return _row(dict(nodes=[(nodes[v], reps[v], batch[v], 1) + second[v] for v in range(V)], routes=routes))


def _candidates(ctx, lo, hi):
    return [_candidate(ctx, j) for j in range(lo, hi)]


# One plan as the bytes of its table column (a canonical encoding: two plans are equal
# iff their columns are): n_nodes, node_comp[16], node_rep[16], node_batch[16] (u16,
# little endian), node_gpus[16], n_alt[8], alt_w[16], alt_node[128], node_rep2[16],
# node_batch2[16] (u16), node_gpus2[16], node_w[16].
_ROW_OFF = dict(n_nodes=0, node_comp=1, node_rep=1 + MAXV, node_batch=1 + 2 * MAXV, node_gpus=1 + 4 * MAXV,
                n_alt=1 + 5 * MAXV, alt_w=1 + 5 * MAXV + MAXT, alt_node=1 + 5 * MAXV + 3 * MAXT)
_ROW_OFF["node_rep2"] = _ROW_OFF["alt_node"] + 2 * MAXT * MAXC
_ROW_OFF["node_batch2"] = _ROW_OFF["node_rep2"] + MAXV
_ROW_OFF["node_gpus2"] = _ROW_OFF["node_batch2"] + 2 * MAXV
_ROW_OFF["node_w"] = _ROW_OFF["node_gpus2"] + MAXV
ROW_BYTES = _ROW_OFF["node_w"] + MAXV
_ROW_TEMPLATE = (bytes(_ROW_OFF["alt_node"]) + bytes([255]) * (2 * MAXT * MAXC) + bytes(4 * MAXV)
                 + bytes([10]) * MAXV)


def _row(pl):
    b = bytearray(_ROW_TEMPLATE)
    b[0] = len(pl["nodes"])
    o = _ROW_OFF
    for v, nd in enumerate(pl["nodes"]):
        cm, rep, bt, g = nd[:4]
        b[o["node_comp"] + v] = cm
        b[o["node_rep"] + v] = rep
        b[o["node_batch"] + 2 * v] = bt & 255
        b[o["node_batch"] + 2 * v + 1] = bt >> 8
        b[o["node_gpus"] + v] = g
        if len(nd) > 4:
            r2, b2, g2, w = nd[4:8]
            b[o["node_rep2"] + v] = r2
            b[o["node_batch2"] + 2 * v] = b2 & 255
            b[o["node_batch2"] + 2 * v + 1] = b2 >> 8
            b[o["node_gpus2"] + v] = g2
            b[o["node_w"] + v] = w
    for t, alts in enumerate(pl["routes"]):
        b[o["n_alt"] + t] = len(alts)
        for a, (w, cmap) in enumerate(alts):
            b[o["alt_w"] + 2 * t + a] = w
            for c, v in cmap.items():
                b[o["alt_node"] + (2 * t + a) * MAXC + c] = v
    return bytes(b)


def table_from_rows(rows):
    """Plan table from column bytes (``_row``), in order."""
    P = len(rows)
    tab = PlanTable(P)
    if P == 0:
        return tab
    R = np.frombuffer(b"".join(rows), np.uint8).reshape(P, ROW_BYTES)
    o = _ROW_OFF
    tab.n_nodes = np.ascontiguousarray(R[:, 0])
    tab.node_comp = np.ascontiguousarray(R[:, o["node_comp"]:o["node_comp"] + MAXV].T)
    tab.node_rep = np.ascontiguousarray(R[:, o["node_rep"]:o["node_rep"] + MAXV].T)
    nb = np.ascontiguousarray(R[:, o["node_batch"]:o["node_batch"] + 2 * MAXV]).view("<u2")
    tab.node_batch = np.ascontiguousarray(nb.T.astype(np.uint16))
    tab.node_gpus = np.ascontiguousarray(R[:, o["node_gpus"]:o["node_gpus"] + MAXV].T)
    tab.n_alt = np.ascontiguousarray(R[:, o["n_alt"]:o["n_alt"] + MAXT].T)
    tab.alt_w = np.ascontiguousarray(R[:, o["alt_w"]:o["alt_w"] + 2 * MAXT].T)
    tab.alt_node = np.ascontiguousarray(R[:, o["alt_node"]:o["alt_node"] + 2 * MAXT * MAXC].T)
    tab.node_rep2 = np.ascontiguousarray(R[:, o["node_rep2"]:o["node_rep2"] + MAXV].T)
    nb2 = np.ascontiguousarray(R[:, o["node_batch2"]:o["node_batch2"] + 2 * MAXV]).view("<u2")
    tab.node_batch2 = np.ascontiguousarray(nb2.T.astype(np.uint16))
    tab.node_gpus2 = np.ascontiguousarray(R[:, o["node_gpus2"]:o["node_gpus2"] + MAXV].T)
    tab.node_w = np.ascontiguousarray(R[:, o["node_w"]:o["node_w"] + MAXV].T)
    return tab


def _sample(model, spec, gpus, have, total, progress=True):
    """Seeded mixed / compound plans until ``total`` distinct plans exist, as column bytes:
    candidates j = 0, 1, 2, ... in order, each drawn from its own Philox stream (key = the
    config's seed, counter = j), the ones over the budget or already present (``have``:
    column bytes) skipped.  Large counts draw the candidates in worker processes; the
    result does not depend on how."""
    names, idx, paths, edges = _model_index(model)
    T, C = len(paths), len(names)
    colocatable = model.get("colocatable")
    if colocatable is not None:
        colocatable = {(idx[a], idx[b]) for a, b in colocatable}
    knobs = [spec["batch"][n] for n in names]
    ctx = (T, C, paths, edges, colocatable, knobs, int(gpus), int(spec["seed"]), float(spec.get("het", 0.0)))
    need = total - len(have)
    seen = set(have)
    out = []
    workers = min(16, os.cpu_count() or 1) if need >= 50000 else 1
    block = 1 << 16 if workers > 1 else 4096
    pool = None
    if workers > 1:
        import concurrent.futures as cfut
        import multiprocessing as mp
        pool = cfut.ProcessPoolExecutor(max_workers=workers, mp_context=mp.get_context("spawn"))

    def submit(j):
        if pool is None:
            return j
        step = block // workers
        return [pool.submit(_candidates, ctx, a, a + step) for a in range(j, j + block, step)]

    def collect(h):
        if pool is None:
            return _candidates(ctx, h, h + block)
        return [k for f in h for k in f.result()]
    try:
        j = 0
        try:
            pending = submit(j)
            keys0 = collect(pending)
        except Exception:  # no worker processes here (e.g. a caller without a main guard)
            if pool is None:
                raise
            pool.shutdown(cancel_futures=True)
            pool, block = None, 4096
            keys0 = None
        pending = j if keys0 is None else None
        while len(out) < need:
            if j > 50 * total + 1000:
                raise RuntimeError("plan sampler could not reach the requested count")
            keys = keys0 if pending is None else collect(pending)
            j += block
            pending = submit(j)  # the next block is drawn while this one is merged
            for key in keys:
                if key is None or key in seen:
                    continue
                seen.add(key)
                out.append(key)
                if len(out) == need:
                    break
            if total >= 200000 and progress:
                print("plans: %d of %d sampled" % (len(have) + len(out), total), file=sys.stderr, flush=True)
    finally:
        if pool is not None:
            pool.shutdown(cancel_futures=True)
    return out


def _cache_path(cfg):
    h = hashlib.sha1(repr((cfg["model"], cfg["plans"], cfg["gpus"], PlanTable.FIELDS)).encode()).hexdigest()[:16]
    d = os.environ.get("CF_PLAN_CACHE", os.path.join(os.path.expanduser("~"), ".cache", "cf_plans"))
    return os.path.join(d, "%s_%s.npz" % (cfg.get("name", "cfg"), h))


def make_plans(cfg, cache=True):
    """Plan table for a configuration (deterministic; cached on disk when large).  A large
    sampled table is drawn in spawned worker processes, which import the caller's main
    script: a script that builds one needs the usual ``if __name__ == "__main__"`` guard
    (without it the table is drawn in this process, with the same result)."""
    cpath = _cache_path(cfg)
    if cache and os.path.exists(cpath):
        z = np.load(cpath)
        tab = PlanTable(int(z["n_nodes"].shape[0]))
        for f in PlanTable.FIELDS:
            setattr(tab, f, np.ascontiguousarray(z[f]))
        return tab
    model, spec, gpus = cfg["model"], cfg["plans"], int(cfg["gpus"])
    plans = []
    for fam in spec.get("families", []):
        if fam["family"] == "colocated":
            plans += _colocated(model, fam, gpus)
        elif fam["family"] == "disaggregated":
            plans += _disaggregated(model, fam, gpus)
        else:
            raise ValueError(fam["family"])
    seen, rows = set(), []
    for p in plans:
        k = _row(p)
        if k not in seen:
            seen.add(k)
            rows.append(k)
    if "sampled" in spec:
        rows += _sample(model, spec["sampled"], gpus, rows, int(spec["sampled"]["total"]))
    tab = table_from_rows(rows)
    if cache and tab.P >= 5000:
        os.makedirs(os.path.dirname(cpath), exist_ok=True)
        tmp = cpath + ".tmp%d.npz" % os.getpid()
        np.savez(tmp, **{f: getattr(tab, f) for f in PlanTable.FIELDS})
        os.replace(tmp, cpath)
    return tab
