"""Small builders for hand-made models, plans and traces used by the tests."""
from fractions import Fraction

import numpy as np

from paper_2512_14098_amd.inputs import plan_table_from_list

TRACE_FIELDS = [("arr_ticks", np.uint64), ("type", np.uint8), ("n_img", np.uint8),
                ("patches", np.uint16), ("prompt", np.uint16), ("out", np.uint16),
                ("aud_in_ms", np.uint32), ("aud_out_ms", np.uint32), ("rkey0", np.uint64),
                ("rkey1", np.uint64), ("akey", np.uint32)]


def ticks_of(t_seconds):
    """Integer tick count (2^-32 s at rate 1) nearest to t, and its exact arrival time."""
    k = int(round(t_seconds * 2 ** 32))
    return k, Fraction(k, 2 ** 32)


def make_trace(reqs, n_seeds=1):
    """reqs: list of dicts with keys t (seconds at rate 1), type, patches, prompt, out,
    aud_in_ms, aud_out_ms, rkey0, rkey1, akey (missing keys are 0)."""
    n = len(reqs)
    tr = {f: np.zeros(n_seeds * n, dt) for f, dt in TRACE_FIELDS}
    for s in range(n_seeds):
        for i, r in enumerate(reqs):
            o = s * n + i
            tr["arr_ticks"][o] = ticks_of(r.get("t", 0.0))[0]
            for f, _ in TRACE_FIELDS[1:]:
                tr[f][o] = r.get(f, 0)
    tr["n_seeds"], tr["n_req"] = n_seeds, n
    return tr


def comp(name, kind, k, x=(), decode=(0.0, 0.0), n_out="out", gate=None, batch_cap=256):
    c = {"name": name, "kind": kind, "k": list(k), "x": list(x), "decode": list(decode),
         "n_out": n_out, "batch_cap": batch_cap}
    if gate:
        c["gate"] = gate
    return c


def rtype(name, comps, edges=(), outputs=None, weight=1, slo=None, **dists):
    t = {"name": name, "weight": weight, "comps": list(comps), "edges": [list(e) for e in edges],
         "outputs": list(outputs or [comps[-1]]), "slo": dict(slo or {})}
    t.update(dists)
    return t


def model(components, types, comm=0.010, cpu_pre=0.0, theta=(9, 10), patches=(256, 1024)):
    return {"components": components, "types": types, "comm_s": comm, "cpu_pre_s": cpu_pre,
            "theta": list(theta), "patches_per_image": list(patches)}


def one_plan(nodes, routes):
    """nodes: list of (comp_mask, rep, batch[, gpus]); routes: per type list of (w, {c: node})."""
    nn = [tuple(n) + ((1,) if len(n) == 3 else ()) for n in nodes]
    return plan_table_from_list([dict(nodes=nn, routes=routes)])


def F(x):
    """Exact rational value of a double."""
    return Fraction(float(x))
