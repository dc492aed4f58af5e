"""The oracle's simulations spread over worker processes (test infrastructure only).

A worker rebuilds the oracle's model from the configuration, generates the trace of its
own seeds with the oracle and simulates its share of the (plan, rate, seed) triples; it
imports neither torch nor the HIP binding.  Used by the GPU tests that compare whole
configurations with the oracle at their full seed counts.
"""
import concurrent.futures as cfut
import multiprocessing as mp
import os

import numpy as np


def workers():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _chunk(args):
    from oracle import oracle as O
    mcfg, tab, seeds, n, rates, seed_idx = args
    m = O.make_model(mcfg)
    tr = O.trace_gen(m, [seeds[s] for s in seed_idx], n)
    n_plans, K = rates.shape
    T = m.n_types
    met = np.zeros((n_plans, K, len(seed_idx), T), np.uint32)
    cnt = np.zeros_like(met)
    ev = np.zeros((n_plans, K, len(seed_idx)), np.uint64)
    st = np.zeros((n_plans, K, len(seed_idx)), np.uint32)
    pst, tst = O.plans_struct(tab), O.trace_struct(tr)
    for i in range(n_plans):
        for k in range(K):
            for j in range(len(seed_idx)):
                o = O.sim_triple(m, tab, i, float(rates[i, k]), tr, j, _pst=pst, _tst=tst)
                met[i, k, j], cnt[i, k, j], ev[i, k, j], st[i, k, j] = o["met"], o["cnt"], o["events"], o["status"]
    return seed_idx, met, cnt, ev, st


def eval_fine_seeds(mcfg, tab, seeds, n, rates, seed_idx):
    """Oracle counts [n_plans, K, len(seed_idx), T], events and status of plans 0..n_plans-1
    of tab at rates [n_plans, K] on the seeds seeds[s] for s in seed_idx, seeds dealt over
    the worker processes."""
    nw = min(workers(), len(seed_idx))
    parts = [list(seed_idx[w::nw]) for w in range(nw)]
    # an executor (not a Pool) so that workers that cannot start raise instead of being restarted
    with cfut.ProcessPoolExecutor(max_workers=nw, mp_context=mp.get_context("spawn")) as pool:
        res = list(pool.map(_chunk, [(mcfg, tab, list(seeds), n, rates, p) for p in parts]))
    pos = {s: j for j, s in enumerate(seed_idx)}
    n_plans, K = rates.shape
    T = res[0][1].shape[3]
    met = np.zeros((n_plans, K, len(seed_idx), T), np.uint32)
    cnt = np.zeros_like(met)
    ev = np.zeros((n_plans, K, len(seed_idx)), np.uint64)
    st = np.zeros((n_plans, K, len(seed_idx)), np.uint32)
    for sidx, a, b, c, d in res:
        for j, s in enumerate(sidx):
            met[:, :, pos[s]], cnt[:, :, pos[s]], ev[:, :, pos[s]], st[:, :, pos[s]] = a[:, :, j], b[:, :, j], c[:, :, j], d[:, :, j]
    return met, cnt, ev, st
