"""bench.py's command line on the host: more than one GPU is refused with a message
before anything touches a GPU; the CPU baseline picks its triples with the oracle."""
import os
import subprocess
import sys
import types

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_cpu_baseline_samples_the_oracles_own_selection():
    import bench
    from paper_2512_14098_amd.inputs import load_config, make_plans, seeds_of
    cfg = load_config("c0")
    tab = make_plans(cfg)
    r = cfg["rates"]
    w = types.SimpleNamespace(cfg=cfg, tab=tab, seeds=seeds_of(cfg), n_req=int(cfg["n_req"]), n_gpus=int(cfg["gpus"]),
                              top_k=int(cfg.get("top_k") or tab.P), explicit_rates=r.get("explicit"),
                              K=len(r["explicit"]), alpha_max=1.0)
    res = bench.cpu_baseline(w, 0.5)
    assert res["kind"] == "oracle" and res["cores"] == 1 and res["value"] > 0
    assert "all_cores" not in res
