"""Workload configuration loading (JSON, no computation)."""
import copy
import json
import os

_DIR = os.path.join(os.path.dirname(os.path.abspath(__file__)), "configs")


def config_names():
    return sorted(f[:-5] for f in os.listdir(_DIR) if f.startswith("c") and f.endswith(".json"))


def load_config(name_or_path):
    """Return the configuration dict; ``model`` may reference a shared model file."""
    path = name_or_path
    if not os.path.exists(path):
        path = os.path.join(_DIR, name_or_path + ".json")
    with open(path) as f:
        cfg = json.load(f)
    if isinstance(cfg.get("model"), str):
        with open(os.path.join(os.path.dirname(path), cfg["model"])) as f:
            cfg["model"] = json.load(f)
    return copy.deepcopy(cfg)


def seeds_of(cfg):
    s = cfg["seeds"]
    if isinstance(s, list):
        return [int(v) for v in s]
    return list(range(int(s["start"]), int(s["start"]) + int(s["count"])))
