"""The counter figures bench.py reports from its stored tables are the ones the rocprofv3
summaries in profiles/ state: for each summary, its kernel source id is a key of the
matching table, and the stored traffic and lane rate equal the summary's figures.

CPU only: reads text files and bench.py's tables, runs nothing on a device.
"""
import os
import re

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# summary file -> the workload string bench.py keys its k_fine tables by
FINE = {
    "k_fine_c4_seed.md": bench._W_C4_STEP,
    "k_fine_c1.md": bench._W_C1,
    "k_fine_c2_two_seeds.md": bench._W_C2_SEEDS2,
    "k_fine_c3_seed0.md": bench._W_C3_SEED0,
}


def _text(name):
    with open(os.path.join(ROOT, "profiles", name)) as f:
        return f.read()


def _sid(txt):
    m = re.search(r"Kernel source id `([0-9a-f]{16})`", txt)
    assert m, "no kernel source id"
    return m.group(1)


def _close(a, b, rel):
    return abs(a - b) <= rel * max(abs(a), abs(b))


@pytest.mark.parametrize("name", sorted(FINE))
def test_fine_tables_match_summaries(name):
    txt = _text(name)
    sid = _sid(txt)
    key = (sid, FINE[name])
    assert key in bench.MEASURED_TRAFFIC, f"{name}: source {sid} has no traffic entry"
    assert key in bench.MEASURED_LANE_FRAC, f"{name}: source {sid} has no lane-rate entry"
    total = float(re.search(r"\| total \| \| ([0-9.e+]+) =", txt).group(1))
    assert _close(bench.MEASURED_TRAFFIC[key], total, 1e-3), (bench.MEASURED_TRAFFIC[key], total)
    lane = float(re.search(r"Counter-measured VALU lane rate\*\*: [0-9.e+]+ lane-ops/s = \*\*([0-9.]+) %", txt).group(1))
    assert abs(bench.MEASURED_LANE_FRAC[key] - lane / 100.0) <= 6e-4, (bench.MEASURED_LANE_FRAC[key], lane)


def test_fine_tables_hold_one_source():
    """Every stored k_fine figure is of one kernel source, the one the summaries name."""
    sids = {k[0] for k in bench.MEASURED_TRAFFIC} | {k[0] for k in bench.MEASURED_LANE_FRAC}
    assert sids == {_sid(_text(n)) for n in FINE}


def test_phase2_table_matches_summary():
    txt = _text("k_mc_c4_phase2.md")
    keys = [k for k in bench.MC_MEASURED_TRAFFIC if k[0] == _sid(txt)]
    assert len(keys) == 1
    per_launch = float(re.search(r"\| HBM bytes per launch \| ([0-9.e+]+) ", txt).group(1))
    assert _close(bench.MC_MEASURED_TRAFFIC[keys[0]], per_launch, 1e-3)
    plans = int(re.search(r"the ([0-9,]+) plans phase 1 keeps", txt).group(1).replace(",", ""))
    assert f"the {plans} plans phase 1 keeps" in keys[0][1]


def test_enum_table_matches_summary():
    """The stored bytes per k_enum_unrank launch: the mean of the summary's per-dispatch
    WRITE_SIZE plus twice its FETCH_SIZE (the copy-probe scaling), in KiB."""
    txt = _text("k_enum_c2_space.md")
    key = (_sid(txt), 1 << 25)
    assert key in bench.ENUM_MEASURED_TRAFFIC
    row = lambda c: [float(x) for x in re.search(r"\| %s \(KiB\) \| ([0-9 /]+) \|" % c, txt).group(1).split("/")]
    w, f = row("WRITE_SIZE"), row("FETCH_SIZE")
    per_launch = (sum(w) / len(w) + 2.0 * sum(f) / len(f)) * 1024.0
    assert _close(bench.ENUM_MEASURED_TRAFFIC[key], per_launch, 1e-3), (bench.ENUM_MEASURED_TRAFFIC[key], per_launch)
