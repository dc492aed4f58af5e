"""Seeded synthetic inputs shared by the HIP path, the oracle and the tests.

This module holds no arithmetic of the evaluation method.  It only

* loads the workload configurations (model graph, latency-model
  coefficients, request-type mix, length distributions, latency targets,
  GPU budget, rate grid, seeds, trace length) from ``configs/*.json``;
* generates physical-plan tables (Sec. 4.2 of the paper: nodes that host one
  or more components, executors per node, per-node batch configuration,
  per-type routing probabilities in steps of 0.1 over at most two parallel
  paths), laid out as a structure of arrays, field-slot major.

Requests themselves are not generated here: drawing the trace is a step of
the evaluated path (``cf_trace_gen``) and each side does its own.
"""
from .configs_io import load_config, config_names, seeds_of  # noqa: F401
from .plans import PlanTable, make_plans, plan_table_from_list  # noqa: F401
