"""Seeded synthetic workloads shaped like the autotuning spaces of BaCO's evaluation.

This package only draws inputs (raw parameter columns, objective values, feasibility
labels, masks and hyperparameters). It contains none of the GP arithmetic: the HIP
library and the CPU oracle both consume the arrays it produces, and nothing else is
shared between them.
"""
from .synth import (Param, Workload, make_workload, WORKLOADS, uniform_columns,
                    cot_example_space, cot_example_constraints, hyper_starts,
                    c3_chain_leaves, c3_known_feasible)

__all__ = ["Param", "Workload", "make_workload", "WORKLOADS", "uniform_columns",
           "cot_example_space", "cot_example_constraints", "hyper_starts",
           "c3_chain_leaves", "c3_known_feasible"]
