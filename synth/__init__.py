"""Seeded synthetic workloads for the ChebBooster online stage.

This module holds the workload definitions (cache shapes, history abscissae,
target abscissae) and the seeded feature generators.  It contains none of the
method's arithmetic: no weights, no combination of history entries.  Both the
oracle side (tests, CPU baseline) and the HIP side (tests, benchmark, smoke
check) draw their inputs from here.
"""
from .configs import CONFIGS, Config, by_name
from .generate import make_history, make_history_f64, split_segments

__all__ = ["CONFIGS", "Config", "by_name", "make_history", "make_history_f64",
           "split_segments"]
