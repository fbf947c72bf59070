"""Seeded synthetic workloads shared by the tests, the bench and the oracle driver.

This package only draws random numbers: input spike trains, weights, delays and
labels with the shapes and statistics of the paper's benchmark tasks.  It holds
none of the method's arithmetic (no neuron dynamics, no loss, no gradients) and
imports neither the HIP library nor the oracle.
"""
from .configs import (CONFIGS, INPUT, LIF, LI, LOSS_CE_SUM, LOSS_CE_MAX, LOSS_DMSE, projections,
                      Config)
from .generators import (Workload, make_workload, make_variant, input_spikes,
                         weights_and_delays, labels)

__all__ = [
    "CONFIGS", "INPUT", "LIF", "LI", "LOSS_CE_SUM", "LOSS_CE_MAX", "LOSS_DMSE", "projections",
    "Config",
    "Workload", "make_workload", "make_variant", "input_spikes", "weights_and_delays", "labels",
]
