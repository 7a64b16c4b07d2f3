"""Seeded synthetic inputs for the DQGAN compression step: the workload table
(parameter-vector shapes shaped like the GANs the paper trains), segment
layouts, gradient and parameter draws.

This module holds no arithmetic of the method itself.  Both the GPU path's
tests/benchmark and the oracle's tests draw their inputs from it.
"""
from .configs import CONFIGS, Workload, get  # noqa: F401
from .gen import gradients, gradients_np, init_params, init_params_np  # noqa: F401
