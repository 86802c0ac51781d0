"""Seeded synthetic inputs shared by the oracle-side tests and the GPU-side tests/bench.

This package only draws random numbers and names workload shapes. It holds none of the
learner's arithmetic (no network, no targets, no loss, no optimiser), so that the oracle
and the HIP path stay independent while reading identical input bytes.
"""
from .gen import (NetShape, Workload, WORKLOADS, param_shapes, param_count, draw_params,
                  draw_rollout, draw_actor_batch, workload)

__all__ = ["NetShape", "Workload", "WORKLOADS", "param_shapes", "param_count", "draw_params",
           "draw_rollout", "draw_actor_batch", "workload"]
