"""Seeded synthetic inputs for the memory-based TGNN batch step.

This package is the only code shared by the GPU product path and the CPU
oracle.  It draws inputs (event streams, masks, negatives, parameters, start
states, loss-gradient noise) and holds none of the method's arithmetic:
no message construction, aggregation, GRU, sampling or attention lives here.
"""

from .configs import WORKLOADS, Workload, workload  # noqa: F401
from .streams import (  # noqa: F401
    Stream,
    make_stream,
    init_params,
    init_params_jodie,
    window_state,
    loss_noise,
    batch_slice,
    node_owner,
)
