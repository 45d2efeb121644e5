"""fp64 CPU oracle for the NOBLE-CosNet linear layer.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py``; never by the HIP product path.
Every function here is pinned by a ``-m "not gpu"`` test (closed forms,
hand-worked examples, finite differences, invariants); none is "parity
unpinned".
"""

from .noble_oracle import (  # noqa: F401
    ACTIVATIONS,
    LEAKY_SLOPE,
    activation_slope,
    activation_value,
    backward,
    backward_grouped,
    branch_backward,
    branch_forward,
    branch_param_shapes,
    cosnet_backward,
    cosnet_forward,
    forward,
    forward_grouped,
)
