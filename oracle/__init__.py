"""fp64 CPU oracle of the Periodic Row-wise Muon optimizer step.

Test infrastructure only: importable from ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py``; never from the product package.
"""
from .prm_oracle import *  # noqa: F401,F403
from .prm_oracle import (NS_COEFFS, NS_ITERS, AdamWConfig, PRMConfig, adamw_step,  # noqa: F401
                         adamw_bytes_per_element, direction, momentum_update,
                         momentum_direction_input, ns5, ns5_closed_form, ns5_flops,
                         ns5_rows_closed_form, orient, orient_inv, phi5, polar, quintic,
                         refresh_indicator, rownorm, shape_scale, step, step_matrix)
