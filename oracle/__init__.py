"""fp64 CPU oracle of the SOLO shared-readout local loss (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline``
leg may import this package.  It shares no code with the GPU path.
"""
from .solo_oracle import (  # noqa: F401
    DEFAULT_EPS,
    module_fwd_bwd,
    readout_bruteforce,
    readout_fwd_bwd,
    rmsnorm_forward,
    softmax_rows,
)
from . import solo_oracle_general  # noqa: F401,E402
from .solo_oracle_general import exit_eval, general_bruteforce, general_fwd_bwd  # noqa: F401,E402
