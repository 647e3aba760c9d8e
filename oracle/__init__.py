"""CPU reference ("oracle") for the PD scan -- TEST INFRASTRUCTURE ONLY.

The tests, the smoke check and the CPU-baseline leg of ``bench.py`` are the
only code allowed to import this package.  The GPU library never calls it and
shares no code with it.

``pdssm_oracle.c`` holds the arithmetic: a plain sequential float64 loop per
(batch, head) sequence, written from the paper's statement of the recurrence
(Flash PD-SSM, App. E.2 recurrence; Sec. 2.3/3.1 column-one-hot maps; Sec. 2.1
eq. (1) readout; App. E.3.1 composition rule; App. E.1 Algorithm 1 chunking;
Sec. 3.1 Prop. 2 straight-through surrogate gradients).
This module only marshals numpy arrays into it.
"""
from .oracle import (  # noqa: F401
    build_oracle,
    oracle_fwd,
    oracle_bwd,
    oracle_compose,
    oracle_ste,
    oracle_softmax_vjp,
    oracle_surrogate_grads,
    oracle_dict_argmax,
    oracle_route,
    oracle_project,
    oracle_num_chunks,
    oracle_lib_path,
)
