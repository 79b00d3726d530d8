"""Doubly-pipelined, dual-root reduction-to-all (Traeff 2021) on one MI355X.

The work happens in libdpar.so (include/dpar.h): host tree builder and round
schedule in C++, the round program in HIP kernels for gfx950.  ``dpar`` is a
thin ctypes binding with the same function names.
"""

from .dpar import (  # noqa: F401
    DparError, allreduce, dpar_allreduce, dpar_allreduce_ex,
    dpar_allreduce_opt, dpar_block_bounds, dpar_block_rule, dpar_check_status,
    dpar_finalize, dpar_last_error, dpar_rounds, dpar_schedule_info,
    dpar_schedule_rounds, dpar_set_phase_event, dpar_tree_info,
    dpar_tree_info_alg, lib, pointers, rows)
