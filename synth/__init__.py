"""Seeded synthetic inputs shared by the oracle side (tests, CPU baseline) and the
library side (tests, benchmark).  Holds no arithmetic of the method itself: it only
draws random arrays with the shapes and statistics of the paper's workloads and rounds
them once to the storage dtype."""

from .workloads import (  # noqa: F401
    LM_HEADS, WORKLOADS, Case, Workload, make_case, make_lm_case, make_memory_case, make_output_grad,
    make_weights)
