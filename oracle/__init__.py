"""fp64 CPU oracle for FOVEA's per-draft-step visual-evidence retrieval and fusion.

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import or call anything in this
package.  The HIP library never calls it, and it imports nothing from the HIP side:
the two implementations share no code.  The seeded input generators (``synth``)
are the only thing both sides consume.

Everything here is written from the paper's Method section (memory construction,
state-conditioned retrieval with the cumulative-mass cardinality rule, gated hidden
correction) and its appendix paragraph on the visual correction module.  Arithmetic
is float64 NumPy throughout; the only non-fp64 step is the optional bf16 rounding of
a gain-folded projection weight, which mirrors a stated storage rounding of the
library (see ``fovea_ref.fold_gain``).

Parity status of each function is stated in ``fovea_ref``'s module docstring.
"""

from .fovea_ref import (  # noqa: F401
    bf16_round,
    build_memory,
    build_memory_backward,
    correction,
    fold_gain,
    fuse,
    layer_norm,
    lm_logits,
    lm_topk,
    lm_topk_from_logits,
    projected_layer_norm,
    query,
    readout,
    retrieve_fuse,
    retrieve_fuse_backward,
    rms_norm,
    scores,
    select_cumulative_mass,
    sigmoid,
    silu,
)
