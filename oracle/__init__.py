"""fp64 CPU oracle of the triangular multiplicative update (Fold-CP, Section 3.3).

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP library.  See oracle/trimul.py for the definition it follows.
"""
from .trimul import (EPS, WEIGHT_NAMES, f64, layer_norm, sigmoid, pair_mask,  # noqa: F401
                     linear, project, contract_outgoing, contract_incoming,
                     epilogue, tri_mul, projected_panels, block_contract,
                     block_epilogue, take_pairs, layer_norm_backward,
                     contract_backward, tri_mul_backward)
