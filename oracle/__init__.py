"""fp64 CPU oracles of the triangular multiplicative update (Fold-CP, Section 3.3),
the outer product mean (Section 3.5) and the triangle attention core
(Section 3.2).

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP library.  See oracle/trimul.py, oracle/opm.py and
oracle/triattn.py for the definitions they follow.
"""
from .trimul import (EPS, WEIGHT_NAMES, f64, layer_norm, sigmoid, pair_mask,  # noqa: F401
                     linear, project, contract_outgoing, contract_incoming,
                     epilogue, tri_mul, projected_panels, block_contract,
                     block_epilogue, take_pairs, layer_norm_backward,
                     contract_backward, tri_mul_backward)
from .opm import (msa_mask, pair_counts, outer_sum, outer_product_mean,  # noqa: F401
                  outer_product_mean_tile)
from .triattn import key_mask, scores, triangle_attention, chunked_attention  # noqa: F401
