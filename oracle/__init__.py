"""CPU oracle of the cache-hit block-sparse attention path.

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke check
of the package entry file and the CPU-baseline leg of the benchmark may
import or call anything in this package.  The HIP library never routes
through it, and it shares no code, tables or helpers with the HIP path.

Every function is plain fp64 NumPy, written from the paper's definitions:

* ``pool_blocks`` / ``block_scores`` / ``select_row`` / ``build_block_mask``:
  the historical block-connectivity mask (Appendix C.3, "Reuse-Scope
  Implementation Details": for each head and query block keep the smallest
  set of key blocks covering a fixed fraction of the attention mass), with the
  mass estimated from the softmax of block-pooled Q.K^T of the historical
  copy and ties within 1e-6 of score resolved towards the lower block index.
* ``merge_target_rows``: target-specific query blocks widened to full rows
  (Sec. 3.3, "Joint Reuse in Intermediate Layers": target-specific computation
  is preserved for the active region).
* ``compact_mask``: the per-row list of kept key blocks that the sparse
  executor walks.
* ``pack_mask`` / ``unpack_mask``: the masks as one bit per block pair, the
  form in which they are stored per step, branch and layer (Appendix C.3).
* ``dilate_frames`` / ``chebyshev_distance`` / ``regions`` / ``smoothstep`` /
  ``latent_fusion`` / ``region_block_flags`` / ``restrict_mask`` /
  ``compact_restricted``: the region-restricted middle-layer path (Sec. 3.3
  "Region-Guided Latent Reuse" and "Joint Reuse in Intermediate Layers";
  Appendix C.3 radii).
* ``exact_block_mass`` / ``select_row_mass`` / ``mask_from_mass``: the
  token-level attention mass of each block pair and the selection on it
  (Appendix C.3, "source attention mass" read literally).
* ``ciede2000`` / ``support_area`` / ``normalized_shape`` / ``d_size`` /
  ``d_shape`` / ``gate`` / ``first_compatible`` / ``clopper_pearson_upper``:
  the compatibility gate of a recalled cache (Sec. 3.2; Appendix F).
* ``block_sparse_attention``: softmax attention of the recomputed target
  Q, K, V restricted to the reused block structure (Sec. 3.3, "Historical
  Sparse-Connectivity Reuse"; Appendix C.3).
* ``cosine_similarity`` / ``topk_cosine``: cosine scoring of an early-step
  signature against a bank of cached signatures (Sec. 3.1 problem setup,
  Sec. 4.1 "Candidate Recall").

Readings taken where the paper is silent are listed in the module docstrings
of each submodule.
"""
from .mask import (pool_blocks, block_scores, select_row, build_block_mask,
                   merge_target_rows, compact_mask, group_rows_order, row_admissible_masks, TIE_EPS,
                   FRAGILE_EPS, pack_mask, unpack_mask)
from .attention import block_sparse_attention, token_mask_from_blocks
from .gate import (ciede2000, support_area, normalized_shape, d_size, d_shape, gate, first_compatible,
                   clopper_pearson_upper, SHAPE_RES)
from .exact_mass import exact_block_mass, select_row_mass, mask_from_mass, row_admissible_masks_mass
from .region import (dilate_frames, chebyshev_distance, smoothstep, regions, latent_fusion,
                     region_block_flags, restrict_mask, compact_restricted)
from .cosine import cosine_similarity, topk_cosine
from .convert import to_f64

__all__ = [
    "pool_blocks", "block_scores", "select_row", "build_block_mask",
    "merge_target_rows", "compact_mask", "group_rows_order", "row_admissible_masks", "TIE_EPS",
    "FRAGILE_EPS", "pack_mask", "unpack_mask", "block_sparse_attention", "token_mask_from_blocks",
    "cosine_similarity", "topk_cosine", "to_f64",
    "dilate_frames", "chebyshev_distance", "smoothstep", "regions", "latent_fusion",
    "region_block_flags", "restrict_mask", "compact_restricted",
    "exact_block_mass", "select_row_mass", "mask_from_mass", "row_admissible_masks_mass",
    "ciede2000", "support_area", "normalized_shape", "d_size", "d_shape", "gate", "first_compatible",
    "clopper_pearson_upper", "SHAPE_RES",
]
