"""CPU oracle for the TurboQuant search hot path -- TEST INFRASTRUCTURE ONLY.

This package is the plain, slow, obviously-correct reference that the GPU
library is checked against.  It is never part of the product path: only the
test-suite, the smoke check and the CPU-baseline leg of the benchmark may
import it.  It shares no code with the HIP library (no kernels, headers,
tables or helpers) and imports nothing from it.

Everything is float64 unless the method fixes another precision.  Each
function cites the passage of the TurboVec paper (arXiv 2607.16973) it
follows:

* marginal   -- the post-rotation coordinate law of section II-B (steps 2-3).
* codebook   -- analytic Lloyd-Max boundaries/centroids, section II-B step 3.
* rotation   -- the seeded random orthogonal matrix, section II-B step 2.
* encode     -- normalise / rotate / quantise / pack / length-renormalise,
                section II-B steps 1-5 (sequential float64 arithmetic in C);
                the optional TQ+ calibration of section II-B.
* search     -- query rotation, scoring, allowlist filter and top-k,
                sections II-B step 5 and III-B; exact ground truth and
                Recall@k as in section IV-A; Hit@k and MRR@20 as in
                section IV-E; the over-fetch post-filter baseline of
                section V-C.
"""
from .marginal import density, tail_prob, cell_mass, cell_first_moment, mse_per_coord
from .codebook import lloyd_max, Codebook
from .rotation import splitmix64, uniforms53, gaussians, haar_rotation
from .encode import (encode, quantise_rotated, pack_codes, unpack_codes, code_bytes_per_vector,
                     tqplus_fit, encode_tqplus)
from .search import (rotate_queries, scores_for_ids, score_all, topk_from_scores, search,
                     exact_search,
                     recall_at_k, hit_at_k, mrr_at_k, allowed_mask, postfilter_search)

__all__ = [
    "density", "tail_prob", "cell_mass", "cell_first_moment", "mse_per_coord",
    "lloyd_max", "Codebook",
    "splitmix64", "uniforms53", "gaussians", "haar_rotation",
    "encode", "quantise_rotated", "pack_codes", "unpack_codes", "code_bytes_per_vector", "tqplus_fit", "encode_tqplus",
    "rotate_queries", "scores_for_ids", "score_all", "topk_from_scores", "search", "exact_search",
    "recall_at_k", "hit_at_k", "mrr_at_k", "allowed_mask", "postfilter_search",
]
