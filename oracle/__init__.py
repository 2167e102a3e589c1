"""OrbitQuant CPU oracle — TEST INFRASTRUCTURE ONLY.

A plain, slow, fp64 numpy/scipy implementation of the quantized linear layer of
OrbitQuant (arXiv 2607.02461), written from the paper's definitions:

  marginal.py  rotated-coordinate marginal f_d            Sec. 3.2, Eq. (2)
  lloydmax.py  Lloyd-Max codebook on f_d                   Sec. 3.2 / Sec. 4.5, Eq. (3)
  plan.py      RPBH plan (permutation + Rademacher signs)  Sec. 4.4, Eq. (9)
  rpbh.py      RPBH forward / inverse transform           Sec. 4.4, Eq. (9); Suppl. A setup
  quantize.py  normalize + nearest-centroid encode + pack Eqs. (5)-(8), Alg. 1
  qlinear.py   contraction of the two code sets           Sec. 4.3 (rotation cancellation)
  adaln_rtn.py INT4 RTN g64 weight-only AdaLN projection  Sec. 5 setup; Suppl. layer list; Sec. 6.2

Only the tests, the package's smoke check and the benchmark's CPU-baseline leg
may import this package.  The product path (the HIP library and its binding)
never imports, links or executes anything here, and this package imports
nothing from the product path: the two share no code.  The only module both
sides read is the seeded input generator, which holds none of the method's
arithmetic.

Every function cites the passage of the paper it follows.  Where the paper is
silent the reading taken is stated at the function.
"""

from .marginal import marginal_pdf, marginal_cdf, marginal_mass, marginal_partial_moment, log_norm_const
from .lloydmax import lloydmax_codebook, Codebook
from .plan import SplitMix64, rpbh_plan, Plan
from .rpbh import rpbh_forward, rpbh_inverse, sylvester_hadamard, fwht_blocks
from .quantize import (normalize_rows, encode, decode_levels, pack_codes, unpack_codes,
                       quantize_act, quantize_weights, near_tie_mask, nearest_threshold, bf16_round, bf16_bits,
                       fp16_round, to_labels, from_labels)
from .qlinear import layer_epilogue, qlinear, qlinear_dense_reference
from .adaln_rtn import rtn_int4_quantize, rtn_int4_dequantize, pack_rtn_int4, unpack_rtn_int4, rtn_int4_linear

EPS_DEFAULT = 1e-10  # Sec. 4.3: the clamp guarding zero-norm (padding) tokens

__all__ = [
    "marginal_pdf", "marginal_cdf", "marginal_mass", "layer_epilogue", "marginal_partial_moment", "log_norm_const",
    "lloydmax_codebook", "Codebook", "SplitMix64", "rpbh_plan", "Plan",
    "rpbh_forward", "rpbh_inverse", "sylvester_hadamard", "fwht_blocks",
    "normalize_rows", "encode", "decode_levels", "pack_codes", "unpack_codes",
    "quantize_act", "quantize_weights", "near_tie_mask", "nearest_threshold", "bf16_round", "bf16_bits", "fp16_round", "to_labels", "from_labels",
    "qlinear", "qlinear_dense_reference", "EPS_DEFAULT",
    "rtn_int4_quantize", "rtn_int4_dequantize", "pack_rtn_int4", "unpack_rtn_int4", "rtn_int4_linear",
]
