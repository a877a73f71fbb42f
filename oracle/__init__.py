"""fp64 CPU oracle (test infrastructure only; never used by the product path)."""
from .meq_oracle import (COL, ROW, HParams, aux_step, coeff_of_variation, col_normalize, equilibrate,
                         frobenius, global_rms_normalize, meq_step, momentum, moonlight_step,
                         newton_schulz, ns_cv_trace, ns_input, round_bf16, row_col_rms, row_normalize, two_sided,
                         vec_step, write_back)

__all__ = ["COL", "ROW", "HParams", "aux_step", "coeff_of_variation", "col_normalize", "equilibrate",
           "frobenius", "global_rms_normalize", "meq_step", "momentum", "moonlight_step",
           "newton_schulz", "ns_cv_trace", "ns_input", "round_bf16", "row_col_rms", "row_normalize", "two_sided",
           "vec_step", "write_back"]
