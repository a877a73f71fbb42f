"""fp64 CPU oracle (test infrastructure only; never used by the product path)."""
from .meq_oracle import (COL, ROW, HParams, coeff_of_variation, col_normalize, equilibrate,
                         frobenius, meq_step, momentum, newton_schulz, ns_input, round_bf16,
                         row_col_rms, row_normalize, write_back)

__all__ = ["COL", "ROW", "HParams", "coeff_of_variation", "col_normalize", "equilibrate",
           "frobenius", "meq_step", "momentum", "newton_schulz", "ns_input", "round_bf16",
           "row_col_rms", "row_normalize", "write_back"]
