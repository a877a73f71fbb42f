"""MeqMuon hidden-weight update for AMD MI355X (gfx950).

The update itself lives in ``libmeq.so`` (HIP kernels behind the C ABI of
``include/meq.h``); :mod:`paper_2609_35701_amd.meq` is its ctypes binding.
"""
from .meq import (BUF_COL_RMS, BUF_NORMSQ, BUF_ROW_RMS, BUF_SCALE, BUF_U, BUF_X0, EXPORTED, KERNEL_NAMES,
                  MEQ_BF16, MEQ_DIR_COL, MEQ_DIR_ROW, MEQ_F32, HiddenWeightUpdate, HParams, MeqError,
                  MeqLibraryMissing, Plan, default_hparams, lib)

__all__ = ["BUF_COL_RMS", "BUF_NORMSQ", "BUF_ROW_RMS", "BUF_SCALE", "BUF_U", "BUF_X0", "EXPORTED", "KERNEL_NAMES",
           "MEQ_BF16", "MEQ_DIR_COL", "MEQ_DIR_ROW", "MEQ_F32", "HiddenWeightUpdate", "HParams", "MeqError",
           "MeqLibraryMissing", "Plan", "default_hparams", "lib"]
