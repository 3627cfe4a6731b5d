"""MI355X-native BaKron solver (arXiv 2608.06291): Python binding of libbakron.so.

The solver itself is hand-written HIP for gfx950 behind a C ABI
(``include/bakron.h``); this package only marshals arguments.
"""
from ._lib import (BAKRON_EHIP, BAKRON_EINVAL, BAKRON_ENOMEM, BAKRON_ENOTSPD, BAKRON_OK,  # noqa: F401
                   BAKRON_KFAC, BAKRON_SHAMPOO,
                   EXPORTED, LIB_PATH, BakronError, Factors, factor, factor_blockdiag, gram,
                   gram_workspace_bytes, mse_scales,
                   kron_factors, load, mlp_local_factors, quadform_weights, sample_weights, solve,
                   solve_antidiag, solve_noalloc,
                   status_string)
