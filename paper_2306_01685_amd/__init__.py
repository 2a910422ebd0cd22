"""MI355X-native (gfx950) hot path of MKOR (arXiv 2306.01685).

The kernels and the C ABI live in libmkor.so (sources in csrc/, header in
include/mkor.h); this package is the ctypes binding around it.
"""
from .binding import (  # noqa: F401
    MkorPlan, MkorError, Params, load_library, read_stats, params_check, workspace_size_raw,
    status_string, last_error, mkor_layer_stats, STATS_BYTES, EXPORTED, LIB_PATH,
    SM_EXACT, SM_PAPER_EQ6, NORM_INF, NORM_MAXABS, DTYPE_F32, DTYPE_BF16, MAX_DIM, MAX_ROWS,
    STAGE_NAMES, NUM_STAGES, Hybrid, step_noalloc, MAX_RANK, OptParams, opt_params_check, OPT_SGD, OPT_LAMB,
    GEMM_AUTO, GEMM_FP32, GEMM_SPLIT,
    MKOR_OK, MKOR_INVALID_ARG, MKOR_WORKSPACE_TOO_SMALL, MKOR_UNSUPPORTED, MKOR_HIP_ERROR,
)
