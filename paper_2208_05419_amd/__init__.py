"""MI355X-native (gfx950) AFNO spectral token-mixing filter of FourCastNet.

The filter (forward real 2-D FFT of a [B,H,W,C] token grid, block-diagonal complex MLP
per Fourier mode, softshrink, hard mode cutoff, inverse real FFT, residual add) runs in
hand-written HIP kernels behind the C ABI of ``include/afno.h``; this package is its
Python binding.  Importing it loads nothing; the library is loaded on first use.
"""
from .afno import (AFNO_DTYPE_BF16, AFNO_DTYPE_FP32, AFNO_ERR_ALIAS, AFNO_ERR_HIP,  # noqa: F401
                   AFNO_ERR_INVALID_ARG, AFNO_ERR_UNSUPPORTED, AFNO_OK, AFNO_PATH_AUTO,
                   AFNO_PATH_GENERIC, AFNO_PATH_VALU_DFT, AFNO_STAGE_DELTA,
                   AFNO_STAGE_MIXED, AFNO_STAGE_SPECTRUM, EXPORTED, LIB_PATH, AfnoError,
                   BLOCK_PARAMS, KERNELS, afno_block_forward, afno_filter_backward, afno_filter_forward, afno_filter_forward_hidden,
                   afno_filter_forward_noalloc, filter_forward_noalloc,
                   afno_filter_stage, afno_filter_stage_hidden,
                   afno_last_error, afno_profile_begin, afno_profile_end, afno_set_kernel_path,
                   afno_version, block_forward, filter_backward, filter_forward, filter_stage,
                   load_library,
                   profile_begin, profile_end, set_kernel_path)
