"""MI355X (gfx950) random-Fourier-feature linear attention (Flexformer, arXiv 2606.27748).

The computation lives in the HIP library ``libflexattn.so`` (C ABI in
include/flex.h); this package is its thin Python binding.
"""
from ._lib import (FlexError, flex_desc, make_desc, workspace_size, flex_feature_map,  # noqa: F401
                   flex_linattn_fwd, flex_linattn_prefill, flex_linattn_fwd_noalloc, flex_linattn_bwd, flex_decode_step,
                   flex_awd_loss, decode_state,
                   decode_state_views, load, status_string,
                   FLEX_OK, FLEX_ERR_INVALID_ARG, FLEX_ERR_UNSUPPORTED, FLEX_ERR_WORKSPACE,
                   FLEX_ERR_HIP, FLEX_PASS_FEATURE_MAP, FLEX_PASS_FWD, FLEX_PASS_BWD, FLEX_PASS_AWD,
                   EXPORTS,
                   KERNELS, flex_timing_enable, flex_timing_read)
