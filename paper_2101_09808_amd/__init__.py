"""MI355X (gfx950) forward convolution, Eq. (1) of arXiv 2101.09808, with a
tile selector built on the paper's data-movement model.

The compute path is the HIP library ``libconvfwd.so`` (C ABI in
``include/conv_fwd.h``); ``conv`` is its Python binding.
"""
from .conv import (  # noqa: F401
    ConvError, ConvPlan, conv_fwd, conv_fwd_bf16, conv_fwd_candidates, conv_fwd_plan,
    conv_fwd_with_plan, conv_model_volume, strerror,
)
