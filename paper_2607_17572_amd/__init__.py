"""MI355X-native JAGG group backward (Jacobian-Aggregated Group Gradient).

The compute path is the HIP library ``libjagg.so`` (C ABI in include/jagg.h);
this package is its thin Python binding (``api``) and its build script
(``build``).  Importing the package does not load the library; the first call
does, and raises if the library has not been built.
"""
from .api import (BF16, DGRAD, DGRAD_GELU, F32, WGRAD, PROF_AGGREGATE, PROF_ATTN_BWD_KV, PROF_ATTN_BWD_Q,  # noqa: F401
                  PROF_ATTN_FWD, PROF_COMPARE, PROF_UPSTREAM, PROF_GEMM_DGRAD, PROF_GEMM_FWD, PROF_GEMM_WGRAD, Config, Context,
                  JaggError, alpha, config, lib, param_layout, prof_begin, prof_end, route)
