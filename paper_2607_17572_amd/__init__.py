"""MI355X-native JAGG group backward (Jacobian-Aggregated Group Gradient).

The compute path is the HIP library ``libjagg.so`` (C ABI in include/jagg.h);
this package is its thin Python binding (``api``) and its build script
(``build``).  Importing the package does not load the library; the first call
does, and raises if the library has not been built.
"""
from .api import (BF16, F32, Config, Context, JaggError, alpha, config, lib,  # noqa: F401
                  param_layout, route)
