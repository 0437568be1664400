"""MI355X-native batched evaluation of exemplar-based clustering.

The compute lives in a C-ABI HIP library (``libexemcl.so``, declared in
``include/exemcl.h``); ``api`` is its thin Python binding and re-exports the
same names here.  Importing the package loads nothing: the library is opened
on first use, and every call fails loudly if it has not been built.
"""
from .api import (EXEMCL_BF16, EXEMCL_FP16, EXEMCL_FP32, ExemclError, exemplar_eval,  # noqa: F401
                  exemplar_gain, exemplar_greedy, exemplar_plan, exemplar_sqnorm, exemplar_version, strerror)
