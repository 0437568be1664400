"""MI355X-native batched evaluation of exemplar-based clustering.

The compute lives in a C-ABI HIP library (``libexemcl.so``); this package is
its thin Python binding.  Importing it loads nothing: the library is opened on
first use, and every call fails loudly if it is missing.
"""
