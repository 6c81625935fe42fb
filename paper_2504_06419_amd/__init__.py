"""Speculative-round attention for MI355X (gfx950).

The product is the C-ABI library libspire.so (include/spire.h) built from the
HIP sources in csrc/; `spire` is its thin Python binding and `workloads` the
seeded synthetic input generator.  Importing the package loads nothing: the
library is loaded on first use and a missing build raises an error.
"""
