"""FQT layer backward on MI355X (gfx950): PTQ / PSQ / BHQ gradient quantizers
with stochastic rounding and the two int8 MFMA contractions of a linear or
conv layer's backward (Chen et al. 2020, Sec. 2.2, Sec. 3.3, Sec. 4).

The compute path is the HIP library ``libfqt.so`` built from ``csrc/``;
``fqt`` is its ctypes binding.  Importing the package loads nothing.
"""
