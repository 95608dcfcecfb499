"""MI355X-native dense matrix-vector kernels in minimal executable programs.

The package holds the HIP kernels and C-ABI library (``csrc/``, built into
``libmep.so``), the seeded input generator (``datagen``) and the Python
binding (``mep``).  Importing the package itself loads nothing: import
``paper_2512_22147_amd.mep`` for the binding, which loads the HIP library on
first use and raises if it is missing.
"""
