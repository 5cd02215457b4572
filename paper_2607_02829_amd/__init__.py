"""MI355X-native hot path of Sparse-Reslim (dense -> sparse -> dense token routing).

The package holds:

* ``csrc/``   - HIP kernels for gfx950 and the C-ABI entry points (``libsr.so``);
* ``abi``     - a thin ctypes binding with the same names as the C entry points;
* ``inputs``  - seeded synthetic inputs (token fields, weights, gradients) shaped
  like the paper's workloads;
* ``build``   - the in-tree build of ``libsr.so``.

Importing the package loads nothing; ``abi.lib()`` loads the shared library and
raises if it has not been built.
"""
