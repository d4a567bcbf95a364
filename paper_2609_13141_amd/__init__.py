"""SAS (Simple Attention Sparsification) hot path for AMD MI355X (gfx950).

The compute path is a C-ABI shared library of hand-written HIP kernels
(``libsas.so``, built from ``csrc/``); ``sas`` is its thin ctypes binding.
Importing this package loads nothing: the library is opened on first use and
a missing library raises an error rather than falling back to anything else.
"""

__all__ = ["configs", "inputs", "sas"]
