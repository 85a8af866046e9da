"""Sequentially-correct parallel SGD over sparse examples on one MI355X.

The HIP library ``libpdb.so`` (sources in ``csrc/``, C ABI in
``include/pdb.h``) does all the work; ``native`` is its ctypes binding.
"""
from . import native  # noqa: F401
