"""Bounded state staging for the Training->Rollout role switch on MI355X (gfx950).

The compute path lives in the HIP/C++ library ``libdr.so`` (``csrc/``), whose
C ABI is declared in ``include/dr.h``; ``paper_2607_22614_amd.dr`` is its thin
ctypes binding.  Importing this package loads nothing: ``dr`` loads the library
on import and raises if it has not been built.
"""
