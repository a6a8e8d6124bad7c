"""COLD pre-ranking scoring path for AMD Instinct MI355X (gfx950).

The scoring work runs in hand-written HIP kernels behind the C-ABI library
``libcold.so`` (declared in ``include/cold.h``); :mod:`.binding` is a thin
ctypes layer over it.  :mod:`.synth` draws seeded synthetic inputs.
Importing this package loads nothing; the library is opened on first use.
"""
