"""Block-routed MoE layer forward for AMD Instinct MI355X (gfx950).

The compute lives in ``libdmoe.so`` (hand-written HIP kernels behind the C ABI
of ``include/dmoe.h``); :mod:`.lib` is its ctypes binding and :mod:`.layer`
chains the entry points into one layer forward.
"""
__version__ = "0.1.0"
