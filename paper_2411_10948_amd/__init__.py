"""ShiftQuant backward path for MI355X (gfx950).

``shiftquant`` is the ctypes binding of the C-ABI library ``libshiftquant.so``
(hand-written HIP kernels); ``workloads`` draws the seeded synthetic inputs.
"""
