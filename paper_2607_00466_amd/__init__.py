"""MI355X-native batched-decode MoE layer (the computation ELDR's routing speeds up).

The compute path is the C-ABI library ``libeldr_moe.so`` built from ``csrc/``
(hand-written HIP kernels for gfx950).  ``paper_2607_00466_amd.binding`` is a
thin ctypes layer over it; importing this package loads nothing.
"""
