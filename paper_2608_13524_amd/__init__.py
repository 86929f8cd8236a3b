"""DARTree fixed-width draft-tree construction on MI355X (gfx950).

The compute path is ``libdartree.so`` (hand-written HIP kernels behind a C ABI,
declared in ``include/dartree.h``); :mod:`.dartree` is its thin ctypes binding
and :mod:`.workloads` draws seeded synthetic inputs.
"""
