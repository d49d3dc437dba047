"""HeadCast routed attention for MI355X (gfx950).

The compute path is the HIP library ``libheadcast.so`` behind the C ABI in
``include/headcast.h``; ``paper_2607_20125_amd.headcast`` is its ctypes binding.
"""
