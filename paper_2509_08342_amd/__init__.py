"""libmoesplit: per-layer MoE forward over split experts on one MI355X.

The compute path is the HIP library ``libmoesplit.so`` (C ABI in
include/moesplit.h); ``paper_2509_08342_amd.moesplit`` is its ctypes binding
and ``paper_2509_08342_amd.build`` compiles it.  Importing this package loads
nothing.
"""
