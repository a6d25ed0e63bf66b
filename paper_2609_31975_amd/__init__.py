"""MI355X-native activation-sparse FFN forward pass at decode.

Hand-written gfx950 HIP kernels behind a C ABI (``include/ffn_sparse.h``); the
Python side only marshals device pointers and streams (``paper_2609_31975_amd.ffn``).
``workloads`` holds the seeded synthetic inputs.
"""
