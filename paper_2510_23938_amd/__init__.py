"""Device-resident model-integrity hashing for AMD MI355X (gfx950).

Chunked SHA-256 of weight bytes in HBM, RFC 6962 Merkle reduction to
per-tensor and manifest roots, and root verification -- all in HIP kernels
behind the C ABI of ``include/hv.h``.  ``paper_2510_23938_amd.hv`` is the
Python binding.
"""
