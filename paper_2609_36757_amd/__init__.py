"""Chunk-wise causal attention for video latent tokens on MI355X (gfx950).

The compute lives in ``libfastvr.so`` (hand-written HIP kernels behind a C ABI,
declared in ``include/fastvr.h``).  ``paper_2609_36757_amd.fastvr`` is the thin
ctypes binding; importing this package does not load the library."""
