"""Incremental ViT encoding with temporal token reuse on MI355X (gfx950).

``paper_2607_12287_amd.incvit`` binds the C ABI of ``libincvit.so`` (HIP
kernels); ``paper_2607_12287_amd.synth`` generates seeded inputs.  Nothing is
imported eagerly, so the input generator can be used without the library.
"""
