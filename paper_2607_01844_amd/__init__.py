"""MI355X-native MoE expert layer (routing, permutation, grouped SwiGLU GEMMs,
combine; forward and backward) from the Mixture-of-Parallelisms training
stack.  The compute lives in libmoe.so (hand-written HIP for gfx950); the
binding in `paper_2607_01844_amd.moe` only marshals arguments.  Submodules
are imported explicitly (`from paper_2607_01844_amd import moe`), so that
building the library never requires it to be present.
"""
