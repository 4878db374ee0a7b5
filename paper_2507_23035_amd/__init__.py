"""OASIS hot path (outlier-aware LUT GEMM on codebook-quantized weights and
activations, arXiv 2507.23035) as a HIP library for MI355X (gfx950).

`oasis` is the ctypes binding of the C-ABI library `liboasis.so`; `synth`
generates seeded synthetic layers.
"""
