"""miconv: MI355X-native (gfx950) convolution hot path of CNN inference.

Dense conv2d (implicit GEMM on MFMA, fp32 and bf16-in/fp32-accumulate),
depthwise conv2d and the glue operators of the evaluated networks, behind a
C-ABI shared library (``include/miconv.h``).  ``miconv`` is the thin Python
binding over that library; ``workloads`` holds the seeded synthetic inputs
and the layer tables.
"""
__all__ = ["miconv", "workloads"]
