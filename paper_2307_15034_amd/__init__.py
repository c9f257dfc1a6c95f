"""MI355X-native FNO spectral-convolution layer (fwd, bwd_data, bwd_weight).

The compute lives in the HIP library libfno_spectral_conv.so (csrc/), reached
through its C ABI (include/fno_spectral_conv.h) by the ctypes binding in
`binding` (importing it fails loudly when the library is missing);
`layer.SpectralConv` allocates device buffers with PyTorch.  The package
import itself loads nothing, so `python -m paper_2307_15034_amd.build` works
before the library exists.
"""
__all__ = ["binding", "layer", "build"]
