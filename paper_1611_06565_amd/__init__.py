"""N-dimensional Winograd correlation forward F(m^N, r^N) on AMD MI355X.

Budden et al., "Deep Tensor Convolution on Multicores" (arXiv 1611.06565),
rebuilt as hand-written HIP for gfx950 behind the C ABI in include/wino.h.
``wino`` is the Python binding (argument marshalling only; PyTorch supplies
device memory and streams).
"""
from .wino import (Plan, WinoError, describe_header_symbols, lib, library_path,  # noqa: F401
                   maxpool3d)
