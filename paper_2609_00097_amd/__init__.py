"""Faster Flash Decoding (FFD) decode attention for AMD MI355X (gfx950).

The compute path is ``libffd.so`` (HIP kernels behind a C ABI, declared in ``include/ffd.h``);
``ffd`` is its ctypes binding.
"""
from .ffd import (BLOCK, HEAD_DIM, FfdError, FfdLibraryError, decode_attention,  # noqa: F401
                  dense_decode_attention, empty_quantized, lib, new_workspace, quantize_keys, quantized_shapes,
                  resolve_splits, workspace_bytes)
