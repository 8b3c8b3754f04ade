"""Sampling-based mini-batch GNN training on AMD Instinct MI355X (gfx950).

The training path lives in libgnnhip.so (HIP kernels behind the C ABI of
include/gnnhip.h); `gnnhip` is its ctypes binding.
"""
from . import gnnhip  # noqa: F401
from .gnnhip import (Csr, Trainer, alloc_blocks, block_caps, check_errors,  # noqa: F401
                     gather_features, layer_bwd, layer_fwd, lib, sample_blocks, sgd,
                     softmax_xent)
