"""MI355X (gfx950) selective-differentiation layers: Conv2d, ConvTranspose2d,
Linear and BatchNorm in evaluation mode whose forward keeps the layer input only when
the weight gradient is requested and whose backward launches only the
requested gradient work (Sec. 2.2.1 of arXiv 2404.12406), and a ReLU that
keeps one bit per element instead of its output and a dropout that keeps its
generator state instead of its mask (Sec. 2.2.2).

The compute lives in libmemsave.so (hand-written HIP kernels, C ABI in
include/memsave.h); this package is its Python binding.  Build the library
with `python -m paper_2404_12406_amd.build`.
"""
from .api import (AvgPool, BatchNormEval, Conv2d, Conv3d, ConvTranspose2d, ConvTranspose3d, Dropout, Linear, MASK_BIAS, MASK_INPUT, MASK_WEIGHT,
                  POLICY_ALL_TRUE, POLICY_PYTORCH_DEFAULT, POLICY_SELECTIVE, PreparedLayer, Record, ReLU,
                  empty_like_layout, layer_backward, layer_forward, ledger_read, ledger_reset, output_shape,
                  policy_account, profile_read, profile_start, PROF_ACT, PROF_ALL, PROF_BN, PROF_DGRAD, PROF_FWD,
                  PROF_RED, PROF_WGRAD,
                  dropout_blocks, relu_mask_bytes, tensor_desc, version)
from ._lib import MemsaveError

__all__ = [
    "AvgPool", "BatchNormEval", "Conv2d", "Conv3d", "ConvTranspose2d", "ConvTranspose3d", "Dropout", "Linear", "MASK_BIAS", "MASK_INPUT", "MASK_WEIGHT",
    "POLICY_ALL_TRUE", "POLICY_PYTORCH_DEFAULT", "POLICY_SELECTIVE", "PreparedLayer", "Record", "ReLU",
    "MemsaveError", "PROF_ACT", "PROF_ALL", "PROF_RED", "relu_mask_bytes", "dropout_blocks",
    "empty_like_layout", "layer_backward", "layer_forward", "ledger_read", "ledger_reset",
    "output_shape", "policy_account", "profile_read", "profile_start", "PROF_BN", "PROF_DGRAD", "PROF_FWD",
    "PROF_WGRAD", "tensor_desc", "version",
]
