"""ctypes view of include/memsave.h.  Loads the in-tree libmemsave.so and
raises if it is not built: there is no other implementation to fall back to."""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libmemsave.so")

MS_OK, MS_E_NULL, MS_E_MASK, MS_E_SHAPE, MS_E_DTYPE, MS_E_LAYOUT = 0, 1, 2, 3, 4, 5
MS_E_UNSUPPORTED, MS_E_CONSUMED, MS_E_NOMEM, MS_E_HIP, MS_E_ARG = 6, 7, 8, 9, 10
MS_RG_INPUT, MS_RG_WEIGHT, MS_RG_BIAS = 1, 2, 4
MS_F32, MS_BF16 = 0, 1
MS_CONV2D, MS_LINEAR, MS_BN_EVAL, MS_AVGPOOL, MS_RELU, MS_CONV_TRANSPOSE2D, MS_DROPOUT = 0, 1, 2, 3, 4, 5, 6
MS_CONV3D, MS_CONV_TRANSPOSE3D = 7, 8
MS_SAVED_X, MS_SAVED_W, MS_SAVED_MEAN, MS_SAVED_VAR, MS_SAVED_BITS, MS_SAVED_Y, MS_SAVED_MASK8 = 1, 2, 4, 8, 16, 32, 64
MS_K_DGRAD, MS_K_WGRAD, MS_K_BGRAD = 1, 2, 4
MS_POLICY_SELECTIVE, MS_POLICY_PYTORCH_DEFAULT, MS_POLICY_ALL_TRUE = 0, 1, 2

# Every function the two public headers declare, with its ctypes signature.
EXPORTS = (
    "ms_layer_forward", "ms_layer_backward", "ms_record_account", "ms_record_free",
    "ms_ledger_read", "ms_ledger_reset", "ms_policy_account", "ms_status_str",
    "ms_last_error", "ms_version", "ms_testing_fail_next_workspace", "ms_testing_live_records",
    "ms_profile_start", "ms_profile_read", "ms_relu_mask_bytes", "ms_relu_forward",
    "ms_dropout_blocks", "ms_dropout_forward", "ms_layer_backward_noalloc", "ms_noalloc_scratch_bytes",
    "ms_testing_gemm_plan",
)
MS_PROF_FWD, MS_PROF_DGRAD, MS_PROF_WGRAD, MS_PROF_BN, MS_PROF_ACT, MS_PROF_RED = 1, 2, 4, 8, 16, 32


class MsTensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * 5), ("stride", ctypes.c_int64 * 5)]


class MsLayer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("stride", ctypes.c_int32 * 2), ("pad", ctypes.c_int32 * 2),
                ("eps", ctypes.c_float), ("running_mean", ctypes.POINTER(MsTensor)),
                ("running_var", ctypes.POINTER(MsTensor)), ("out_pad", ctypes.c_int32 * 2),
                ("stride_d", ctypes.c_int32), ("pad_d", ctypes.c_int32), ("out_pad_d", ctypes.c_int32)]


class MsAccount(ctypes.Structure):
    _fields_ = [("saved_activation_bytes", ctypes.c_uint64), ("referenced_param_bytes", ctypes.c_uint64),
                ("transient_workspace_bytes", ctypes.c_uint64), ("mask", ctypes.c_uint32),
                ("borrowed", ctypes.c_uint32), ("kernels", ctypes.c_uint32), ("reserved", ctypes.c_uint32)]

    def as_dict(self):
        return {f[0]: int(getattr(self, f[0])) for f in self._fields_ if f[0] != "reserved"}


_T = ctypes.POINTER(MsTensor)
_lib = None


class MemsaveError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str = ""):
        self.status = status
        super().__init__(f"{where}: {status_str(status)} ({status}){': ' + detail if detail else ''}")


def configure(lib: ctypes.CDLL) -> ctypes.CDLL:
    """Declare the C signatures of include/memsave.h on a loaded library."""
    lib.ms_layer_forward.argtypes = [ctypes.POINTER(MsLayer), _T, _T, _T, ctypes.c_uint32, _T,
                                     ctypes.POINTER(ctypes.c_void_p), ctypes.c_void_p]
    lib.ms_layer_forward.restype = ctypes.c_int
    lib.ms_layer_backward.argtypes = [ctypes.c_void_p, _T, _T, _T, _T, ctypes.c_void_p]
    lib.ms_layer_backward.restype = ctypes.c_int
    lib.ms_layer_backward_noalloc.argtypes = [ctypes.c_void_p, _T, _T, _T, _T, ctypes.c_void_p]
    lib.ms_layer_backward_noalloc.restype = ctypes.c_int
    lib.ms_noalloc_scratch_bytes.argtypes = []
    lib.ms_noalloc_scratch_bytes.restype = ctypes.c_uint64
    lib.ms_record_account.argtypes = [ctypes.c_void_p, ctypes.POINTER(MsAccount)]
    lib.ms_record_account.restype = ctypes.c_int
    lib.ms_record_free.argtypes = [ctypes.c_void_p]
    lib.ms_record_free.restype = None
    lib.ms_ledger_read.argtypes = [ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_uint64)]
    lib.ms_ledger_read.restype = ctypes.c_int
    lib.ms_ledger_reset.argtypes = []
    lib.ms_ledger_reset.restype = ctypes.c_int
    lib.ms_policy_account.argtypes = [ctypes.POINTER(MsLayer), _T, _T, _T, ctypes.c_uint32, ctypes.c_int32,
                                      ctypes.POINTER(MsAccount)]
    lib.ms_policy_account.restype = ctypes.c_int
    lib.ms_status_str.argtypes = [ctypes.c_int32]
    lib.ms_status_str.restype = ctypes.c_char_p
    lib.ms_last_error.argtypes = []
    lib.ms_last_error.restype = ctypes.c_char_p
    lib.ms_version.argtypes = []
    lib.ms_version.restype = ctypes.c_char_p
    lib.ms_testing_fail_next_workspace.argtypes = [ctypes.c_int32]
    lib.ms_testing_fail_next_workspace.restype = None
    lib.ms_testing_live_records.argtypes = []
    lib.ms_testing_live_records.restype = ctypes.c_int64
    lib.ms_testing_gemm_plan.argtypes = [ctypes.c_int32, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32)]
    lib.ms_testing_gemm_plan.restype = ctypes.c_int32
    lib.ms_profile_start.argtypes = [ctypes.c_uint32]
    lib.ms_profile_start.restype = ctypes.c_int
    lib.ms_profile_read.argtypes = [ctypes.c_uint32, ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_double)]
    lib.ms_profile_read.restype = ctypes.c_int
    lib.ms_relu_mask_bytes.argtypes = [ctypes.c_int64]
    lib.ms_relu_mask_bytes.restype = ctypes.c_uint64
    lib.ms_relu_forward.argtypes = [_T, _T, ctypes.c_void_p, ctypes.c_uint32, ctypes.POINTER(ctypes.c_void_p),
                                    ctypes.c_void_p]
    lib.ms_relu_forward.restype = ctypes.c_int
    lib.ms_dropout_blocks.argtypes = [ctypes.c_int64]
    lib.ms_dropout_blocks.restype = ctypes.c_uint64
    lib.ms_dropout_forward.argtypes = [_T, _T, ctypes.c_float, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint32,
                                       ctypes.POINTER(ctypes.c_void_p), ctypes.c_void_p]
    lib.ms_dropout_forward.restype = ctypes.c_int
    return lib


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -m paper_2404_12406_amd.build` "
                           "(the HIP library is the only implementation)")
    lib = configure(ctypes.CDLL(path))
    _lib = lib
    return lib


def status_str(status: int) -> str:
    return load().ms_status_str(int(status)).decode()


def check(status: int, where: str):
    if status != MS_OK:
        detail = load().ms_last_error().decode()
        raise MemsaveError(status, where, detail)
