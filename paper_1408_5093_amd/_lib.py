"""ctypes loader for ``libcaffe_conv.so`` and the C structs of its ABI.

The library is never built or replaced on the fly by this module: build it
with ``paper_1408_5093_amd.build`` (or ``__graft_entry__.build()``) first.
If it is missing, every call raises -- there is no fallback path.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcaffe_conv.so")

CAFFE_OK = 0
CAFFE_ERR_INVALID_ARG = -1
CAFFE_ERR_ALIGN = -2
CAFFE_ERR_WORKSPACE = -3
CAFFE_ERR_UNSUPPORTED = -4
CAFFE_ERR_HIP = -5

CAFFE_F32 = 0
CAFFE_BF16 = 1
CAFFE_BF16_F32_BOTTOM = 2

BACKWARD_TOP_DIFF_MASKED = 1
BACKWARD_MASK_BOTTOM_DIFF = 2
BACKWARD_BOTTOM_STAGED = 4
BACKWARD_TOP_STAGED = 16
BACKWARD_POOL_MASK_OFFSETS = 32
FORWARD_BOTTOM_STAGED = 1
POOL_RELU_INPUT = 1
POOL_LRN_STAGE_ONLY = 2
POOL_MASK_OFFSETS = 4

PASS_FORWARD = 0
PASS_BACKWARD_DATA = 1
PASS_BACKWARD_WEIGHTS = 2
PASS_BACKWARD = 3
PASS_BACKWARD_POOL_LRN = 4

NOALLOC_SCRATCH_BYTES = 64 << 20  # CAFFE_CONV_NOALLOC_SCRATCH_BYTES

CAFFE_LR_FIXED = 0
CAFFE_LR_STEP = 1
CAFFE_LR_EXP = 2
CAFFE_LR_INV = 3

# every symbol the public headers declare
EXPORTS = (
    "caffe_conv_out_shape", "caffe_conv_workspace_size", "caffe_conv_forward",
    "caffe_conv_backward_data", "caffe_conv_backward_weights", "caffe_conv_backward",
    "caffe_status_string", "caffe_last_error", "caffe_version",
    "caffe_pool_out_shape", "caffe_maxpool_forward", "caffe_maxpool_backward",
    "caffe_lrn_forward", "caffe_lrn_backward", "caffe_cast_f32_to_bf16",
    "caffe_sgd_learning_rate", "caffe_softmax_loss", "caffe_sgd_update",
    "caffe_pool_lrn_forward", "caffe_lrn_pool_backward", "caffe_sgd_update_device_lr",
    "caffe_conv_workspace_bytes", "caffe_conv_status_string", "caffe_conv_forward_noalloc",
    "caffe_conv_backward_pool_lrn", "caffe_relu_backward", "caffe_conv_backward_ex",
    "caffe_conv_backward_pool_lrn_ex", "caffe_conv_backward_into",
    "caffe_conv_stage_below_supported", "caffe_conv_forward_ex", "caffe_pool_lrn_forward_into",
    "caffe_pool_lrn_stage_supported", "caffe_lrn_pool_backward_ex",
)


class ConvDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "N", "C", "H", "W", "K", "kernel_h", "kernel_w", "stride_h", "stride_w",
        "pad_h", "pad_w", "group", "relu", "dtype")]


class PoolDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "N", "C", "H", "W", "kernel_h", "kernel_w", "stride_h", "stride_w", "pad_h", "pad_w")]


class LrnDesc(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int32), ("C", ctypes.c_int32), ("H", ctypes.c_int32),
                ("W", ctypes.c_int32), ("local_size", ctypes.c_int32),
                ("alpha", ctypes.c_float), ("beta", ctypes.c_float), ("k", ctypes.c_float)]


class LrSchedule(ctypes.Structure):
    _fields_ = [("policy", ctypes.c_int32), ("base_lr", ctypes.c_float),
                ("gamma", ctypes.c_float), ("power", ctypes.c_float),
                ("stepsize", ctypes.c_int32)]


class CaffeError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{message} ({status})")
        self.status = status


_lib = None


def load():
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with `python -m paper_1408_5093_amd.build`")
    try:  # the library shares PyTorch's HIP runtime; load torch's first when present
        import torch  # noqa: F401
    except Exception:
        pass
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    cdp, pdp, ldp = ctypes.POINTER(ConvDesc), ctypes.POINTER(PoolDesc), ctypes.POINTER(LrnDesc)
    pi32 = ctypes.POINTER(i32)
    sig = {
        "caffe_conv_out_shape": [cdp, pi32, pi32],
        "caffe_conv_workspace_size": [cdp, i32, ctypes.POINTER(sz)],
        "caffe_conv_forward": [cdp, vp, vp, vp, vp, vp, sz, vp],
        "caffe_conv_forward_ex": [cdp, vp, vp, vp, vp, vp, sz, i32, vp],
        "caffe_conv_forward_noalloc": [cdp, vp, vp, vp, vp, vp],
        "caffe_conv_backward_data": [cdp, vp, vp, vp, vp, vp, sz, vp],
        "caffe_conv_backward_weights": [cdp, vp, vp, vp, vp, vp, i32, vp, sz, vp],
        "caffe_conv_backward": [cdp, vp, vp, vp, vp, vp, vp, vp, i32, i32, vp, sz, vp],
        "caffe_conv_backward_ex": [cdp, vp, vp, vp, vp, vp, vp, vp, i32, i32, vp, sz, vp, vp],
        "caffe_conv_backward_into": [cdp, vp, vp, vp, vp, vp, vp, i32, i32, vp, sz, cdp, vp, sz,
                                     vp, vp],
        "caffe_conv_stage_below_supported": [cdp, cdp],
        "caffe_pool_out_shape": [pdp, pi32, pi32],
        "caffe_maxpool_forward": [pdp, vp, vp, vp, i32, vp],
        "caffe_maxpool_backward": [pdp, vp, vp, vp, vp],
        "caffe_lrn_forward": [ldp, vp, vp, vp],
        "caffe_lrn_backward": [ldp, vp, vp, vp, vp, vp],
        "caffe_cast_f32_to_bf16": [vp, vp, i64, vp],
        "caffe_relu_backward": [vp, vp, vp, i64, vp],
        "caffe_pool_lrn_forward": [pdp, ldp, vp, vp, vp, vp, i32, vp],
        "caffe_pool_lrn_forward_into": [pdp, ldp, vp, vp, vp, vp, i32, cdp, vp, sz, vp],
        "caffe_pool_lrn_stage_supported": [pdp, ldp, cdp],
        "caffe_lrn_pool_backward_ex": [pdp, ldp, vp, vp, vp, vp, vp, i32, vp],
        "caffe_lrn_pool_backward": [pdp, ldp, vp, vp, vp, vp, vp, vp],
        "caffe_conv_backward_pool_lrn": [cdp, pdp, ldp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                         i32, i32, vp, sz, vp],
        "caffe_conv_backward_pool_lrn_ex": [cdp, pdp, ldp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                            vp, i32, i32, vp, sz, vp, vp],
        "caffe_sgd_learning_rate": [ctypes.POINTER(LrSchedule), i64,
                                    ctypes.POINTER(ctypes.c_float)],
        "caffe_softmax_loss": [vp, vp, i32, i32, ctypes.c_float, vp, vp, vp, vp, vp],
        "caffe_sgd_update": [vp, vp, vp, i64, ctypes.c_float, ctypes.c_float, ctypes.c_float,
                             vp],
        "caffe_sgd_update_device_lr": [vp, vp, vp, i64, vp, ctypes.c_float, ctypes.c_float, vp],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    for name in ("caffe_status_string", "caffe_conv_status_string"):
        getattr(lib, name).argtypes = [i32]
        getattr(lib, name).restype = ctypes.c_char_p
    lib.caffe_conv_workspace_bytes.argtypes = [cdp, i32]
    lib.caffe_conv_workspace_bytes.restype = sz
    lib.caffe_last_error.argtypes = []
    lib.caffe_last_error.restype = ctypes.c_char_p
    lib.caffe_version.argtypes = []
    lib.caffe_version.restype = i32
    _lib = lib
    return lib


def check(status):
    if status != CAFFE_OK:
        lib = load()
        raise CaffeError(lib.caffe_status_string(status).decode(),
                         lib.caffe_last_error().decode())
    return status
