"""ctypes declarations of libtfk.so (include/tfk.h).  Marshalling only."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtfk.so")

TFK_OK = 0
STATUS_NAMES = {0: "TFK_OK", 1: "TFK_ERR_NULL", 2: "TFK_ERR_SHAPE", 3: "TFK_ERR_DTYPE", 4: "TFK_ERR_ALIGN",
                5: "TFK_ERR_OVERFLOW", 6: "TFK_ERR_ALIAS", 7: "TFK_ERR_WORKSPACE", 8: "TFK_ERR_HIP",
                9: "TFK_ERR_ARG"}
TFK_F32 = 0
TFK_BF16 = 1

# every symbol include/tfk.h declares
EXPORTS = ["tfk_conv2d_fwd", "tfk_conv2d_fwd_bias_relu", "tfk_maxpool_bwd_relu_bwd", "tfk_conv2d_bwd_input",
           "tfk_conv2d_bwd_input_relu_bwd", "tfk_conv2d_bwd_filter", "tfk_conv2d_bwd_filter_noalloc",
           "tfk_conv2d_fwd_bias_relu_maxpool",
           "tfk_conv2d_workspace_bytes",
           "tfk_bias_relu_fwd", "tfk_bias_relu_bwd", "tfk_bias_relu_bwd_workspace_bytes",
           "tfk_last_bias_partials", "tfk_bias_grad_finish",
           "tfk_maxpool_fwd", "tfk_maxpool_bwd", "tfk_maxpool_fwd_taps", "tfk_maxpool_bwd_taps",
           "tfk_maxpool_bwd_relu_bwd_taps", "tfk_apply_sgd", "tfk_apply_sgd_multi",
           "tfk_apply_momentum", "tfk_apply_adam", "tfk_softmax_xent", "tfk_gather_rows_t",
           "tfk_sampled_softmax_xent", "tfk_scatter_apply_sgd", "tfk_stream_wait", "tfk_mark_create", "tfk_mark_destroy",
           "tfk_mark_record", "tfk_stream_wait_mark", "tfk_program_create",
           "tfk_program_destroy", "tfk_program_begin", "tfk_program_end", "tfk_program_length", "tfk_program_run",
           "tfk_status_string", "tfk_last_error", "tfk_abi_version"]


class Nhwc(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("h", ctypes.c_int32), ("w", ctypes.c_int32), ("c", ctypes.c_int32),
                ("pixel_stride", ctypes.c_int64)]


class Window(ctypes.Structure):
    _fields_ = [("kh", ctypes.c_int32), ("kw", ctypes.c_int32), ("stride_h", ctypes.c_int32),
                ("stride_w", ctypes.c_int32), ("pad_top", ctypes.c_int32), ("pad_bottom", ctypes.c_int32),
                ("pad_left", ctypes.c_int32), ("pad_right", ctypes.c_int32)]


class TfkError(RuntimeError):
    def __init__(self, status, message):
        self.status = status
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, status), message))


_lib = None


def load(path: str = LIB_PATH):
    """Loads the HIP library; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("libtfk.so is not built (%s): run `python -m paper_1605_08695_amd.build`" % path)
    lib = ctypes.CDLL(path)
    vp, i32, i64, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
    st = ctypes.c_int
    lib.tfk_conv2d_fwd.argtypes = [vp, Nhwc, vp, i32, Window, st, vp, Nhwc, vp, sz, vp]
    lib.tfk_conv2d_fwd_bias_relu.argtypes = [vp, Nhwc, vp, i32, vp, Window, st, vp, Nhwc, vp, sz, vp]
    lib.tfk_conv2d_fwd_bias_relu_maxpool.argtypes = [vp, Nhwc, vp, i32, vp, Window, st, vp, Nhwc, Window, vp, Nhwc,
                                                     vp, vp, sz, vp]
    lib.tfk_conv2d_bwd_input.argtypes = [vp, Nhwc, vp, Window, st, vp, Nhwc, f32, vp, sz, vp]
    lib.tfk_conv2d_bwd_filter.argtypes = [vp, Nhwc, vp, Nhwc, Window, st, vp, vp, sz, vp]
    lib.tfk_conv2d_bwd_filter_noalloc.argtypes = [vp, Nhwc, vp, Nhwc, Window, st, vp, vp]
    lib.tfk_conv2d_bwd_input_relu_bwd.argtypes = [vp, Nhwc, vp, Window, st, vp, vp, Nhwc, f32, vp, vp, sz, vp]
    lib.tfk_conv2d_workspace_bytes.argtypes = [i32, Nhwc, i32, Window, st]
    lib.tfk_conv2d_workspace_bytes.restype = sz
    lib.tfk_bias_relu_fwd.argtypes = [vp, Nhwc, vp, st, vp]
    lib.tfk_bias_relu_bwd.argtypes = [vp, vp, Nhwc, vp, vp, st, vp, sz, vp]
    lib.tfk_bias_relu_bwd_workspace_bytes.argtypes = [Nhwc, st]
    lib.tfk_bias_relu_bwd_workspace_bytes.restype = sz
    lib.tfk_maxpool_fwd.argtypes = [vp, Nhwc, Window, st, vp, Nhwc, vp, vp]
    lib.tfk_maxpool_bwd.argtypes = [vp, vp, Nhwc, Window, st, vp, Nhwc, f32, vp]
    lib.tfk_maxpool_bwd_relu_bwd.argtypes = [vp, vp, Nhwc, Window, st, vp, vp, i64, vp, Nhwc, f32, vp, vp, sz, vp]
    lib.tfk_maxpool_fwd_taps.argtypes = lib.tfk_maxpool_fwd.argtypes
    lib.tfk_maxpool_bwd_taps.argtypes = lib.tfk_maxpool_bwd.argtypes
    lib.tfk_maxpool_bwd_relu_bwd_taps.argtypes = lib.tfk_maxpool_bwd_relu_bwd.argtypes
    lib.tfk_apply_sgd.argtypes = [vp, vp, i64, f32, vp, vp]
    lib.tfk_apply_sgd_multi.argtypes = [i32, ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(i64), f32,
                                        ctypes.POINTER(vp), vp]
    lib.tfk_apply_momentum.argtypes = [vp, vp, vp, i64, f32, f32, i32, vp, vp]
    lib.tfk_apply_adam.argtypes = [vp, vp, vp, vp, i64, f32, f32, f32, f32, i64, vp, vp]
    lib.tfk_softmax_xent.argtypes = [vp, st, i64, i32, vp, vp, f32, vp, vp, vp]
    lib.tfk_gather_rows_t.argtypes = [vp, st, i64, i32, vp, i32, i32, vp, vp]
    lib.tfk_sampled_softmax_xent.argtypes = [vp, st, i64, i32, i32, i32, vp, vp, vp, vp, f32, vp, vp, vp]
    lib.tfk_scatter_apply_sgd.argtypes = [vp, vp, i64, i32, vp, i32, vp, i64, f32, vp]
    for name in ("tfk_conv2d_fwd", "tfk_conv2d_fwd_bias_relu", "tfk_conv2d_fwd_bias_relu_maxpool", "tfk_conv2d_bwd_input", "tfk_conv2d_bwd_input_relu_bwd",
                 "tfk_conv2d_bwd_filter", "tfk_conv2d_bwd_filter_noalloc", "tfk_bias_relu_fwd",
                 "tfk_bias_relu_bwd", "tfk_maxpool_fwd", "tfk_maxpool_bwd", "tfk_maxpool_bwd_relu_bwd",
                 "tfk_maxpool_fwd_taps", "tfk_maxpool_bwd_taps", "tfk_maxpool_bwd_relu_bwd_taps", "tfk_apply_sgd",
                 "tfk_apply_sgd_multi", "tfk_apply_momentum", "tfk_apply_adam", "tfk_softmax_xent", "tfk_gather_rows_t",
                 "tfk_sampled_softmax_xent", "tfk_scatter_apply_sgd"):
        getattr(lib, name).restype = st
    lib.tfk_last_bias_partials.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(i32)]
    lib.tfk_bias_grad_finish.argtypes = [i32, ctypes.POINTER(vp), ctypes.POINTER(i32), ctypes.POINTER(i32),
                                         ctypes.POINTER(vp), vp]
    for name in ("tfk_last_bias_partials", "tfk_bias_grad_finish"):
        getattr(lib, name).restype = st
    lib.tfk_stream_wait.argtypes = [vp, vp]
    lib.tfk_mark_create.argtypes = [ctypes.POINTER(vp)]
    lib.tfk_mark_destroy.argtypes = [vp]
    lib.tfk_mark_destroy.restype = None
    lib.tfk_mark_record.argtypes = [vp, vp]
    lib.tfk_stream_wait_mark.argtypes = [vp, vp]
    for name in ("tfk_mark_create", "tfk_mark_record", "tfk_stream_wait_mark"):
        getattr(lib, name).restype = st
    lib.tfk_program_create.argtypes = [ctypes.POINTER(vp)]
    lib.tfk_program_destroy.argtypes = [vp]
    lib.tfk_program_destroy.restype = None
    for name in ("tfk_program_begin", "tfk_program_end", "tfk_program_run"):
        getattr(lib, name).argtypes = [vp]
    lib.tfk_program_length.argtypes = [vp]
    lib.tfk_program_length.restype = i64
    for name in ("tfk_stream_wait", "tfk_program_create", "tfk_program_begin", "tfk_program_end", "tfk_program_run"):
        getattr(lib, name).restype = st
    lib.tfk_status_string.argtypes = [st]
    lib.tfk_status_string.restype = ctypes.c_char_p
    lib.tfk_last_error.argtypes = []
    lib.tfk_last_error.restype = ctypes.c_char_p
    lib.tfk_abi_version.argtypes = []
    lib.tfk_abi_version.restype = i32
    _lib = lib
    return lib


def check(status: int):
    if status != TFK_OK:
        msg = _lib.tfk_last_error().decode()
        raise TfkError(status, msg)
