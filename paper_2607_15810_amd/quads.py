"""ctypes binding of libquads.so (declared in include/quads.h).

Argument marshalling only: every step of the layer runs in the library's HIP
kernels.  The library is loaded on first use; if it has not been built the
binding raises instead of falling back to anything else.
"""

import ctypes
import os
from ctypes import POINTER, c_char_p, c_float, c_int, c_int32, c_int64, c_size_t, c_void_p

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libquads.so")

QD_OK = 0
QD_ERR_NULL = -1
QD_ERR_SHAPE = -2
QD_ERR_ALIGN = -3
QD_ERR_DTYPE = -4
QD_ERR_WORKSPACE = -5
QD_ERR_UNSUPPORTED = -6
QD_ERR_HIP = -7

QD_DTYPE_BF16 = 0
QD_DTYPE_F32 = 1
QD_EPI_NONE = 0
QD_EPI_SWIGLU = 1

STAGE_NAMES = ["route", "quant_x", "select", "w13", "quant_h", "w2", "combine"]

VIEW_NAMES = ["topk_ids", "topk_w", "offsets", "row_token", "inv_row", "xq_codes",
              "xq_scales", "xq_gscale", "scores", "ramax", "sel", "rq_codes", "rq_scales",
              "rq_gscale", "h", "h_amax", "hq_codes", "hq_scales", "hq_gscale", "z", "rq_sel",
              "h_scores", "h_ramax", "sel2", "hr_codes", "hr_scales", "hr_gscale", "hr_sel"]


class NVFP4(ctypes.Structure):
    """qd_nvfp4: device pointers, the shape, the optional fragment-ordered scales."""
    _fields_ = [("codes", c_void_p), ("scales", c_void_p), ("gscale", c_void_p),
                ("groups", c_int64), ("rows", c_int64), ("cols", c_int64),
                ("scales_frag", c_void_p)]


PN = POINTER(NVFP4)

# name -> (restype, argtypes)
SIGNATURES = {
    "qd_status_string": (c_char_p, [c_int]),
    "qd_version": (c_int, []),
    "nvfp4_quantize_act_workspace": (c_size_t, [c_int64, c_int64]),
    "nvfp4_quantize_act": (c_int, [c_void_p, c_int, c_int64, c_int64, c_void_p, c_int64, PN,
                                   c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    "nvfp4_quantize_weight_workspace": (c_size_t, [c_int64, c_int64, c_int64]),
    "nvfp4_quantize_weight": (c_int, [c_void_p, c_int64, c_int64, c_int64, PN, c_void_p,
                                      c_size_t, c_void_p]),
    "nvfp4_dequantize": (c_int, [PN, c_int, c_void_p, c_int, c_void_p]),
    "moe_route_permute_workspace": (c_size_t, [c_int64, c_int32, c_int32]),
    "moe_route_permute": (c_int, [c_void_p, c_int64, c_int32, c_int32, c_int32, c_void_p,
                                  c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t,
                                  c_void_p]),
    "rac_select_channels_workspace": (c_size_t, [c_int64, c_int64]),
    "rac_select_channels": (c_int, [c_void_p, PN, c_int32, c_void_p, c_void_p, c_int32,
                                    c_void_p, PN, c_void_p, c_size_t, c_void_p]),
    "rac_select_channels_per_expert_workspace": (c_size_t, [c_int64, c_int64, c_int32]),
    "rac_select_channels_per_expert": (c_int, [c_void_p, PN, c_int32, c_void_p, c_void_p,
                                               c_int32, c_int64, c_void_p, c_void_p, c_void_p,
                                               PN, c_void_p, c_void_p, c_size_t, c_void_p]),
    "rac_selected_width": (c_int32, [c_int32]),
    "rac_gather_selected": (c_int, [PN, c_void_p, c_int32, c_void_p, c_void_p]),
    "rac_residual_gemm": (c_int, [PN, c_void_p, c_int32, c_void_p, c_void_p, c_int64, PN,
                                  c_void_p, c_void_p]),
    "moe_w4a4_grouped_gemm_amax_count": (c_int64, [c_int64, c_int64, c_int64, c_int32, c_int32,
                                                   c_int32]),
    "moe_w4a4_grouped_gemm_residual_form": (c_int32, [c_int64, c_int64, c_int64, c_int32,
                                                      c_int32, c_int32]),
    "nvfp4_frag_scales_bytes": (c_int64, [c_int64, c_int64, c_int64]),
    "nvfp4_pack_frag_scales": (c_int, [PN, c_void_p, c_void_p]),
    "moe_w4a4_grouped_gemm": (c_int, [PN, c_void_p, c_void_p, c_int32, c_int64, PN, PN,
                                      c_void_p, c_int32, c_void_p, c_int32, c_void_p, c_void_p,
                                      c_void_p]),
    "moe_w4a4_grouped_gemm_per_expert_amax_count": (c_int64, [c_int64, c_int64, c_int64,
                                                              c_int32, c_int32, c_int32]),
    "moe_w4a4_grouped_gemm_per_expert": (c_int, [PN, c_void_p, c_void_p, c_int32, c_int64, PN,
                                                 PN, c_void_p, c_int32, c_void_p, c_int32,
                                                 c_void_p, c_void_p, c_void_p]),
    "moe_unpermute_combine": (c_int, [c_void_p, c_void_p, c_void_p, c_int64, c_int32, c_int64,
                                      c_void_p, c_void_p]),
    "fp8_quantize_rows": (c_int, [c_void_p, c_int32, c_int64, c_int64, c_void_p, c_void_p,
                                  c_void_p]),
    "moe_fp8_grouped_gemm": (c_int, [c_void_p, c_void_p, c_int64, c_void_p, c_void_p, c_int32,
                                     c_int64, c_void_p, c_void_p, c_int64, c_int64, c_int32,
                                     c_void_p, c_void_p]),
    "qd_fp8_moe_layer_workspace": (c_size_t, [c_int64, c_int64, c_int32, c_int32, c_int64]),
    "qd_fp8_moe_layer_forward": (c_int, [c_void_p, c_void_p, c_int64, c_int64, c_int32, c_int32,
                                         c_int64, c_int32, c_void_p, c_void_p, c_void_p,
                                         c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    "mxfp4_quantize_rows": (c_int, [c_void_p, c_int32, c_int64, c_int64, c_void_p, c_void_p,
                                    c_void_p]),
    "moe_mxfp4_grouped_gemm": (c_int, [c_void_p, c_void_p, c_int64, c_void_p, c_void_p, c_int32,
                                       c_int64, c_void_p, c_void_p, c_int64, c_int64, c_int32,
                                       c_void_p, c_void_p]),
    "qd_mxfp4_moe_layer_workspace": (c_size_t, [c_int64, c_int64, c_int32, c_int32, c_int64]),
    "qd_mxfp4_moe_layer_forward": (c_int, [c_void_p, c_void_p, c_int64, c_int64, c_int32,
                                           c_int32, c_int64, c_int32, c_void_p, c_void_p,
                                           c_void_p, c_void_p, c_void_p, c_void_p, c_size_t,
                                           c_void_p]),
    "moe_w4a16_grouped_gemm": (c_int, [c_void_p, c_int64, c_void_p, c_void_p, c_int32, c_int64,
                                       PN, c_int32, c_void_p, c_void_p]),
    "qd_moe_layer_workspace": (c_size_t, [c_int64, c_int64, c_int32, c_int32, c_int64]),
    "qd_moe_layer_forward": (c_int, [c_void_p, c_void_p, c_int64, c_int64, c_int32, c_int32,
                                     c_int64, c_int32, c_int32, c_int32, PN, PN, c_void_p,
                                     c_void_p, c_size_t, c_void_p]),
    "qd_moe_layer_forward_timed": (c_int, [c_void_p, c_void_p, c_int64, c_int64, c_int32,
                                           c_int32, c_int64, c_int32, c_int32, c_int32, PN, PN,
                                           c_void_p, c_void_p, c_size_t, c_void_p, c_void_p]),
    "qd_moe_layer_views": (c_int, [c_int64, c_int64, c_int32, c_int32, c_int64,
                                   POINTER(c_int64)]),
    "qd_moe_block_workspace": (c_size_t, [c_int64, c_int64, c_int32, c_int32, c_int64]),
    "qd_moe_block_views": (c_int, [c_int64, c_int64, c_int32, c_int32, c_int64,
                                   POINTER(c_int64)]),
    "qd_moe_block_forward": (c_int, [c_void_p, c_void_p, ctypes.c_float, c_void_p, c_int64,
                                     c_int64, c_int32, c_int32, c_int64, c_int32, c_int32,
                                     c_int32, PN, PN, c_void_p, c_void_p, c_size_t, c_void_p]),
    "qd_moe_block_forward_timed": (c_int, [c_void_p, c_void_p, ctypes.c_float, c_void_p,
                                           c_int64, c_int64, c_int32, c_int32, c_int64, c_int32,
                                           c_int32, c_int32, PN, PN, c_void_p, c_void_p,
                                           c_size_t, c_void_p, c_void_p]),
    "qd_moe_layer_per_expert_workspace": (c_size_t, [c_int64, c_int64, c_int32, c_int32,
                                                     c_int64, c_int32]),
    "qd_moe_layer_forward_per_expert": (c_int, [c_void_p, c_void_p, c_int64, c_int64, c_int32,
                                                c_int32, c_int64, c_int32, c_int32, PN, PN,
                                                c_void_p, c_void_p, c_size_t, c_void_p]),
    "qd_probe_hbm_read_out_count": (c_int64, []),
    "qd_probe_hbm_read": (c_int, [c_void_p, c_int64, c_void_p, c_void_p]),
    "qd_probe_mfma_f16_flops": (ctypes.c_double, [c_int64, c_int32]),
    "qd_probe_mfma_f16": (c_int, [c_int64, c_int32, c_int32, c_void_p, c_void_p]),
    "qd_moe_layer_noalloc_max_bytes": (c_size_t, []),
    "qd_moe_layer_forward_noalloc": (c_int, [c_void_p, c_void_p, c_int64, c_int64, c_int32,
                                             c_int32, c_int64, c_int32, c_int32, c_int32, PN, PN,
                                             c_void_p, c_void_p]),
}

_lib = None


class QuadsError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__(f"{fn} failed: {status_string(status)} (status {status})")


def lib():
    """The loaded library (raises if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2607_15810_amd.build`;"
                " the layer has no other implementation")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def status_string(st):
    return lib().qd_status_string(st).decode()


def call(name, *args):
    """Call an entry point and raise QuadsError on a non-zero status."""
    st = getattr(lib(), name)(*args)
    if st != QD_OK:
        raise QuadsError(name, st)
    return st


def raw(name, *args):
    """Call an entry point and return its status (tests of the error paths)."""
    return getattr(lib(), name)(*args)
