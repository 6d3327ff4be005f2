"""ctypes loader for libda2.so and the C structures of include/da2.h.

The library must have been built (``python -m paper_2609_32628_amd.build``);
loading fails loudly otherwise: there is no fallback implementation.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libda2.so")

DA2_OK, DA2_ERR_INVALID_ARG, DA2_ERR_UNSUPPORTED, DA2_ERR_WORKSPACE, DA2_ERR_HIP = 0, -1, -2, -3, -4
DA2_BF16, DA2_FP32 = 0, 1
DA2_SCOPE_HEAD, DA2_SCOPE_ROW = 0, 1
DA2_PART_TILES8, DA2_PART_RAGGED = 0, 1
DA2_FMT4_NVFP4, DA2_FMT4_MXFP4 = 0, 1
DA2_RANK_NOALLOC_MAX_BYTES = 8 << 20   # include/da2.h
DA2_OPS_LAYOUT_VERSION = 2
DA2_ATTN_ERR_LAYOUT, DA2_ATTN_ERR_FMT4, DA2_ATTN_ERR_NO16 = 1, 2, 4
TAG_MARKER = 0xDA200000   # encoding tag in word 3 of each head's g entry

# Every symbol include/da2.h declares.
EXPORTS = ("da2_status_string", "da2_sizes", "da2_ops_layout_version", "da2_layout_build", "da2_draft_map", "da2_ws_draft_offsets",
           "da2_rank_assign", "da2_rank_assign_noalloc", "da2_lists_offsets", "da2_prep_operands", "da2_ops_offsets", "da2_mixed_attn")


class Problem(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("H", ctypes.c_int32), ("d", ctypes.c_int32),
                ("T", ctypes.c_int32), ("Hg", ctypes.c_int32), ("Wg", ctypes.c_int32),
                ("partition", ctypes.c_int32)]


class Tensor(ctypes.Structure):
    _fields_ = [("stride_b", ctypes.c_int64), ("stride_h", ctypes.c_int64), ("stride_n", ctypes.c_int64),
                ("dtype", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class Sizes(ctypes.Structure):
    _fields_ = [("R", ctypes.c_int32), ("Npad", ctypes.c_int32),
                ("layout_bytes", ctypes.c_int64), ("A_bytes", ctypes.c_int64), ("cls_bytes", ctypes.c_int64),
                ("stats_bytes", ctypes.c_int64), ("lists_bytes", ctypes.c_int64), ("ops_bytes", ctypes.c_int64),
                ("ws_draft_bytes", ctypes.c_int64), ("ws_rank_bytes", ctypes.c_int64),
                ("ws_prep_bytes", ctypes.c_int64)]


class Da2Error(RuntimeError):
    def __init__(self, call, status, lib):
        msg = lib.da2_status_string(status).decode()
        super().__init__(f"{call} failed: {msg} ({status})")
        self.status = status


_LIB = None


def lib():
    """The loaded library (raises if libda2.so has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_32628_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, dbl = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        P, T, S = ctypes.POINTER(Problem), ctypes.POINTER(Tensor), ctypes.POINTER(Sizes)
        pi64, pi32 = ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int32)
        sig = {
            "da2_status_string": (ctypes.c_char_p, [i32]),
            "da2_sizes": (i32, [P, i32, i32, i32, S]),
            "da2_ops_layout_version": (i32, []),
            "da2_layout_build": (i32, [P, pi32, i64]),
            "da2_draft_map": (i32, [vp, vp, T, vp, P, dbl, vp, vp, vp, i64, vp]),
            "da2_ws_draft_offsets": (i32, [P, pi64]),
            "da2_rank_assign": (i32, [vp, P, i32, i32, i32, i32, i32, vp, vp, vp, i64, vp]),
            "da2_rank_assign_noalloc": (i32, [vp, P, i32, i32, i32, i32, i32, vp, vp, vp]),
            "da2_lists_offsets": (i32, [P, pi64]),
            "da2_prep_operands": (i32, [vp, vp, vp, T, vp, P, i32, i32, vp, vp, i64, vp, i64, vp]),
            "da2_ops_offsets": (i32, [P, i32, i32, pi64]),
            "da2_mixed_attn": (i32, [vp, i64, vp, vp, P, i32, T, vp, vp]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype, f.argtypes = res, args
        _LIB = L
    return _LIB


def check(call, status):
    if status != DA2_OK:
        raise Da2Error(call, status, lib())
