"""Python binding of libda2: the C entry points under the same names.

Argument marshalling only: tensors are torch tensors on the GPU (device
memory and streams come from PyTorch); every step of the path runs in the
library's HIP kernels. Each call is enqueued on ``stream`` (default: torch's
current stream) and returns without synchronizing.
"""
import ctypes
from dataclasses import dataclass

import numpy as np
import torch

from . import _lib
from ._lib import (DA2_BF16, DA2_FMT4_MXFP4, DA2_FMT4_NVFP4, DA2_FP32, DA2_PART_RAGGED, DA2_PART_TILES8,
                   DA2_SCOPE_HEAD, DA2_SCOPE_ROW, Problem, Tensor, check, lib)

SCOPES = {"head": DA2_SCOPE_HEAD, "row": DA2_SCOPE_ROW}
PARTITIONS = {"tiles8": DA2_PART_TILES8, "ragged": DA2_PART_RAGGED}
FMT4 = {"nvfp4": DA2_FMT4_NVFP4, "mxfp4": DA2_FMT4_MXFP4}


def problem(B, H, d, T, Hg, Wg, partition="tiles8"):
    return Problem(B, H, d, T, Hg, Wg, PARTITIONS[partition])


def _tensor_desc(x):
    if x.dim() != 4 or x.stride(3) != 1:
        raise ValueError("expected a [B, H, N, d] tensor with d contiguous")
    dt = {torch.bfloat16: DA2_BF16, torch.float32: DA2_FP32}.get(x.dtype)
    if dt is None:
        raise ValueError(f"unsupported dtype {x.dtype}")
    return Tensor(x.stride(0), x.stride(1), x.stride(2), dt, 0)


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def da2_sizes(p, scope="head", fmt4="nvfp4", with16=False):
    s = _lib.Sizes()
    check("da2_sizes", lib().da2_sizes(ctypes.byref(p), SCOPES[scope], FMT4[fmt4], int(with16), ctypes.byref(s)))
    return {f: getattr(s, f) for f, _ in _lib.Sizes._fields_}


def da2_ops_layout_version():
    return lib().da2_ops_layout_version()


def da2_layout_build(p):
    """Host-side region layout (int32 numpy array: n_a, slot2tok, tok2slot)."""
    n = da2_sizes(p)["layout_bytes"] // 4
    out = np.empty(n, dtype=np.int32)
    check("da2_layout_build", lib().da2_layout_build(
        ctypes.byref(p), out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), n))
    return out


def _offsets(fn, p, n, *extra):
    arr = (ctypes.c_int64 * n)()
    check(fn, getattr(lib(), fn)(ctypes.byref(p), *extra, arr))
    return list(arr)


def da2_ws_draft_offsets(p):
    return _offsets("da2_ws_draft_offsets", p, 7)


def da2_lists_offsets(p):
    return _offsets("da2_lists_offsets", p, 4)


def da2_ops_offsets(p, fmt4="nvfp4", with16=False):
    """Byte offsets of the 16 ops sections for a run with (fmt4, with16); -1
    for a section such a run does not use."""
    return _offsets("da2_ops_offsets", p, 16, FMT4[fmt4], int(with16))


def da2_draft_map(Q, K, layout, p, lam, A, stats, ws, stream=None):
    check("da2_draft_map", lib().da2_draft_map(
        _ptr(Q), _ptr(K), ctypes.byref(_tensor_desc(Q)), _ptr(layout), ctypes.byref(p), float(lam),
        _ptr(A), _ptr(stats), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def da2_rank_assign(A, p, num16, num8, num4, den, scope, cls, lists, ws, stream=None):
    check("da2_rank_assign", lib().da2_rank_assign(
        _ptr(A), ctypes.byref(p), num16, num8, num4, den, SCOPES[scope], _ptr(cls), _ptr(lists), _ptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))


def da2_rank_assign_noalloc(A, p, num16, num8, num4, den, scope, cls, lists, stream=None):
    check("da2_rank_assign_noalloc", lib().da2_rank_assign_noalloc(
        _ptr(A), ctypes.byref(p), num16, num8, num4, den, SCOPES[scope], _ptr(cls), _ptr(lists), _stream(stream)))


def da2_prep_operands(Q, K, V, layout, p, with16, fmt4, stats, ops, ws, stream=None):
    if not (Q.shape == K.shape == V.shape and Q.stride() == K.stride() == V.stride() and Q.dtype == K.dtype == V.dtype):
        raise ValueError("Q, K and V must share shape, strides and dtype")
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    check("da2_prep_operands", lib().da2_prep_operands(
        _ptr(Q), _ptr(K), _ptr(V), ctypes.byref(_tensor_desc(Q)), _ptr(layout), ctypes.byref(p), int(with16),
        FMT4[fmt4], _ptr(stats), _ptr(ops), ops.numel() * ops.element_size(), None if ws is None else _ptr(ws),
        ws_bytes, _stream(stream)))


def da2_mixed_attn(ops, lists, layout, p, O, stream=None, fmt4="nvfp4"):
    check("da2_mixed_attn", lib().da2_mixed_attn(
        _ptr(ops), ops.numel() * ops.element_size(), _ptr(lists), _ptr(layout), ctypes.byref(p), FMT4[fmt4],
        ctypes.byref(_tensor_desc(O)), _ptr(O), _stream(stream)))


@dataclass
class Buffers:
    """Device buffers of one problem, sized by da2_sizes (allocation only).
    ``fmt4`` and ``with16`` are the 4-bit encoding and 16-bit option the ops
    buffer is sized for."""
    p: Problem
    scope: str
    fmt4: str
    with16: bool
    sizes: dict
    layout: torch.Tensor
    A: torch.Tensor
    cls: torch.Tensor
    stats: torch.Tensor
    lists: torch.Tensor
    ops: torch.Tensor
    ws_draft: torch.Tensor
    ws_rank: torch.Tensor


def alloc(p, scope="head", device="cuda", fmt4="nvfp4", with16=False):
    s = da2_sizes(p, scope, fmt4, with16)
    R = s["R"]
    B, H = p.B, p.H

    def raw(n):
        return torch.empty(max(int(n), 1), dtype=torch.uint8, device=device)

    layout = torch.from_numpy(da2_layout_build(p)).to(device)
    return Buffers(p, scope, fmt4, bool(with16), s, layout,
                   A=torch.empty((B, H, R, R), dtype=torch.float32, device=device),
                   cls=torch.empty((B, H, R, R), dtype=torch.uint8, device=device),
                   stats=raw(s["stats_bytes"]), lists=raw(s["lists_bytes"]), ops=raw(s["ops_bytes"]),
                   ws_draft=raw(s["ws_draft_bytes"]), ws_rank=raw(s["ws_rank_bytes"]))


def attention(Q, K, V, buf, lam, budgets, O, stream=None, num16=0, fmt4=None):
    """The four calls in order: draft map, ranking, operand preparation,
    attention. budgets = (num8, num4, den); num16/den go to the 16-bit path;
    fmt4 ("nvfp4" or "mxfp4", default: the buffers' encoding) is the encoding
    of the 4-bit path."""
    p = buf.p
    fmt4 = buf.fmt4 if fmt4 is None else fmt4
    if fmt4 != buf.fmt4 or (num16 > 0 and not buf.with16):
        raise ValueError(f"buffers sized for fmt4={buf.fmt4}, with16={buf.with16}; asked for fmt4={fmt4}, "
                         f"num16={num16}")
    da2_draft_map(Q, K, buf.layout, p, lam, buf.A, buf.stats, buf.ws_draft, stream)
    da2_rank_assign(buf.A, p, num16, *budgets, buf.scope, buf.cls, buf.lists, buf.ws_rank, stream)
    da2_prep_operands(Q, K, V, buf.layout, p, int(num16 > 0), fmt4, buf.stats, buf.ops, None, stream)
    da2_mixed_attn(buf.ops, buf.lists, buf.layout, p, O, stream, fmt4)
    return O
