"""Host-only checks of the C ABI (no GPU needed): the library loads, exports
every entry point include/da2.h declares, sizes / offsets / layout are
consistent, and every argument error is reported before the GPU is touched."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

from oracle import partition
from paper_2609_32628_amd import _lib, api
from synth import configs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "da2.h")


def _declared():
    text = open(HEADER).read()
    return set(re.findall(r"^\s*(?:const char\*|int32_t)\s+(da2_\w+)\s*\(", text, flags=re.M))


def test_header_and_exports_agree():
    declared = _declared()
    assert declared == set(_lib.EXPORTS)
    out = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (da2_\w+)$", out, flags=re.M))
    assert declared <= exported
    L = _lib.lib()
    for name in declared:
        assert getattr(L, name) is not None


def test_status_strings():
    L = _lib.lib()
    for s in (0, -1, -2, -3, -4, 7):
        assert isinstance(L.da2_status_string(s), bytes)
    assert b"INVALID_ARG" in L.da2_status_string(-1)


def _p(w):
    return api.problem(w.B, w.H, w.d, w.T, w.Hg, w.Wg)


def test_sizes_mid_layer():
    s = api.da2_sizes(_p(configs.MID), "head")
    assert s["R"] == 588 and s["Npad"] == 37632
    assert s["A_bytes"] == 4 * 12 * 588 * 588
    assert s["cls_bytes"] == 12 * 588 * 588
    assert s["layout_bytes"] == 4 * (588 + 37632 + 32760)
    off = api.da2_ops_offsets(_p(configs.MID))
    assert off == sorted(off) and all(o % 256 == 0 for o in off)
    e = 12 * 37632 * 128
    assert off[1] - off[0] >= 2 * e and off[4] - off[3] >= e
    mx = 12 * 588 * 5 * 1024   # MXFP4 sections: d/32 + 1 fragments of 1 KB per block
    assert off[13] - off[12] >= 2 * e and off[14] - off[13] >= mx and off[15] - off[14] >= mx
    assert s["ops_bytes"] >= off[15] + mx and len(off) == 16
    lo = api.da2_lists_offsets(_p(configs.MID))
    assert lo[1] >= 2 * 12 * 588 * 588 and lo[2] - lo[1] >= 16 * 12 * 588 and s["lists_bytes"] >= lo[3] + 32
    wo = api.da2_ws_draft_offsets(_p(configs.MID))
    assert wo[6] >= wo[5] + 8 * 12 * 588 * 588 and len(wo) == 7
    assert s["ws_draft_bytes"] >= wo[6] + 2 * 4 * 12 * 588


@pytest.mark.parametrize("T,Hg,Wg", [(2, 16, 16), (2, 13, 11), (3, 7, 17), (21, 30, 52)])
def test_layout_matches_tile_definition(T, Hg, Wg):
    p = api.problem(1, 1, 64, T, Hg, Wg)
    L = api.da2_layout_build(p)
    slot2tok, n_a, tok2slot = partition.tile_partition(T, Hg, Wg)
    R = n_a.size
    assert np.array_equal(L[:R], n_a)
    assert np.array_equal(L[R:R + 64 * R], slot2tok)
    assert np.array_equal(L[R + 64 * R:], tok2slot)


@pytest.mark.parametrize("T,Hg,Wg", [(2, 16, 16), (2, 13, 11), (3, 7, 17), (21, 30, 52), (1, 45, 80), (1, 2, 100),
                                     (1, 100, 2), (2, 1, 1), (1, 33, 7)])
def test_ragged_layout_matches_oracle_partition(T, Hg, Wg):
    """The library's ragged layout (host C++) and the oracle's ragged partition
    (independent Python) give the same blocks, slots and inverse map."""
    p = api.problem(1, 1, 64, T, Hg, Wg, "ragged")
    L = api.da2_layout_build(p)
    slot2tok, n_a, tok2slot = partition.ragged_partition(T, Hg, Wg)
    R = n_a.size
    assert api.da2_sizes(p)["R"] == R == T * (-(-Hg * Wg // 64))
    assert np.array_equal(L[:R], n_a)
    assert np.array_equal(L[R:R + 64 * R], slot2tok)
    assert np.array_equal(L[R + 64 * R:], tok2slot)


def test_invalid_problems():
    s = _lib.Sizes()
    L = _lib.lib()
    for bad in [(0, 1, 64, 1, 8, 8), (1, 1, 96, 1, 8, 8), (1, 1, 128, 1, 0, 8), (1, 1, 128, -1, 8, 8)]:
        assert L.da2_sizes(ctypes.byref(api.problem(*bad)), 0, ctypes.byref(s)) == _lib.DA2_ERR_INVALID_ARG
    assert L.da2_sizes(ctypes.byref(api.problem(1, 1, 64, 1, 8, 8)), 5, ctypes.byref(s)) == _lib.DA2_ERR_INVALID_ARG
    odd = api.problem(1, 1, 64, 1, 8, 8)
    odd.partition = 2
    assert L.da2_sizes(ctypes.byref(odd), 0, ctypes.byref(s)) == _lib.DA2_ERR_INVALID_ARG
    assert L.da2_sizes(None, 0, ctypes.byref(s)) == _lib.DA2_ERR_INVALID_ARG
    # more than 65535 blocks
    assert L.da2_sizes(ctypes.byref(api.problem(1, 1, 64, 2000, 80, 80)), 0, ctypes.byref(s)) == _lib.DA2_ERR_INVALID_ARG
    # more than 32767 heads in total
    assert L.da2_sizes(ctypes.byref(api.problem(2, 16384, 64, 1, 8, 8)), 0, ctypes.byref(s)) == _lib.DA2_ERR_INVALID_ARG
    assert L.da2_sizes(ctypes.byref(api.problem(1, 32767, 64, 1, 8, 8)), 0, ctypes.byref(s)) == _lib.DA2_OK
    n = 10
    buf = (ctypes.c_int32 * n)()
    assert L.da2_layout_build(ctypes.byref(api.problem(1, 1, 64, 1, 8, 8)), buf, n) == _lib.DA2_ERR_INVALID_ARG


FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: validation fails first


def _desc(dtype=_lib.DA2_BF16, sn=128):
    return _lib.Tensor(12 * 32760 * 128, 32760 * 128, sn, dtype, 0)


def test_compute_calls_validate_before_gpu():
    L = _lib.lib()
    p = _p(configs.MID)
    s = api.da2_sizes(p)
    d = _desc()
    ws = s["ws_draft_bytes"]
    E, W = _lib.DA2_ERR_INVALID_ARG, _lib.DA2_ERR_WORKSPACE
    assert L.da2_draft_map(None, FAKE, d, FAKE, p, 0.2, FAKE, FAKE, FAKE, ws, None) == E
    assert L.da2_draft_map(FAKE, FAKE, d, FAKE, p, 1.5, FAKE, FAKE, FAKE, ws, None) == E
    assert L.da2_draft_map(FAKE, FAKE, d, FAKE, p, float("nan"), FAKE, FAKE, FAKE, ws, None) == E
    assert L.da2_draft_map(FAKE, FAKE, _desc(dtype=7), FAKE, p, 0.2, FAKE, FAKE, FAKE, ws, None) == E
    assert L.da2_draft_map(FAKE, FAKE, _desc(sn=64), FAKE, p, 0.2, FAKE, FAKE, FAKE, ws, None) == E
    assert L.da2_draft_map(FAKE, FAKE, d, FAKE, p, 0.2, FAKE, FAKE, FAKE, ws - 1, None) == W
    wr = s["ws_rank_bytes"]
    for n16, n8, n4, den in [(0, 50, 60, 100), (0, -1, 10, 100), (0, 10, 10, 0), (0, 10, -5, 100), (-1, 10, 10, 100),
                             (70, 10, 30, 100)]:
        assert L.da2_rank_assign(FAKE, p, n16, n8, n4, den, 0, FAKE, FAKE, FAKE, wr, None) == E
    assert L.da2_rank_assign(FAKE, p, 0, 10, 30, 100, 3, FAKE, FAKE, FAKE, wr, None) == E
    assert L.da2_rank_assign(None, p, 0, 10, 30, 100, 0, FAKE, FAKE, FAKE, wr, None) == E
    assert L.da2_rank_assign(FAKE, p, 0, 10, 30, 100, 0, FAKE, FAKE, FAKE, wr - 1, None) == W
    big = api.problem(1, 1, 128, 33, 128, 128)           # R^2 >= 2^22 in head scope
    assert L.da2_rank_assign(FAKE, big, 0, 10, 30, 100, 0, FAKE, FAKE, FAKE, 1 << 40, None) == E
    assert L.da2_prep_operands(FAKE, None, FAKE, d, FAKE, p, 0, 0, FAKE, FAKE, None, 0, None) == E
    assert L.da2_prep_operands(FAKE, FAKE, FAKE, _desc(dtype=3), FAKE, p, 0, 0, FAKE, FAKE, None, 0, None) == E
    assert L.da2_prep_operands(FAKE, FAKE, FAKE, d, FAKE, p, 2, 0, FAKE, FAKE, None, 0, None) == E
    assert L.da2_prep_operands(FAKE, FAKE, FAKE, d, FAKE, p, 0, 2, FAKE, FAKE, None, 0, None) == E
    assert L.da2_prep_operands(FAKE, FAKE, FAKE, d, FAKE, p, 0, -1, FAKE, FAKE, None, 0, None) == E
    assert L.da2_mixed_attn(FAKE, FAKE, None, p, 0, d, FAKE, None) == E
    assert L.da2_mixed_attn(FAKE, FAKE, FAKE, p, 0, _desc(dtype=9), FAKE, None) == E
    assert L.da2_mixed_attn(FAKE, FAKE, FAKE, p, 2, d, FAKE, None) == E
    assert L.da2_mixed_attn(FAKE, FAKE, FAKE, p, -1, d, FAKE, None) == E


def test_inputs_must_allow_16_byte_loads():
    """Q, K, V are read in 16-byte vectors: misaligned bases or strides that
    are not a multiple of 16 bytes are rejected before any GPU work."""
    L = _lib.lib()
    p = _p(configs.MID)
    s = api.da2_sizes(p)
    E = _lib.DA2_ERR_INVALID_ARG
    odd = ctypes.c_void_p(0x1000 + 2)
    ws = s["ws_draft_bytes"]
    assert L.da2_draft_map(odd, FAKE, _desc(), FAKE, p, 0.2, FAKE, FAKE, FAKE, ws, None) == E
    assert L.da2_draft_map(FAKE, odd, _desc(), FAKE, p, 0.2, FAKE, FAKE, FAKE, ws, None) == E
    assert L.da2_prep_operands(FAKE, FAKE, odd, _desc(), FAKE, p, 0, 0, FAKE, FAKE, None, 0, None) == E
    assert L.da2_draft_map(FAKE, FAKE, _desc(sn=132), FAKE, p, 0.2, FAKE, FAKE, FAKE, ws, None) == E
    assert L.da2_prep_operands(FAKE, FAKE, FAKE, _desc(sn=130), FAKE, p, 0, 0, FAKE, FAKE, None, 0, None) == E
    f32 = _lib.Tensor(12 * 32760 * 128 + 2, 32760 * 128, 128, _lib.DA2_FP32, 0)
    assert L.da2_draft_map(FAKE, FAKE, f32, FAKE, p, 0.2, FAKE, FAKE, FAKE, ws, None) == E
    # fp32 rows need only 4-element alignment: the stride check passes and the
    # (deliberately short) workspace is what gets reported
    ok32 = _lib.Tensor(12 * 32760 * 132, 32760 * 132, 132, _lib.DA2_FP32, 0)
    assert L.da2_draft_map(FAKE, FAKE, ok32, FAKE, p, 0.2, FAKE, FAKE, FAKE, ws - 1, None) == _lib.DA2_ERR_WORKSPACE


@pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="checks the no-GPU path")
def test_no_device_is_reported_not_crashed():
    L = _lib.lib()
    p = _p(configs.TINY)
    s = api.da2_sizes(p)
    d = _lib.Tensor(2 * 512 * 64, 512 * 64, 64, _lib.DA2_FP32, 0)
    st = L.da2_draft_map(FAKE, FAKE, d, FAKE, p, 0.2, FAKE, FAKE, FAKE, s["ws_draft_bytes"], None)
    assert st in (_lib.DA2_ERR_UNSUPPORTED, _lib.DA2_ERR_HIP)
