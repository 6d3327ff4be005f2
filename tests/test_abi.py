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
    lo = api.da2_lists_offsets(_p(configs.MID))
    assert lo[1] >= 2 * 12 * 588 * 588 and lo[2] - lo[1] >= 16 * 12 * 588 and s["lists_bytes"] >= lo[3] + 32
    wo = api.da2_ws_draft_offsets(_p(configs.MID))
    assert wo[6] >= wo[5] + 8 * 12 * 588 * 588 and len(wo) == 7
    assert s["ws_draft_bytes"] >= wo[6] + 2 * 4 * 12 * 588


SECTION_BYTES = {  # per (head, block) at d = 128
    "nv": 36 * 128, "8": 64 * 128, "16": 2 * 64 * 128, "mx": 5 * 1024}


@pytest.mark.parametrize("fmt4", ["nvfp4", "mxfp4"])
@pytest.mark.parametrize("with16", [False, True])
def test_ops_sized_by_encoding(fmt4, with16):
    """The ops buffer holds exactly the sections a run with (fmt4, with16)
    writes: the 8-bit sections and scales, the 4-bit encoding in use, then the
    16-bit sections; the others are reported at offset -1."""
    p = _p(configs.MID)
    BH, R, d = 12, 588, 128
    off = api.da2_ops_offsets(p, fmt4, with16)
    s = api.da2_sizes(p, "head", fmt4, with16)
    four = [0, 1, 2] if fmt4 == "nvfp4" else [13, 14, 15]
    other4 = [13, 14, 15] if fmt4 == "nvfp4" else [0, 1, 2]
    present = [3, 4, 5, 6, 7, 8, 9] + four + ([10, 11, 12] if with16 else [])
    assert all(off[i] < 0 for i in range(16) if i not in present)
    assert all(off[i] >= 0 and off[i] % 256 == 0 for i in present)
    assert [off[i] for i in present] == sorted(off[i] for i in present)   # the documented order
    assert off[3] == 0
    size4 = SECTION_BYTES["nv" if fmt4 == "nvfp4" else "mx"] * BH * R
    for a, b in zip(four, four[1:]):
        assert off[b] - off[a] >= size4
    assert off[four[0]] >= off[9] + 16 * BH
    if with16:
        assert off[10] >= off[four[2]] + size4 and s["ops_bytes"] >= off[12] + SECTION_BYTES["16"] * BH * R
    else:
        assert s["ops_bytes"] >= off[four[2]] + size4
        assert s["ops_bytes"] < off[four[2]] + size4 + 4096
    # no offset other than the 16-bit ones depends on with16
    alt = api.da2_ops_offsets(p, fmt4, not with16)
    assert all(off[i] == alt[i] for i in range(16) if i not in (10, 11, 12))
    assert all(o < 0 for i, o in enumerate(off) if i in other4)


def test_nvfp4_sections_are_4_5_bits_per_value():
    """The packed NVFP4 operands take 36 d bytes per block (4-bit codes plus
    one E4M3 scale byte per 16 values): the mid layer's NVFP4 run needs about
    half the ops bytes of round-trip fp16 sections."""
    p = _p(configs.MID)
    s = api.da2_sizes(p, "head", "nvfp4", False)
    e = 12 * 37632 * 128
    assert s["ops_bytes"] < 3 * e + 3 * 36 * 128 * 12 * 588 + 64 * 1024 + 12 * 4 * (2 * 588 + 128 + 4)
    assert api.da2_ops_layout_version() == _lib.DA2_OPS_LAYOUT_VERSION == 2


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
    sz = lambda p, scope=0, fmt4=0, with16=0: L.da2_sizes(p, scope, fmt4, with16, ctypes.byref(s))
    for bad in [(0, 1, 64, 1, 8, 8), (1, 1, 128, 1, 0, 8), (1, 1, 128, -1, 8, 8)]:
        assert sz(ctypes.byref(api.problem(*bad))) == _lib.DA2_ERR_INVALID_ARG
    # a valid head dimension the kernels do not implement
    assert sz(ctypes.byref(api.problem(1, 1, 96, 1, 8, 8))) == _lib.DA2_ERR_UNSUPPORTED
    ok = ctypes.byref(api.problem(1, 1, 64, 1, 8, 8))
    assert sz(ok, 5) == _lib.DA2_ERR_INVALID_ARG
    assert sz(ok, 0, 2) == _lib.DA2_ERR_INVALID_ARG
    assert sz(ok, 0, 0, 2) == _lib.DA2_ERR_INVALID_ARG
    odd = api.problem(1, 1, 64, 1, 8, 8)
    odd.partition = 2
    assert sz(ctypes.byref(odd)) == _lib.DA2_ERR_INVALID_ARG
    assert sz(None) == _lib.DA2_ERR_INVALID_ARG
    # more than 65535 blocks
    assert sz(ctypes.byref(api.problem(1, 1, 64, 2000, 80, 80))) == _lib.DA2_ERR_INVALID_ARG
    # more than 32767 heads in total
    assert sz(ctypes.byref(api.problem(2, 16384, 64, 1, 8, 8))) == _lib.DA2_ERR_INVALID_ARG
    assert sz(ctypes.byref(api.problem(1, 32767, 64, 1, 8, 8))) == _lib.DA2_OK
    off = (ctypes.c_int64 * 16)()
    assert L.da2_ops_offsets(ok, 3, 0, off) == _lib.DA2_ERR_INVALID_ARG
    assert L.da2_ops_offsets(ok, 0, -1, off) == _lib.DA2_ERR_INVALID_ARG
    n = 10
    buf = (ctypes.c_int32 * n)()
    assert L.da2_layout_build(ok, buf, n) == _lib.DA2_ERR_INVALID_ARG


FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: validation fails first


def _desc(dtype=_lib.DA2_BF16, sn=128):
    return _lib.Tensor(12 * 32760 * 128, 32760 * 128, sn, dtype, 0)


def test_compute_calls_validate_before_gpu():
    L = _lib.lib()
    p = _p(configs.MID)
    s = api.da2_sizes(p)
    d = _desc()
    ws = s["ws_draft_bytes"]
    big_ops = 1 << 40
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
    assert L.da2_prep_operands(FAKE, None, FAKE, d, FAKE, p, 0, 0, FAKE, FAKE, big_ops, None, 0, None) == E
    assert L.da2_prep_operands(FAKE, FAKE, FAKE, _desc(dtype=3), FAKE, p, 0, 0, FAKE, FAKE, big_ops, None, 0, None) == E
    assert L.da2_prep_operands(FAKE, FAKE, FAKE, d, FAKE, p, 2, 0, FAKE, FAKE, big_ops, None, 0, None) == E
    assert L.da2_prep_operands(FAKE, FAKE, FAKE, d, FAKE, p, 0, 2, FAKE, FAKE, big_ops, None, 0, None) == E
    assert L.da2_prep_operands(FAKE, FAKE, FAKE, d, FAKE, p, 0, -1, FAKE, FAKE, big_ops, None, 0, None) == E
    assert L.da2_mixed_attn(FAKE, big_ops, FAKE, None, p, 0, d, FAKE, None) == E
    assert L.da2_mixed_attn(FAKE, big_ops, FAKE, FAKE, p, 0, _desc(dtype=9), FAKE, None) == E
    assert L.da2_mixed_attn(FAKE, big_ops, FAKE, FAKE, p, 2, d, FAKE, None) == E
    assert L.da2_mixed_attn(FAKE, big_ops, FAKE, FAKE, p, -1, d, FAKE, None) == E
    # an ops buffer smaller than the encoding's sections
    need = api.da2_sizes(p, "head", "nvfp4", False)["ops_bytes"]
    assert L.da2_prep_operands(FAKE, FAKE, FAKE, d, FAKE, p, 0, 0, FAKE, FAKE, need - 1, None, 0, None) == E
    need16 = api.da2_sizes(p, "head", "nvfp4", True)["ops_bytes"]
    assert L.da2_prep_operands(FAKE, FAKE, FAKE, d, FAKE, p, 1, 0, FAKE, FAKE, need16 - 1, None, 0, None) == E
    assert L.da2_mixed_attn(FAKE, need - 1, FAKE, FAKE, p, 0, d, FAKE, None) == E
    mx = api.da2_sizes(p, "head", "mxfp4", False)["ops_bytes"]
    assert L.da2_mixed_attn(FAKE, mx - 1, FAKE, FAKE, p, 1, d, FAKE, None) == E


def test_inputs_must_allow_16_byte_loads():
    """Q, K, V are read in 16-byte vectors: misaligned bases or strides that
    are not a multiple of 16 bytes are rejected before any GPU work."""
    L = _lib.lib()
    p = _p(configs.MID)
    s = api.da2_sizes(p)
    E = _lib.DA2_ERR_INVALID_ARG
    odd = ctypes.c_void_p(0x1000 + 2)
    ws = s["ws_draft_bytes"]
    big_ops = 1 << 40
    assert L.da2_draft_map(odd, FAKE, _desc(), FAKE, p, 0.2, FAKE, FAKE, FAKE, ws, None) == E
    assert L.da2_draft_map(FAKE, odd, _desc(), FAKE, p, 0.2, FAKE, FAKE, FAKE, ws, None) == E
    assert L.da2_prep_operands(FAKE, FAKE, odd, _desc(), FAKE, p, 0, 0, FAKE, FAKE, big_ops, None, 0, None) == E
    assert L.da2_draft_map(FAKE, FAKE, _desc(sn=132), FAKE, p, 0.2, FAKE, FAKE, FAKE, ws, None) == E
    assert L.da2_prep_operands(FAKE, FAKE, FAKE, _desc(sn=130), FAKE, p, 0, 0, FAKE, FAKE, big_ops, None, 0, None) == E
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
