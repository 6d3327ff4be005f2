"""Device format checks (gfx950): the library's software E4M3 / E2M1 encoders
and the hardware conversion instructions used by the attention kernel, against
the oracle's format definitions on exhaustive code tables, every midpoint
(ties), neighbours of every midpoint and random values."""
import ctypes
import os

import numpy as np
import pytest
import torch

from oracle import formats as F

pytestmark = pytest.mark.gpu
PROBE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "probes", "libda2_probe.so")


def _values():
    e4 = np.unique(np.abs(F.e4m3_decode(np.arange(0x7F))))
    mids4 = (e4[:-1] + e4[1:]) / 2
    e2 = F.E2M1_VALUES
    mids2 = (e2[:-1] + e2[1:]) / 2
    ints = np.arange(0, 131, dtype=np.float64)
    base = np.concatenate([e4, mids4, e2, mids2, ints, ints + 0.5,
                           [448.0, 449.0, 464.0, 470.0, 500.0, 1e6, 6.0, 6.5, 7.0, 100.0]])
    base = base.astype(np.float32)
    up = np.nextafter(base, np.float32(np.inf))
    down = np.nextafter(base, np.float32(0))
    rng = np.random.default_rng(0)
    rand = np.concatenate([rng.uniform(0, 8, 20000), rng.uniform(0, 460, 20000),
                           np.exp(rng.uniform(-25, 6, 20000))]).astype(np.float32)
    x = np.concatenate([base, up, down, rand])
    return np.concatenate([x, -x]).astype(np.float32)


@pytest.fixture(scope="module")
def probe():
    assert torch.cuda.is_available()
    lib = ctypes.CDLL(PROBE)
    x = _values()
    n = x.size
    xd = torch.from_numpy(x).cuda()
    outs = {k: torch.empty(n, dtype=dt, device="cuda") for k, dt in
            [("e2m1_sw", torch.float32), ("e2m1_hw", torch.float32), ("e2m1_hw_s2", torch.float32),
             ("e2m1_hw_back3", torch.float32), ("e4m3_sw", torch.int32), ("e4m3_hw", torch.int32),
             ("e4m3_mag_sw", torch.float32), ("e4m3_mag_hw", torch.float32), ("int8_code", torch.int32)]}
    order = ["e2m1_sw", "e2m1_hw", "e2m1_hw_s2", "e2m1_hw_back3", "e4m3_sw", "e4m3_hw", "e4m3_mag_sw", "e4m3_mag_hw",
             "int8_code"]
    args = [ctypes.c_void_p(xd.data_ptr()), ctypes.c_int(n)] + [ctypes.c_void_p(outs[k].data_ptr()) for k in order]
    args.append(ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert lib.da2_probe_formats(*args) == 0
    torch.cuda.synchronize()
    return x.astype(np.float64), {k: v.cpu().numpy() for k, v in outs.items()}


def test_software_e2m1(probe):
    x, o = probe
    np.testing.assert_array_equal(o["e2m1_sw"], F.e2m1(x))


def test_software_e4m3(probe):
    x, o = probe
    np.testing.assert_array_equal(o["e4m3_sw"].astype(np.uint8), F.e4m3_code(F.e4m3(x)))
    np.testing.assert_array_equal(o["e4m3_mag_sw"], F.e4m3(np.abs(x)))


def test_hardware_fp8_conversion_is_rne_in_range(probe):
    """v_cvt_pk_fp8_f32 (used for the 8-bit path's weights, all in [0, 448])."""
    x, o = probe
    inr = np.abs(x) <= 448.0
    want = F.e4m3_code(F.e4m3(x[inr]))
    got = o["e4m3_hw"][inr].astype(np.uint8)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, [(x[inr][i], got[i], want[i]) for i in bad[:10]]


def test_int8_code(probe):
    """The INT8 encoder's rounding (operand preparation): round half away from
    zero, clamped to [-127, 127], on every integer +- 0.5 tie up to 130, their
    float32 neighbours and the rest of the probe set."""
    x, o = probe
    want = np.clip(F.half_away(x.astype(np.float32)), -127, 127)
    bad = np.nonzero(o["int8_code"] != want)[0]
    assert bad.size == 0, [(x[i], o["int8_code"][i], want[i]) for i in bad[:10]]


def test_hardware_fp8_round_trip_value(probe):
    """v_cvt_pk_fp8_f32 then v_cvt_f32_fp8 on |x| clamped to 448 (how the
    attention rounds the NVFP4 weight scales sigma_P) gives the E4M3 value."""
    x, o = probe
    want = F.e4m3(np.minimum(np.abs(x), 448.0))
    bad = np.nonzero(o["e4m3_mag_hw"] != want)[0]
    assert bad.size == 0, [(x[i], o["e4m3_mag_hw"][i], want[i]) for i in bad[:10]]


def test_hardware_fp4_conversion(probe):
    """v_cvt_scalef32_pk_fp4_f32 then v_cvt_scalef32_pk_f16_fp4, unit scales:
    round to nearest even with saturation and signed zeros, like the E2M1 cast
    definition."""
    x, o = probe
    want = F.e2m1(x)
    bad = np.nonzero(o["e2m1_hw"] != want)[0]
    print("fp4 hw mismatches:", bad.size, [(x[i], o["e2m1_hw"][i], want[i]) for i in bad[:12]])
    # how the scale operands act (recorded for the kernel design)
    s2_div = np.mean(o["e2m1_hw_s2"] == F.e2m1(x / 2))
    s2_mul = np.mean(o["e2m1_hw_s2"] == F.e2m1(x * 2))
    b3_full = np.mean(o["e2m1_hw_back3"] == F.e2m1(x) * 3)
    b3_exp = np.mean(o["e2m1_hw_back3"] == F.e2m1(x) * 2)
    # the operand encoder relies on E2M1 zeros keeping the sign of their input
    zero = want == 0
    assert np.array_equal(np.signbit(o["e2m1_hw"][zero]), np.signbit(want[zero]))
    print(f"encode scale 2: matches x/2 {s2_div:.4f}, x*2 {s2_mul:.4f}; "
          f"decode scale 3: full {b3_full:.4f}, exponent only {b3_exp:.4f}")
    assert bad.size == 0


def test_lds_dma_placement():
    """global_load_lds_dwordx4 puts lane i's 16 bytes at base + 16 i (the
    attention kernel stages 1 KB operand fragments this way)."""
    lib = ctypes.CDLL(PROBE)
    src = torch.arange(256, dtype=torch.int32, device="cuda") * 7 + 3
    out = torch.zeros(1024, dtype=torch.int32, device="cuda")
    assert lib.da2_probe_lds_dma(ctypes.c_void_p(src.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                                 ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)) == 0
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    assert np.array_equal(o[64:320], src.cpu().numpy())
    assert np.all(o[:64] == -1) and np.all(o[320:] == -1)


def test_scaled_fp4_mfma_layout():
    """v_mfma_scale_f32_32x32x64_f8f6f4 with E2M1 operands: lane l of A holds row
    l%32 and k = 32(l/32) + i at nibble i (little-endian), lane l of B holds
    column l%32 with the same k, each lane's E8M0 byte (chosen by the selector)
    scales its 32 values, and accumulator register i of lane l is row
    8(i/4) + 4(l/32) + i%4, column l%32 (the layout the MX 4-bit phase uses)."""
    lib = ctypes.CDLL(PROBE)
    rng = np.random.default_rng(3)
    codes_a = rng.integers(0, 16, (64, 32)).astype(np.uint32)
    codes_b = rng.integers(0, 16, (64, 32)).astype(np.uint32)

    def pack(c):
        words = np.zeros((64, 4), np.uint32)
        for i in range(32):
            words[:, i // 8] |= c[:, i] << (4 * (i % 8))
        return words

    sa = rng.integers(120, 134, (64, 4)).astype(np.uint32)
    sb = rng.integers(120, 134, (64, 4)).astype(np.uint32)
    sa_w = (sa[:, 0] | (sa[:, 1] << 8) | (sa[:, 2] << 16) | (sa[:, 3] << 24)).astype(np.uint32)
    sb_w = (sb[:, 0] | (sb[:, 1] << 8) | (sb[:, 2] << 16) | (sb[:, 3] << 24)).astype(np.uint32)
    dev = [torch.from_numpy(x.view(np.int32).copy()).cuda() for x in (pack(codes_a), pack(codes_b), sa_w, sb_w)]
    out = torch.zeros(4 * 64 * 16, dtype=torch.float32, device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    assert lib.da2_probe_mfma_fp4(*[ctypes.c_void_p(t.data_ptr()) for t in dev], ctypes.c_void_p(out.data_ptr()),
                                  stream) == 0
    torch.cuda.synchronize()
    got = out.cpu().numpy().reshape(4, 64, 16)
    mag = F.E2M1_VALUES
    val = lambda c: np.where(c & 8, -1.0, 1.0) * mag[c & 7]
    va, vb = val(codes_a), val(codes_b)
    for sel in range(4):
        A = np.zeros((32, 64))
        B = np.zeros((64, 32))
        for l in range(64):
            r, h = l % 32, l // 32
            A[r, 32 * h:32 * h + 32] = va[l] * 2.0 ** (int(sa[l, sel]) - 127)
            B[32 * h:32 * h + 32, r] = vb[l] * 2.0 ** (int(sb[l, sel]) - 127)
        D = A @ B
        for l in range(64):
            for i in range(16):
                row = 8 * (i // 4) + 4 * (l // 32) + i % 4
                assert got[sel, l, i] == pytest.approx(D[row, l % 32], rel=1e-6, abs=1e-30), (sel, l, i)
