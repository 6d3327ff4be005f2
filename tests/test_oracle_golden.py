"""The oracle's constants against the values the paper prints (tests/golden)."""
import os

import numpy as np

from oracle import attention, encode, formats

HERE = os.path.dirname(os.path.abspath(__file__))


def _golden():
    vals = {}
    with open(os.path.join(HERE, "golden", "format_constants.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                name, value = line.split()[:2]
                vals[name] = float(value)
    return vals


def test_constants_match_paper():
    g = _golden()
    assert formats.E4M3_MAX == g["e4m3_max"] and formats.E2M1_MAX == g["e2m1_max"]
    assert attention.FP4_P_SCALE == g["fp4_p_scale"] == g["e2m1_max"] * g["e4m3_max"]
    assert attention.GROUP == encode.GROUP == g["nvfp4_group"]
    # eta is the inverse of the exp2 amplification, to the digits printed
    assert abs(attention.ETA - g["eta"]) < 5e-10
    assert abs(attention.AMP - 2.0 ** g["exp2_offset"]) < 1e-12
    # "amplifying the weights by approximately 448", and never above the E4M3 maximum
    assert attention.AMP < g["e4m3_max"] and abs(attention.AMP / g["e4m3_max"] - 1) < 1e-3
    # the E4M3 V codes stay in range: 2.25 is a representable E4M3 value
    assert formats.e4m3(g["v_e4m3_divisor"]) == g["v_e4m3_divisor"]
    # INT8 scale: delta = amax/127 + 1e-7 maps amax to a code just under 127
    amax = np.float32(3.0)
    delta = formats.f32(formats.f32(amax / np.float32(g["int8_code_max"])) + np.float32(g["int8_scale_eps"]))
    assert 126.99 < float(amax) / float(delta) < 127.0
