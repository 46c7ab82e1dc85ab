"""Pins for the oracle's int4 affine group-64 format (CPU only).

Each check fixes the oracle to something other than itself: the sizes the
paper prints (§3.1 Problem, §3.2 Motivation), brute force over the 16 levels,
exact rational arithmetic and hand-built extreme cases.
"""

import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import quant

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_paper_byte_counts():
    g = json.load(open(os.path.join(GOLD, "paper_sizes.json")))
    e = quant.expert_bytes(2048, 512)
    assert e == 1_769_472
    assert round(e / 1e6, 2) == g["expert_MB"]
    layer = e * g["experts"]
    assert round(layer / 1e6) == g["layer_MB_256_experts"]
    routed = layer * g["layers"]
    assert round(routed / 1e9) == g["routed_GB_40_layers"]
    assert round(routed / 2 ** 30, 1) == g["routed_GiB_40_layers"]
    assert round(4 * e / 1e6) == g["k4_layer_experts_MB_approx"]
    # 0.5625 bytes per weight
    assert quant.projection_bytes(512, 2048) * 8 == 512 * 2048 * 4.5


def test_lora_bytes():
    # fp16 A [r, in] and B [out, r] on gate, up, down for the 35B-class shape
    assert quant.lora_bytes(2048, 512, 16) == 2 * (16 * 2048 * 2 + 512 * 16 * 2 + 16 * 512 + 2048 * 16)
    assert quant.lora_bytes(2048, 512, 16) == 245_760


def test_nibble_order():
    packed = np.array([[0x21, 0xF0]], dtype=np.uint8)
    assert quant.unpack_nibbles(packed).tolist() == [[1, 2, 0, 15]]
    rs = np.random.default_rng(0)
    q = rs.integers(0, 16, size=(5, 128)).astype(np.uint8)
    assert np.array_equal(quant.unpack_nibbles(quant.pack_nibbles(q)), q)


def test_quantize_exact_rational_group():
    # lo = -1, hi = 14: s = 1 and z = -1 exactly; w_j = -1 + 15 j / 63,
    # so the code is round(5 j / 21), which never sits on a half.
    j = np.arange(64)
    w = (-1.0 + 15.0 * j / 63.0).astype(np.float32)[None, :]
    q, s, z = quant.quantize_g64(w)
    assert float(s[0, 0]) == 1.0 and float(z[0, 0]) == -1.0
    want = [round(Fraction(5 * int(i), 21)) for i in j]
    assert q[0].tolist() == want


def test_quantize_brute_force_nearest_level():
    rs = np.random.default_rng(1)
    w = rs.normal(0, 0.02, size=(64, 256)).astype(np.float32)
    q, s, z = quant.quantize_g64(w)
    assert q.min() >= 0 and q.max() <= 15
    s64 = np.repeat(s.astype(np.float64), 64, axis=1)
    z64 = np.repeat(z.astype(np.float64), 64, axis=1)
    levels = s64[..., None] * np.arange(16) + z64[..., None]        # [rows, cols, 16]
    dist = np.abs(w.astype(np.float64)[..., None] - levels)
    best = np.argmin(dist, axis=-1)
    t = (w.astype(np.float64) - z64) / s64
    frac = np.abs(t - np.floor(t) - 0.5)
    clear = (frac > 1e-4) & (t > -0.5 + 1e-4) & (t < 15.5 - 1e-4)
    assert clear.mean() > 0.99
    assert np.array_equal(q[clear], best[clear])
    # reconstruction error within half a step for unclamped weights
    what = quant.dequantize_g64(q, s, z)
    inside = (t >= -0.5) & (t <= 15.5)
    assert np.all(np.abs(what - w)[inside] <= 0.5 * s64[inside] * (1 + 1e-3))


def test_quantize_clamps_and_extremes():
    w = np.linspace(-1.0, 1.0, 64, dtype=np.float32)[None, :]
    q, s, z = quant.quantize_g64(w)
    assert q[0, 0] == 0 and q[0, -1] == 15
    # all-zero codes give z, all-15 codes give 15 s + z
    zeros = quant.dequantize_g64(np.zeros((1, 64), np.uint8), s, z)
    full = quant.dequantize_g64(np.full((1, 64), 15, np.uint8), s, z)
    assert np.all(zeros == float(z[0, 0]))
    assert np.all(full == 15 * float(s[0, 0]) + float(z[0, 0]))


def test_quantize_constant_group():
    w = np.full((2, 64), 0.3, dtype=np.float32)
    q, s, z = quant.quantize_g64(w)
    assert np.all(s == 0) and np.all(q == 0)
    assert np.all(z == np.float16(0.3))
    assert np.all(quant.dequantize_g64(q, s, z) == float(np.float16(0.3)))


def test_quantize_group_axis_is_input_dim():
    # scaling one 64-wide input block of a row changes only that block's (s, z)
    rs = np.random.default_rng(2)
    w = rs.normal(0, 0.02, size=(3, 192)).astype(np.float32)
    w2 = w.copy()
    w2[1, 64:128] *= 4
    _, s1, _ = quant.quantize_g64(w)
    _, s2, _ = quant.quantize_g64(w2)
    diff = (s1 != s2)
    assert diff.tolist() == [[False, False, False], [False, True, False], [False, False, False]]


def test_dequantize_is_exact():
    rs = np.random.default_rng(3)
    q = rs.integers(0, 16, size=(4, 128)).astype(np.uint8)
    s = rs.uniform(0.001, 0.01, size=(4, 2)).astype(np.float16)
    z = rs.uniform(-0.05, 0.0, size=(4, 2)).astype(np.float16)
    got = quant.dequantize_g64(q, s, z)
    for r in range(4):
        for c in range(128):
            exact = Fraction(float(s[r, c // 64])) * int(q[r, c]) + Fraction(float(z[r, c // 64]))
            assert Fraction(float(got[r, c])) == exact


@pytest.mark.parametrize("shape", [(1, 64), (7, 128)])
def test_quantize_rejects_ragged_groups(shape):
    with pytest.raises(ValueError):
        quant.quantize_g64(np.zeros((shape[0], shape[1] + 1), np.float32))


def test_input_recipe_quantizer_matches_the_oracle():
    """The seeded inputs' quantized weights (synth.quantized_projection, the
    configuration's recipe) carry exactly the codes, scales and zeros of the
    oracle's quantizer on the same fp32 masters."""
    import synth
    for key, (o, i) in (((3, 1, 4), (16, 128)), ((3, 5, 9), (64, 512)), ((7, 0, 2), (8, 2048))):
        q, s, z = synth.quantized_projection(key, o, i)
        qo, so, zo = quant.quantize_g64(synth.fp32_weights(key, o, i))
        un = np.empty((o, i), dtype=np.uint8)
        un[:, 0::2] = q & 15
        un[:, 1::2] = q >> 4
        assert np.array_equal(un, qo)
        assert np.array_equal(s.view(np.uint16), so.view(np.uint16))
        assert np.array_equal(z.view(np.uint16), zo.view(np.uint16))
