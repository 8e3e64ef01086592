"""Input generator: rounding to the 16-bit input types, exact widening, and
determinism.  The expected bit patterns are written out by hand from the
formats' definitions (bfloat16: 8 exponent bits, 7 fraction bits; IEEE half: 5
exponent bits, 10 fraction bits; ties round to the even neighbour)."""

import numpy as np
import pytest

from paper_2410_17243_amd import synth


def _f32(*vals):
    return np.array(vals, dtype=np.float32)


def test_bf16_round_to_nearest_even():
    x = _f32(1.0, 1.0 + 2.0**-8, 1.0 + 3 * 2.0**-8, 1.0 + 2.0**-8 + 2.0**-20, -(1.0 + 2.0**-8 + 2.0**-20), 0.0, -2.0)
    # 1+2^-8 is the midpoint of 1 and 1+2^-7: even (1.0); 1+3*2^-8 is the
    # midpoint of 1+2^-7 and 1+2^-6: even (1+2^-6); just above a midpoint rounds up
    want = np.array([0x3F80, 0x3F80, 0x3F82, 0x3F81, 0xBF81, 0x0000, 0xC000], dtype=np.uint16)
    np.testing.assert_array_equal(synth.f32_to_bf16_bits(x), want)
    np.testing.assert_array_equal(synth.bf16_bits_to_f32(want), _f32(1.0, 1.0, 1.0 + 2.0**-6, 1.0 + 2.0**-7,
                                                                      -(1.0 + 2.0**-7), 0.0, -2.0))


def test_f16_generator_rounding_and_widening():
    img, txt = synth.clip_pairs(300, 64, 1.0, seed=4, dtype="f16")
    assert img.dtype == np.uint16 and txt.dtype == np.uint16
    f32i, f32t = synth.clip_pairs(300, 64, 1.0, seed=4, dtype="f32")
    # round to nearest even from the same float32 values, then exact widening
    np.testing.assert_array_equal(img, f32i.astype(np.float16).view(np.uint16))
    wide = synth.as_f64(img, "f16")
    np.testing.assert_array_equal(wide, f32i.astype(np.float16).astype(np.float64))
    # half-format spot checks: 1 + 2^-11 ties to 1.0, 1 + 3*2^-11 to 1 + 2^-9
    h = _f32(1.0 + 2.0**-11, 1.0 + 3 * 2.0**-11, -0.5).astype(np.float16).view(np.uint16)
    np.testing.assert_array_equal(h, np.array([0x3C00, 0x3C02, 0xB800], dtype=np.uint16))
    # rows stay unit vectors within the half rounding (2^-11 relative per element)
    nrm = np.linalg.norm(wide, axis=1)
    assert np.all(np.abs(nrm - 1.0) < 2e-3)


@pytest.mark.parametrize("dtype", ["bf16", "f16", "f32"])
def test_generator_deterministic_and_chunked(dtype):
    a1, b1 = synth.clip_pairs(1000, 32, 0.5, seed=9, dtype=dtype)
    a2, b2 = synth.clip_pairs(1000, 32, 0.5, seed=9, dtype=dtype)
    np.testing.assert_array_equal(a1, a2)
    np.testing.assert_array_equal(b1, b2)
    # rows of a smaller batch are the leading rows of a larger one (per-chunk seeds)
    a3, _ = synth.clip_pairs(400, 32, 0.5, seed=9, dtype=dtype)
    np.testing.assert_array_equal(a3, a1[:400])
    a4, _ = synth.clip_pairs(400, 32, 0.5, seed=10, dtype=dtype)
    assert not np.array_equal(a4, a3)


def test_generator_rejects_unknown_dtype():
    with pytest.raises(ValueError):
        synth.clip_pairs(4, 8, 1.0, dtype="fp8")
