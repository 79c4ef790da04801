"""The seeded input generators' bf16 rounding: round to nearest, ties to even,
on hand-picked bit patterns whose correct results follow from the format."""
import numpy as np

from paper_2607_07740_amd import synth


def _bits(u32):
    return np.array(u32, dtype=np.uint32).view(np.float32)


def test_bf16_rounding_ties_carries_and_specials():
    cases = {
        0x3F800000: 0x3F80,  # 1.0 exact
        0x3F808000: 0x3F80,  # tie, even below: down
        0x3F818000: 0x3F82,  # tie, odd below: up
        0x3F808001: 0x3F81,  # just above the tie: up
        0x3F807FFF: 0x3F80,  # just below the tie: down
        0x3FFF8000: 0x4000,  # tie rounding up carries into the exponent (1.99.. -> 2)
        0x7F7FFFFF: 0x7F80,  # largest float rounds to +inf in bf16
        0x7F800000: 0x7F80,  # +inf
        0xFF800000: 0xFF80,  # -inf
        0x00000000: 0x0000,
        0x80000000: 0x8000,  # -0 keeps its sign
        0xBF818000: 0xBF82,  # negative tie, odd below: away from zero
        0x00008000: 0x0000,  # subnormal tie to even (zero)
        0x00018000: 0x0002,  # subnormal tie, odd below: up
        0x7FC00000: 0x7FC0,  # quiet NaN
    }
    got = synth.bf16_bits(_bits(list(cases)))
    assert [int(x) for x in got] == list(cases.values())


def test_bf16_round_trip_is_exact_and_nearest():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(1 << 16).astype(np.float32)
    b = synth.bf16_bits(x)
    y = synth.bf16_to_f32(b)
    assert np.array_equal(synth.bf16_bits(y), b)  # representable values are fixed points
    # no other bf16 value is nearer: compare with both neighbours
    up = synth.bf16_to_f32(b + 1).astype(np.float64)
    dn = synth.bf16_to_f32(b - 1).astype(np.float64)
    err = np.abs(y.astype(np.float64) - x)
    assert (err <= np.abs(up - x)).all() and (err <= np.abs(dn - x)).all()
