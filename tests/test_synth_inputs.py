"""Seeded input generator: Philox-4x32-10 known-answer vectors and value ranges.

The known-answer vectors are the published ones for Philox-4x32 with 10 rounds
(Salmon et al., SC'11, distributed with the Random123 library); the paper's RNG
is this generator (Sec. 3 (iv)).
"""
import numpy as np

from paper_2609_10632_amd import synth


def test_philox_known_answers():
    assert synth.philox4x32_10([0, 0, 0, 0], [0, 0]) == [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]
    assert synth.philox4x32_10([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2) == [
        0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]
    assert synth.philox4x32_10([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344],
                               [0xA4093822, 0x299F31D0]) == [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]


def test_streams_are_deterministic_and_distinct():
    a = synth.bf16((4097,), 7)
    b = synth.bf16((4097,), 7)
    c = synth.bf16((4097,), 8)
    assert np.array_equal(a, b)
    assert not np.array_equal(a, c)
    # a prefix of a longer draw is the shorter draw (counter-based)
    assert np.array_equal(synth.bf16((1000,), 7), a[:1000])


def test_distributions():
    z = synth.bf16_to_f64(synth.bf16((1 << 20,), 11))
    assert abs(z.mean()) < 5e-3 and abs(z.std() - 1) < 5e-3
    u = synth.bf16_to_f64(synth.bf16((1 << 20,), 12, synth.UNIFORM, 0.0, 1.0))
    assert u.min() >= 0 and u.max() <= 1 and abs(u.mean() - 0.5) < 5e-3
    assert abs(u.var() - 1 / 12) < 1e-3


def test_bf16_rounding_round_trip():
    v = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 0.0, 1e-30])
    bits = synth.f64_to_bf16_bits(v)
    back = synth.bf16_to_f64(bits)
    # ties go to even: 1 + 2^-8 -> 1, 1 + 3*2^-8 -> 1 + 2^-6
    assert back[0] == 1.0 and back[1] == 1.0 and back[2] == 1.0 + 2 ** -6
    assert back[3] == -2.5 and back[4] == 0.0


def test_kaiming_uniform_width_ratio_matches_paper(golden):
    """Kaiming-normal (gain sqrt 2): std sqrt(2/fan_in).  Kaiming-uniform (a=sqrt 5): bound
    1/sqrt(fan_in), std 1/sqrt(3 fan_in).  The ratio is sqrt(6), printed as 2.45x."""
    fan_in = 432
    bound = synth.kaiming_uniform_bound(fan_in)
    w = synth.bf16_to_f64(synth.bf16((1 << 18,), 13, synth.UNIFORM, -bound, bound))
    assert np.all(np.abs(w) <= bound * (1 + 2 ** -8))
    std_u = w.std()
    assert abs(std_u - 1 / np.sqrt(3 * fan_in)) / std_u < 1e-2
    ratio = np.sqrt(2.0 / fan_in) / std_u
    assert round(ratio, 2) == golden["kaiming_normal_over_uniform_width"]["value"]
