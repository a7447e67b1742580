"""The counter-based input generator of the device-resident loop (CPU side).

Philox4x32-10 is pinned to the known-answer vectors published with the
generator's reference implementation (Random123, accompanying Salmon et al.,
SC 2011); the rest of the recipe to its stated arithmetic.
"""
import numpy as np
import torch

import oracle

from workloads import synth

# (counter, key) -> output, Philox4x32-10 known-answer tests
KAT = [
    ((0x00000000, 0x00000000, 0x00000000, 0x00000000), (0x00000000, 0x00000000),
     (0x6627e8d5, 0xe169c58d, 0xbc57ac4c, 0x9b00dbd8)),
    ((0xffffffff, 0xffffffff, 0xffffffff, 0xffffffff), (0xffffffff, 0xffffffff),
     (0x408f276d, 0x41c83b0e, 0xa20bc7c6, 0x6d5451fd)),
    ((0x243f6a88, 0x85a308d3, 0x13198a2e, 0x03707344), (0xa4093822, 0x299f31d0),
     (0xd16cfe09, 0x94fdcceb, 0x5001e420, 0x24126ea1)),
]


def test_philox_known_answers():
    for ctr, key, want in KAT:
        got = tuple(int(w) for w in synth.philox4x32_10(*ctr, *key))
        assert got == want, (ctr, [hex(g) for g in got])


def test_philox_vectorised_equals_scalar():
    rng = np.random.default_rng(0)
    c = rng.integers(0, 2 ** 32, (4, 50), dtype=np.uint64)
    vec = synth.philox4x32_10(c[0], c[1], c[2], c[3], 123, 456)
    for j in range(50):
        one = synth.philox4x32_10(int(c[0, j]), int(c[1, j]), int(c[2, j]), int(c[3, j]), 123, 456)
        assert all(int(vec[k][j]) == int(one[k]) for k in range(4))


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(20000).astype(np.float32) * 4,
                        (rng.integers(-510, 511, 2000) * 2.0 ** -7).astype(np.float32),
                        np.float32([1.00390625, 1.01171875, -1.00390625, 0.0, -0.0])])  # exact halfway cases
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(synth.bf16_bits(x), want)


def test_background_statistics_and_spike():
    V = 8192
    bits = synth.row_bits(7, 2, 5, 3, V)
    vals = synth.bf16_to_f32(bits).astype(np.float64)
    tok = synth.spike_token(7, 2, 5, V)
    h = float(synth.spike_height(7, 2, 5, 3))
    bg = np.delete(vals, tok)
    # sum of 4 uniform bytes: mean 510, variance 4 * (256^2 - 1) / 12, scaled by 2^-7
    assert abs(bg.mean()) < 0.05
    assert abs(bg.std() - np.sqrt(4 * (256 ** 2 - 1) / 12) / 128) < 0.05
    assert np.all(np.abs(bg) <= 510 / 128)
    assert 0.0 <= h < 14.0
    assert np.argmax(vals) == tok or h < 4.5
    # the token is fixed across steps, the height is not
    assert synth.spike_token(7, 2, 5, V) == tok
    assert any(float(synth.spike_height(7, 2, 5, t)) != h for t in range(4, 8))
    # reproducible and different per step
    assert np.array_equal(bits, synth.row_bits(7, 2, 5, 3, V))
    assert not np.array_equal(bits, synth.row_bits(7, 2, 5, 4, V))


def test_spike_height_modes():
    hs = np.array([float(synth.spike_height(11, b, i, 0)) for b in range(20) for i in range(20)])
    hi = hs >= 8.0
    assert 0.5 < hi.mean() < 0.7                   # P(u1 < 0.6) = 0.6
    assert np.all(hs[hi] < 14.0) and np.all(hs[~hi] < 6.0)
