"""The seeded generator: Philox4x32-10 known-answer vectors and the Box-Muller
stream layout (CPU)."""
import math

import numpy as np

import synth


def test_philox_known_answers():
    # Known-answer vectors published with Random123 (Salmon et al., SC'11).
    assert list(synth.philox([0, 0, 0, 0], [0, 0])) == [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]
    assert list(synth.philox([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2)) == [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]
    assert list(synth.philox([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0])) == [
        0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]


def test_box_muller_stream_layout():
    seed = synth.seed_of("unit", 7)
    z = synth.normal_f32(seed, (64,), std=1.0)
    for j in range(16):
        w = synth.philox([j, 0, 0, 0], [seed & 0xFFFFFFFF, seed >> 32])
        u = [(int(x) + 1.0) / 4294967296.0 for x in w]
        r0, r1 = math.sqrt(-2 * math.log(u[0])), math.sqrt(-2 * math.log(u[2]))
        ref = [r0 * math.cos(2 * math.pi * u[1]), r0 * math.sin(2 * math.pi * u[1]),
               r1 * math.cos(2 * math.pi * u[3]), r1 * math.sin(2 * math.pi * u[3])]
        np.testing.assert_allclose(z[4 * j:4 * j + 4], np.float32(ref), rtol=1e-6, atol=1e-6)


def test_offsets_and_bf16_rounding():
    seed = synth.seed_of("unit", 8)
    full = synth.normal_f32(seed, (1001,), std=0.02)
    part = synth.normal_f32(seed, (500,), std=0.02, offset=333)
    np.testing.assert_array_equal(full[333:833], part)
    b = synth.normal_bf16(seed, (1001,), std=0.02)
    widened = synth.bf16_to_f32(b)
    # RNE: each bf16 value is the nearest representable to the float32 value
    ulp = 2.0 ** (np.floor(np.log2(np.abs(full.astype(np.float64)))) - 7)
    assert np.all(np.abs(widened.astype(np.float64) - full) <= ulp * 0.5)
    np.testing.assert_array_equal(synth.f32_to_bf16(full), b)


def test_moments_and_independence():
    a = synth.as_f32(synth.normal_bf16(synth.seed_of("m", 1), (1 << 20,), std=0.02))
    b = synth.as_f32(synth.normal_bf16(synth.seed_of("m", 2), (1 << 20,), std=0.02))
    assert abs(a.std() - 0.02) < 2e-4 and abs(a.mean()) < 1e-4
    assert abs(np.corrcoef(a, b)[0, 1]) < 5e-3
