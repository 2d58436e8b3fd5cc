"""The seeded input generator: Philox known answers, determinism, stream
independence, distribution moments, and its bf16 rounding."""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import moe_inputs as mi


def test_philox_known_answers():
    # Known-answer vectors published with the Random123 library (Salmon et al.,
    # SC'11) for Philox4x32 with 10 rounds.
    assert mi.philox4x32_10([0, 0, 0, 0], [0, 0]) == [0x6627E8D5, 0xE169C58D, 0xBC57AC4C,
                                                       0x9B00DBD8]
    assert mi.philox4x32_10([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2) == [0x408F276D, 0x41C83B0E,
                                                                      0xA20BC7C6, 0x6D5451FD]
    assert mi.philox4x32_10([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344],
                            [0xA4093822, 0x299F31D0]) == [0xD16CFE09, 0x94FDCCEB, 0x5001E420,
                                                          0x24126EA1]


def test_z_is_irwin_hall_of_philox_halves():
    seed, stream = 7, mi.stream_id(mi.KIND_GATE, 3, 5)
    for index in (0, 1, 12345, (1 << 32) + 17):
        r = mi.philox4x32_10([index & 0xFFFFFFFF, index >> 32, 0, 0], [seed, stream])
        s = sum((v & 0xFFFF) + (v >> 16) for v in r)
        assert mi.z_at(seed, stream, index) == 2 * s - 8 * 65535


def test_determinism_and_offsets():
    a = mi.gen_bf16(0, mi.stream_id(mi.KIND_X), (64, 33), 1.0)
    b = mi.gen_bf16(0, mi.stream_id(mi.KIND_X), (64, 33), 1.0)
    assert np.array_equal(a, b)
    # element i of the stream does not depend on how the tensor is cut
    c = mi.gen_bf16(0, mi.stream_id(mi.KIND_X), (100,), 1.0, start=1000)
    assert np.array_equal(c, a.reshape(-1)[1000:1100])


def test_streams_and_seeds_differ():
    base = mi.gen_bf16(0, mi.stream_id(mi.KIND_GATE, 0, 0), (4096,), 0.02)
    others = [
        mi.gen_bf16(1, mi.stream_id(mi.KIND_GATE, 0, 0), (4096,), 0.02),
        mi.gen_bf16(0, mi.stream_id(mi.KIND_UP, 0, 0), (4096,), 0.02),
        mi.gen_bf16(0, mi.stream_id(mi.KIND_GATE, 1, 0), (4096,), 0.02),
        mi.gen_bf16(0, mi.stream_id(mi.KIND_GATE, 0, 1), (4096,), 0.02),
    ]
    for o in others:
        assert np.mean(o == base) < 0.05
        # and they are uncorrelated
        fa = mi.bf16_bits_to_f32(base).astype(np.float64)
        fb = mi.bf16_bits_to_f32(o).astype(np.float64)
        assert abs(np.corrcoef(fa, fb)[0, 1]) < 0.06


@pytest.mark.parametrize("sigma", [1.0, 0.02, 0.006])
def test_moments(sigma):
    v = mi.gen_f32(3, mi.stream_id(mi.KIND_ROUTER), (400_000,), sigma).astype(np.float64)
    assert abs(v.mean()) < 0.01 * sigma
    assert abs(v.std() / sigma - 1.0) < 0.01
    # Irwin-Hall(8): excess kurtosis -6/(5*8) = -0.15; support +-sqrt(24) sd
    k = ((v / v.std()) ** 4).mean() - 3.0
    assert abs(k + 0.15) < 0.03
    assert np.abs(v).max() <= math.sqrt(24.0) * sigma * (1 + 1e-6)


def test_f32_is_rounded_double():
    seed, stream = 0, mi.stream_id(mi.KIND_ROUTER)
    c = mi.scale_for(0.02)
    got = mi.gen_f32(seed, stream, (50,), 0.02)
    for i in range(50):
        assert got[i] == np.float32(mi.z_at(seed, stream, i) * c)


def _bf16_nearest_even(v: float) -> int:
    """Brute force: the bf16 value nearest to v (exactly), ties to even bits."""
    x = Fraction(v)
    f32 = np.array([v], dtype=np.float32)
    base = int(f32.view(np.uint32)[0]) >> 16
    cands = set()
    for b in range(base - 2, base + 3):
        if 0 <= b < 0x10000 and (b & 0x7F80) != 0x7F80:
            cands.add(b)
        nb = b ^ 0x8000
        if 0 <= nb < 0x10000 and (nb & 0x7F80) != 0x7F80:
            cands.add(nb)

    def val(b):
        return Fraction(float(mi.bf16_bits_to_f32(np.array([b], dtype=np.uint16))[0]))

    best = min(cands, key=lambda b: (abs(val(b) - x), b & 1))
    return best


def test_generator_bf16_rounding_vs_torch_and_brute_force():
    rng = np.random.default_rng(1)
    f = rng.standard_normal(20000).astype(np.float32) * np.float32(3.0)
    f = np.concatenate([f, np.array([0.0, -0.0, 1e-40, -1e-40, 3e38, -3e38], np.float32)])
    want = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([mi.bf16_rne(float(v)) for v in f], dtype=np.uint16)
    assert np.array_equal(got, want)
    # doubles just off a bf16 midpoint (not representable in fp32)
    for v in rng.standard_normal(300):
        b = int(np.array([v], np.float32).view(np.uint32)[0] >> 16)
        lo = float(mi.bf16_bits_to_f32(np.array([b], np.uint16))[0])
        hi = float(mi.bf16_bits_to_f32(np.array([b + 1], np.uint16))[0])
        mid = (lo + hi) / 2
        for cand in (mid, math.nextafter(mid, math.inf), math.nextafter(mid, -math.inf)):
            assert mi.bf16_rne(cand) == _bf16_nearest_even(cand)
