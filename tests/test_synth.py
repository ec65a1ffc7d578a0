"""Seeded input generator: SplitMix64 known-answer vector, value ranges, bf16 rounding."""
import numpy as np
import torch

import synth


def test_splitmix64_published_sequence():
    # SplitMix64 started from state 0 (Steele, Lea & Flood 2014; the widely
    # reproduced reference outputs of Vigna's splitmix64.c).
    x = synth.splitmix64(0, 0, 3)
    assert [int(v) for v in x] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_counter_based_start_offset():
    full = synth.splitmix64(7, 3, 100)
    part = synth.splitmix64(7, 3, 40, start=60)
    assert np.array_equal(full[60:], part)


def test_streams_differ():
    a = synth.uniform(0, 0, (1000,), -1, 1)
    b = synth.uniform(0, 1, (1000,), -1, 1)
    assert not np.array_equal(a, b)


def test_uniform_range_and_grid():
    u = synth.uniform(0, 5, (200000,), -1.0 / 64, 1.0 / 64)
    assert u.dtype == np.float32
    assert u.min() >= -1.0 / 64 and u.max() < 1.0 / 64
    assert abs(float(u.mean())) < 1e-4


def test_normal_moments():
    z = synth.normal(0, 9, (400000,)).astype(np.float64)
    assert abs(z.mean()) < 0.01
    assert abs(z.std() - 1.0) < 0.01
    assert np.all(np.isfinite(z))


def test_bf16_rne_matches_torch_random():
    v = synth.normal(0, 11, (1_000_000,), scale=3.0)
    mine = synth.to_bf16_bits(v)
    ref = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(mine, ref)


def test_bf16_rne_ties_to_even():
    # Exact halfway cases: low 16 bits == 0x8000; even mantissa stays, odd rounds up.
    bits = np.array([0x3F808000, 0x3F818000, 0xBF808000, 0xBF818000, 0x3F80FFFF, 0x3F807FFF],
                    dtype=np.uint32)
    v = bits.view(np.float32)
    mine = synth.to_bf16_bits(v)
    ref = torch.from_numpy(v.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(mine, ref)
    assert list(mine) == [0x3F80, 0x3F82, 0xBF80, 0xBF82, 0x3F81, 0x3F80]


def test_bf16_roundtrip_exact():
    b = synth.to_bf16_bits(synth.normal(0, 12, (4096,)))
    assert np.array_equal(synth.to_bf16_bits(synth.bf16_bits_to_f32(b)), b)
