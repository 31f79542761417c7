"""The seeded generator: determinism and the laws the workloads state."""
import numpy as np
import pytest

from paper_2402_09900_amd import tapes


def test_same_seed_same_bytes():
    a = tapes.make_diag(2, T=3000, d=8)
    b = tapes.make_diag(2, T=3000, d=8)
    assert tapes.flags_sha256(a.start) == tapes.flags_sha256(b.start)
    np.testing.assert_array_equal(a.x, b.x)
    np.testing.assert_array_equal(a.a, b.a)
    c = tapes.make_diag(2, seed=99, T=3000, d=8)
    assert tapes.flags_sha256(a.start) != tapes.flags_sha256(c.start)


@pytest.mark.parametrize("key", [1, 2, 4, 5])
def test_every_tape_begins_with_a_start(key):
    w = tapes.make_diag(key, B=3 if key == 4 else None, T=2048, d=4)
    assert np.all(w.start[:, 0] != 0)
    assert w.start.dtype == np.uint8


def test_episode_length_laws():
    rng = np.random.default_rng(0)
    T = 400_000
    f2 = tapes.WORKLOADS[2].episodes(np.random.Generator(np.random.PCG64(1)), T)
    lens = np.diff(np.flatnonzero(f2))
    assert abs(lens.mean() - 200) < 200 * 4 / np.sqrt(len(lens))
    f4 = tapes.WORKLOADS[4].episodes(np.random.Generator(np.random.PCG64(2)), T)
    lens = np.diff(np.flatnonzero(f4))
    assert lens.min() >= 10 and lens.max() <= 1000
    assert abs(lens.mean() - 505) < 5 * 286 / np.sqrt(len(lens))
    f5 = tapes.WORKLOADS[5].episodes(np.random.Generator(np.random.PCG64(3)), 4 * T)
    lens = np.diff(np.flatnonzero(f5))
    assert abs(np.median(lens) - np.exp(5.0)) < 0.15 * np.exp(5.0)
    f1 = tapes.WORKLOADS[1].episodes(np.random.Generator(np.random.PCG64(4)), 1024)
    assert int((f1 != 0).sum()) == 8


def test_value_ranges_and_dtypes():
    w = tapes.make_diag(4, B=2, T=500, d=16)
    assert w.a.dtype == np.uint16 and w.x.dtype == np.uint16
    a = tapes.bf16_bits_to_f32(w.a)
    assert a.min() >= 0.8 - 1e-2 and a.max() <= 1.0
    w2 = tapes.make_diag(2, T=100, d=16)
    assert w2.a.shape == (16,) and w2.a.dtype == np.complex64
    assert np.all((np.abs(w2.a) > 0.899) & (np.abs(w2.a) < 0.9991))
    w5 = tapes.make_diag(5, T=100, d=16)
    assert w5.g is not None and w5.g.shape == (1, 100, 16)
    la = tapes.make_linattn(T=256)
    assert la.q.shape == (256, 4, 64) and la.start[0] == 1


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5, 0.0,
                  np.inf, 1.0 + 2 ** -8 + 2 ** -20], dtype=np.float32)
    got = tapes.bf16_bits_to_f32(tapes.f32_to_bf16_bits(x))
    np.testing.assert_array_equal(got, np.array([1.0, 1.0, 1.0 + 2 ** -6, 1.0, -2.5, 0.0,
                                                 np.inf, 1.0 + 2 ** -7], dtype=np.float32))
    assert np.isnan(tapes.bf16_bits_to_f32(tapes.f32_to_bf16_bits(np.array([np.nan], np.float32))))[0]
