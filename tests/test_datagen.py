"""The seeded input generator (CPU only)."""
import numpy as np

import datagen


def test_splitmix64_published_outputs():
    # First outputs of SplitMix64 for two seeds, as printed by the reference splitmix64.c.
    assert datagen.splitmix64_int(1234567, 5) == [
        6457827717110365317, 3203168211198807973, 9817491932198370423,
        4593380528125082431, 16408922859458223821]
    assert datagen.splitmix64_int(0, 2) == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4]


def test_vector_stream_matches_scalar_generator():
    start = datagen.stream_start(7, 1)
    z = datagen.raw_stream(7, 1, 1000, chunk=97)
    assert [int(v) for v in z] == datagen.splitmix64_int(start, 1000)


def test_uniform_range_grid_and_determinism():
    a = datagen.draw(5, 0, (1000, 7))
    b = datagen.draw(5, 0, (1000, 7))
    np.testing.assert_array_equal(a, b)
    assert a.min() >= -1.0 and a.max() < 1.0
    grid = a.astype(np.float64) * 2 ** 23
    np.testing.assert_array_equal(grid, np.round(grid))
    assert abs(a.mean()) < 0.02 and abs(a.std() - 1 / np.sqrt(3)) < 0.01
    assert not np.array_equal(a, datagen.draw(5, 1, (1000, 7)))
    assert not np.array_equal(a, datagen.draw(6, 0, (1000, 7)))


def test_integer_mode():
    v = datagen.draw(3, 0, (50000,), "integer")
    assert set(np.unique(v).tolist()) == set(range(-4, 5))


def test_bf16_rounding_matches_torch():
    import torch
    a = datagen.draw(9, 0, (100000,)) * np.float32(37.0)
    a = np.concatenate([a, np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8,
                                     0.0, -0.0], np.float32)])
    ours = datagen.bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    r = datagen.round_bf16(a)
    np.testing.assert_array_equal(datagen.round_bf16(r), r)


def test_config2_weight_scale():
    cs = datagen.CONFIGS["cfg2"]
    x, w, b = datagen.make_inputs(cs)
    assert np.abs(w).max() <= 1.0 / 24 + 1e-9
    raw = datagen.draw(cs.seed, 1, cs.w_shape())
    np.testing.assert_array_equal(w, (raw.astype(np.float64) / 24.0).astype(np.float32))
