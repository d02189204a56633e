"""The seeded input generator: determinism, key independence, chunking, casts."""
import numpy as np
import pytest

import zo_draws as zd


def test_draw_deterministic_and_keyed():
    a = zd.draw(0, "Z", (3, 1, 7), (16, 16))
    b = zd.draw(0, "Z", (3, 1, 7), (16, 16))
    np.testing.assert_array_equal(a, b)
    assert zd.sha256(a) == zd.sha256(b)
    for other in [zd.draw(1, "Z", (3, 1, 7), (16, 16)), zd.draw(0, "Z", (3, 2, 7), (16, 16)),
                  zd.draw(0, "OMEGA_U", (3, 1, 7), (16, 16))]:
        assert not np.array_equal(a, other)


def test_draw_chunked_fill_matches_definition():
    """Chunk c of the flat array is the c-th keyed stream, whatever the thread count."""
    n = zd.CHUNK * 2 + 1000
    a = zd.draw(5, "X", (2,), (n,), 0.5)
    for c in range(3):
        lo, hi = c * zd.CHUNK, min(n, (c + 1) * zd.CHUNK)
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(entropy=5, spawn_key=(zd.KIND["X"], 2, c))))
        np.testing.assert_array_equal(a[lo:hi], 0.5 * g.standard_normal(hi - lo))


def test_draw_statistics():
    a = zd.draw(0, "W0", (0,), (200000,), 0.02)
    assert abs(a.mean()) < 4 * 0.02 / np.sqrt(a.size)
    assert abs(a.std() - 0.02) < 0.02 * 4 * np.sqrt(0.5 / a.size) * 2


def test_bf16_cast_matches_torch():
    torch = pytest.importorskip("torch")
    x = zd.f32(zd.draw(0, "X", (9,), (100000,), 3.0))
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(zd.bf16_bits(x), ref)
    back = zd.bf16_to_f32(zd.bf16_bits(x))
    assert np.max(np.abs(back - x) / np.abs(x)) <= 2.0 ** -8


def test_block_roll_rows():
    x0 = np.arange(12.0).reshape(6, 2)
    xs = zd.block_roll_rows(x0, 3)
    assert xs.shape == (18, 2)
    np.testing.assert_array_equal(xs[:6], x0)
    np.testing.assert_array_equal(xs[6:12], np.roll(x0, 2, axis=0))


def test_tiny_inputs_shapes():
    d = zd.tiny_inputs(0)
    assert d["W"].shape == (256, 512) and d["W"].dtype == np.float32
    assert d["X"].shape == (64, 512)
    assert d["Ystar"].shape == (64, 256)
