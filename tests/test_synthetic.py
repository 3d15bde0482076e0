"""The seeded input generator is deterministic and produces the workloads' shapes."""
import numpy as np

from paper_1711_10275_amd import synthetic as S


def test_shell_32_shape_and_determinism():
    a, b = S.shell_32(), S.shell_32()
    np.testing.assert_array_equal(a, b)
    assert 1500 < a.shape[0] < 2200 and a.dtype == np.int32
    assert np.all(a[:, 1:] >= 0) and np.all(a[:, 1:] < 32)
    # sorted, unique rows
    assert np.all(np.diff(a[:, 1] * 1024 + a[:, 2] * 32 + a[:, 3]) > 0)


def test_bf16_round_properties():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 0.0, 3.0e38], np.float32)
    r = S.bf16_round(x)
    assert r[0] == 1.0 and r[1] == 1.0          # tie to even (down)
    assert r[2] == np.float32(1.0 + 4 * 2 ** -8)  # tie to even (up)
    assert r[3] == -2.5 and r[4] == 0.0
    assert np.all((r.view(np.uint32) & 0xFFFF) == 0)


def test_features_and_weights_seeded():
    np.testing.assert_array_equal(S.features(10, 4, 1), S.features(10, 4, 1))
    w = S.weights(27, 64, 64, 3001)
    assert w.shape == (27, 64, 64) and abs(w.std() - 1 / np.sqrt(27 * 64)) < 1e-3
