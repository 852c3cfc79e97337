"""Host-side token-selection rules (the strategy comparison of Table 3)
that hand given rows to the step: random and token-type selection."""
import numpy as np
import pytest

from paper_2503_12450_amd import selection as SEL


def _valid(rows, n_slots, seq, n):
    assert rows.shape == (n_slots, n) and rows.dtype == np.int32
    for r in rows:
        assert np.all(np.diff(r) > 0)
        assert r.size == 0 or (r[0] >= 0 and r[-1] < seq)


@pytest.mark.parametrize("n", [0, 1, 37, 320])
def test_random_rows_are_valid_and_seeded(n):
    a = SEL.random_rows(5, 320, n, np.random.default_rng(7))
    b = SEL.random_rows(5, 320, n, np.random.default_rng(7))
    _valid(a, 5, 320, n)
    np.testing.assert_array_equal(a, b)


def test_random_rows_cover_tokens_uniformly():
    # every token is picked about n / seq of the time over many slots
    rows = SEL.random_rows(4000, 20, 5, np.random.default_rng(3))
    counts = np.bincount(rows.reshape(-1), minlength=20)
    expected = 4000 * 5 / 20
    assert np.all(np.abs(counts - expected) < 6 * np.sqrt(expected))


def test_observation_rows_type_first_then_fill():
    decoded = np.zeros((3, 10), dtype=bool)
    decoded[0, [1, 4, 7]] = True          # fewer decoded tokens than n
    decoded[1, :] = True                  # all decoded
    decoded[2, [0, 2, 3, 5, 6, 8]] = True  # more decoded than n
    n = 4
    d = SEL.observation_rows(decoded, n, SEL.COMPUTE_DECODED)
    np.testing.assert_array_equal(d[0], [0, 1, 4, 7])   # 1, 4, 7 then the lowest undecoded
    np.testing.assert_array_equal(d[1], [0, 1, 2, 3])
    np.testing.assert_array_equal(d[2], [0, 2, 3, 5])
    u = SEL.observation_rows(decoded, n, SEL.COMPUTE_UNDECODED)
    np.testing.assert_array_equal(u[0], [0, 2, 3, 5])
    np.testing.assert_array_equal(u[1], [0, 1, 2, 3])   # no undecoded token: lowest decoded
    np.testing.assert_array_equal(u[2], [1, 4, 7, 9])
    for rows in (d, u):
        _valid(rows, 3, 10, n)


def test_observation_rows_complement():
    rng = np.random.default_rng(5)
    decoded = rng.random((6, 64)) < 0.4
    k = decoded.sum(axis=1)
    for b in range(6):
        d = SEL.observation_rows(decoded[b:b + 1], int(k[b]), SEL.COMPUTE_DECODED)[0]
        np.testing.assert_array_equal(d, np.flatnonzero(decoded[b]))
        u = SEL.observation_rows(decoded[b:b + 1], 64 - int(k[b]), SEL.COMPUTE_UNDECODED)[0]
        np.testing.assert_array_equal(u, np.flatnonzero(~decoded[b]))


def test_rules_reject_bad_arguments():
    with pytest.raises(ValueError):
        SEL.random_rows(2, 10, 11, np.random.default_rng(0))
    with pytest.raises(ValueError):
        SEL.observation_rows(np.zeros((2, 10), bool), 3, "predicted")
    with pytest.raises(ValueError):
        SEL.observation_rows(np.zeros(10, bool), 3, SEL.COMPUTE_DECODED)
