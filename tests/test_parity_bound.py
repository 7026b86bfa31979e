"""The fast evaluation of the T2' bound (prefix sums for the term every key shares,
significant keys only for the rest) against the plain sum over every key."""
import numpy as np

from parity import _abs_dev_sums, _weighted_abs_dev


def direct(A, z, v, o):
    e = A + z[:, None]
    return np.stack([np.einsum("rj,rj->r", e, np.abs(v[None, :, c] - o[:, c][:, None])) for c in range(v.shape[1])],
                    axis=1)


def test_abs_dev_sums_equal_the_plain_sum():
    rng = np.random.default_rng(90)
    v = rng.standard_normal((1000, 7))
    o = np.vstack([rng.standard_normal((5, 7)) * 3, v[:2]])      # queries inside, outside and on the values
    want = np.abs(v[None, :, :] - o[:, None, :]).sum(axis=1)
    assert np.allclose(_abs_dev_sums(v, o), want, rtol=1e-12, atol=1e-9)


def test_weighted_sum_is_an_upper_bound_within_1e9():
    rng = np.random.default_rng(91)
    for sharp in (0.1, 5.0, 60.0):        # diffuse rows, sharp rows, rows with most weights negligible
        logits = rng.standard_normal((6, 3000)) * sharp
        A = np.exp2(logits - logits.max(axis=1, keepdims=True) + 8.0) * 0.07
        z = np.full(6, 2.0 ** -10)
        v = rng.standard_normal((3000, 5))
        o = rng.standard_normal((6, 5))
        got, want = _weighted_abs_dev(A, z, v, o), direct(A, z, v, o)
        assert np.all(got >= want * (1 - 1e-12)), sharp
        assert np.all(got <= want * (1 + 1e-8)), (sharp, (got / want).max())
