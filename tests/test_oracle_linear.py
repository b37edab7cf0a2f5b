"""The projection oracle pinned against pure-Python loops and closed forms."""
import numpy as np
import pytest

from oracle import linear as ol


def _loops(x, w):
    m, k = x.shape
    n = w.shape[0]
    out = np.zeros((m, n))
    for i in range(m):
        for j in range(n):
            acc = 0.0
            for l in range(k):
                acc += float(x[i, l]) * float(w[j, l])
            out[i, j] = acc
    return out


@pytest.mark.parametrize("m,n,k", [(1, 1, 1), (3, 5, 7), (8, 4, 16), (2, 9, 33)])
def test_linear_equals_loops(m, n, k):
    rng = np.random.default_rng(m * 100 + n * 10 + k)
    x = rng.standard_normal((m, k))
    w = rng.standard_normal((n, k))
    assert np.allclose(ol.linear(x, w), _loops(x, w), rtol=0, atol=1e-12)


def test_linear_closed_forms():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((6, 8))
    # identity weight copies the tokens; a one-hot row selects one input feature
    assert np.array_equal(ol.linear(x, np.eye(8)), x)
    w = np.zeros((3, 8))
    w[0, 5] = 1.0
    w[2, 0] = -2.0
    out = ol.linear(x, w)
    assert np.array_equal(out[:, 0], x[:, 5]) and np.array_equal(out[:, 2], -2.0 * x[:, 0])
    assert not out[:, 1].any()
    # the weight is [n][k]: a transposed weight gives a different result
    w2 = rng.standard_normal((8, 8))
    assert not np.allclose(ol.linear(x, w2), x @ w2)


def test_linear_rejects_mismatched_shapes():
    with pytest.raises(ValueError):
        ol.linear(np.zeros((2, 3)), np.zeros((4, 5)))
