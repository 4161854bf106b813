"""Pins of oracle.toy_gradient, the gradient of Appendix B's diagnostic loss
(1/B) sum over B sampled entries of c_i (w_i - w*_i)^4 (CPU)."""
import numpy as np

import oracle


def setup(seed, n=257, batch=400):
    rng = np.random.default_rng(seed)
    w = rng.normal(0, 1, n).astype(np.float32)
    t = rng.normal(0, 1, n).astype(np.float32)
    c = (10.0 ** rng.uniform(-3, 3, n)).astype(np.float32)
    idx = rng.integers(0, n, batch)
    return w, t, c, idx, batch


def loss(w, t, c, idx, batch):
    """The sampled loss in fp64, summed over the samples themselves."""
    w, t, c = (np.asarray(a, np.float64) for a in (w, t, c))
    return float(np.sum(c[idx] * (w[idx] - t[idx]) ** 4) / batch)


def test_matches_the_fp64_derivative_within_fp32_rounding():
    for seed in range(5):
        w, t, c, idx, b = setup(seed)
        g = oracle.toy_gradient(w, t, c, idx, b).astype(np.float64)
        cnt = np.array([np.sum(idx == i) for i in range(w.size)], np.float64)   # brute force
        ref = 4.0 / b * cnt * c.astype(np.float64) * (w.astype(np.float64) - t) ** 3
        # six fp32 roundings (d, 4/B, two products forming s, three by d)
        assert np.all(np.abs(g - ref) <= 8 * 2.0 ** -24 * np.abs(ref) + 1e-300)
        assert np.all((g == 0) == (cnt == 0) | (w == t))


def test_is_the_gradient_of_the_sampled_loss():
    w, t, c, idx, b = setup(11, n=64, batch=100)
    g = oracle.toy_gradient(w, t, c, idx, b).astype(np.float64)
    h = 1e-5
    for i in range(0, 64, 7):
        wp, wm = w.astype(np.float64).copy(), w.astype(np.float64).copy()
        wp[i] += h
        wm[i] -= h
        fd = (loss(wp, t, c, idx, b) - loss(wm, t, c, idx, b)) / (2 * h)
        assert abs(fd - g[i]) <= 1e-4 * max(1.0, abs(fd)), (i, fd, g[i])


def test_unsampled_entries_and_out_of_range_samples():
    w, t, c, _, b = setup(3, n=16, batch=4)
    g = oracle.toy_gradient(w, t, c, np.array([2, 2, 5, 99]), 4)
    assert np.count_nonzero(g) == 2 and g[2] != 0 and g[5] != 0
    assert np.float32(g[2]) == np.float32(2 * g[2] / 2)
    # an entry drawn twice weighs twice an entry drawn once (same d, c)
    w2, t2, c2 = np.zeros(4, np.float32), -np.ones(4, np.float32), np.ones(4, np.float32)
    g2 = oracle.toy_gradient(w2, t2, c2, np.array([0, 0, 1]), 3)
    assert g2[0] == 2 * g2[1] and g2[1] == np.float32(4.0 / 3) and g2[2] == 0
