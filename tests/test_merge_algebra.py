"""The decomposition the GPU path relies on (Section 2's statistics built
from per-vocabulary-tile partials): per tile the maximum m_j, its lowest
index, s_j = sum e^(z - m_j) and t_j = sum e^(z - m_j)(z - m_j); merged over
tiles by rebasing to the common maximum,
    m = max m_j,  s = sum s_j e^(m_j - m),
    t = sum e^(m_j - m) (t_j + (m_j - m) s_j),
gives conf = 1/s, entropy = log s - t/s, log q = -log s, lse = m + log s.
Checked in binary64 against the oracle's two-pass statistics for random
vocabulary splits and merge orders (CPU only)."""
import numpy as np
import pytest

import oracle


def _partial(z, v0):
    m = z.max()
    idx = v0 + int(np.argmax(z))          # numpy returns the first maximum
    e = np.exp(z - m)
    return m, e.sum(), (e * (z - m)).sum(), idx


def _merge(a, b):
    m = max(a[0], b[0])
    ea, eb = np.exp(a[0] - m), np.exp(b[0] - m)
    s = a[1] * ea + b[1] * eb
    t = ea * (a[2] + (a[0] - m) * a[1]) + eb * (b[2] + (b[0] - m) * b[1])
    if a[0] > b[0] or (a[0] == b[0] and a[3] < b[3]):
        idx = a[3]
    else:
        idx = b[3]
    return m, s, t, idx


@pytest.mark.parametrize("seed", range(8))
def test_tile_merge_reproduces_oracle_statistics(seed):
    rng = np.random.default_rng(seed)
    d, V = 16, int(rng.integers(2, 3000))
    h = (rng.standard_normal((3, d)) * rng.uniform(0.1, 4)).astype(np.float32)
    W = rng.standard_normal((V, d)).astype(np.float32)
    if seed % 2:
        W[rng.integers(0, V, 5)] = W[0]        # exact ties across tiles
    ref = oracle.row_stats(h, W)
    z = h.astype(np.float64) @ W.astype(np.float64).T
    for r in range(3):
        cuts = np.sort(rng.choice(np.arange(1, V), size=min(V - 1, int(rng.integers(1, 12))),
                                  replace=False)) if V > 1 else np.array([], int)
        bounds = np.concatenate([[0], cuts, [V]])
        parts = [_partial(z[r, a:b], a) for a, b in zip(bounds[:-1], bounds[1:])]
        order = rng.permutation(len(parts))
        acc = parts[order[0]]
        for j in order[1:]:
            acc = _merge(acc, parts[j])
        m, s, t, idx = acc
        assert idx == ref["argmax"][r]
        np.testing.assert_allclose(1.0 / s, ref["conf"][r], rtol=1e-12)
        np.testing.assert_allclose(np.log(s) - t / s, ref["entropy"][r], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(-np.log(s), ref["logp"][r], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(m + np.log(s), ref["lse"][r], rtol=1e-12)
