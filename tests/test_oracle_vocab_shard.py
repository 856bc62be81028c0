"""Pins of ``oracle.vocab_shard_stats`` (one vocabulary shard's share of the
log-softmax normaliser of Sec. 3.1, Eq. 3): merging the shards' (max, sum)
pairs by the log-sum-exp rule gives ``scipy.special.logsumexp`` of the whole
row for any split, exactly one shard owns each token and reports its logit,
and excluded rows report nothing."""
import numpy as np
import pytest
from scipy.special import logsumexp

import oracle


def _merge(parts):
    m = np.max([p[0] for p in parts], axis=0)
    s = sum(p[1] * np.exp2(p[0] - m) for p in parts)
    return np.log(2.0) * (m + np.log2(s))


@pytest.mark.parametrize("splits", [[0, 7], [0, 3, 7], [0, 1, 2, 6, 7], [0, 5, 6, 7]])
@pytest.mark.parametrize("inv_temp", [1.0, 0.6])
def test_shard_merge_equals_full_logsumexp(splits, inv_temp):
    rng = np.random.default_rng(11)
    N, V = 6, 7
    x = rng.normal(0.0, 3.0, (N, V))
    x[2, 4] = -np.inf  # a -inf column inside one shard
    y = rng.integers(0, V, N).astype(np.int32)
    parts = []
    for a, b in zip(splits, splits[1:]):
        parts.append(oracle.vocab_shard_stats(x[:, a:b], a, y, inv_temp=inv_temp))
    lse = _merge(parts)
    np.testing.assert_allclose(lse, logsumexp(inv_temp * x, axis=1), rtol=1e-14, atol=1e-14)
    owners = sum(p[3] for p in parts)
    assert np.all(owners == 1)
    zy = sum(p[2] for p in parts)
    np.testing.assert_array_equal(zy, x[np.arange(N), y])


def test_excluded_and_all_minus_inf_rows():
    x = np.array([[1.0, 2.0, 3.0], [-np.inf, -np.inf, -np.inf], [0.5, 0.5, 0.5]])
    y = np.array([1, 0, 5], np.int32)
    m2, s, zy, owned = oracle.vocab_shard_stats(x, 0, y, w=np.array([0.0, 1.0, 1.0]))
    assert m2[0] == -np.inf and s[0] == 0 and owned[0] == 1 and zy[0] == 0.0  # not read
    assert m2[1] == -np.inf and s[1] == 0
    assert owned[2] == 0 and zy[2] == 0
    # a uniform row: s = V exactly
    assert s[2] == 3.0 and m2[2] == pytest.approx(0.5 * np.log2(np.e), rel=1e-15)
