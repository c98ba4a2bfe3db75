"""Pins for the oracle's candidate confidence features (implementation appendix: five scalars
per candidate read from the drafter's distribution at its slot), CPU only.

feat = (logp, p, gap to the slot's most likely token, rank in [0, 1], top-choice indicator).
Checked against what the definitions fix independently of the formula: the probabilities of a
full top-K (K = V) sum to 1 and are the softmax of the row; gaps are zero for rank 0 and for exact
ties with the top, non-decreasing down the sorted list, and equal log-odds against the top; the
rank feature is 0 at the top and 1 at the bottom with equal steps; the indicator is one-hot on
rank 0; K = 1 gives (logp, p, 0, 0, 1). Inputs come from the oracle's own top-K on logits.
"""
import numpy as np
import pytest
from scipy.special import softmax

import oracle


def _topk(rng, rows, V, K, ties=False):
    x = (rng.standard_normal((1, rows, V)) * 2).astype(np.float32)
    if ties:  # ids 0..3 share the row's largest value
        x[..., 0] = x.max(-1) + 1.0
        x[..., 1:4] = x[..., :1]
    return oracle.topk(x, K), x


def test_full_distribution_probabilities_and_softmax():
    rng = np.random.default_rng(1)
    (ids, logp), x = _topk(rng, 6, 40, 40)
    f = oracle.candidate_features(logp)
    assert np.allclose(f[..., 1].sum(-1), 1.0, atol=1e-6)
    sm = softmax(x.astype(np.float64), axis=-1)
    assert np.allclose(f[..., 1], np.take_along_axis(sm, ids.astype(np.int64), -1), rtol=1e-6)
    assert np.array_equal(f[..., 0], logp)


@pytest.mark.parametrize("K", [2, 5, 16, 64])
def test_gap_rank_indicator(K):
    rng = np.random.default_rng(K)
    (ids, logp), x = _topk(rng, 9, 300, K, ties=True)
    f = oracle.candidate_features(logp)
    gap, rank, top = f[..., 2], f[..., 3], f[..., 4]
    assert (gap[..., 0] == 0).all() and (gap >= 0).all()
    assert (np.diff(gap, axis=-1) >= 0).all()                 # sorted list: gaps only grow
    # the gap is the log-odds of the top candidate against this one: log(p_top / p_k)
    assert np.allclose(gap, np.log(f[..., :1, 1].astype(np.float64) / f[..., 1]), atol=2e-5)
    # exact ties with the top (planted at ids 0..3, the first four ranks) have zero gap
    assert (ids[..., :min(K, 4)] == np.arange(min(K, 4))).all()
    assert (gap[..., :4] == 0).all() and (K <= 4 or (gap[..., 4] > 0).all())
    assert (rank[..., 0] == 0).all() and np.allclose(rank[..., -1], 1.0)
    assert np.allclose(np.diff(rank, axis=-1), 1.0 / (K - 1))
    assert (top[..., 0] == 1).all() and (top[..., 1:] == 0).all()


def test_single_candidate():
    logp = np.array([[[-0.25]], [[-3.0]]], np.float32)
    f = oracle.candidate_features(logp)
    assert np.allclose(f[:, 0, 0], [[-0.25, np.exp(-0.25), 0, 0, 1], [-3.0, np.exp(-3.0), 0, 0, 1]])
