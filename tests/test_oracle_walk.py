"""Pins for the oracle's step 4 (greedy walk + local log-likelihood), CPU only.

The greedy rule of Sec. 3.5 commits, left to right, the candidate that maximises the matching
term with the candidate just committed; Eq. (localar) normalises those terms with a softmax
over the K candidates of the slot. Checked against brute-force enumeration of all K^B paths,
the hand-worked fixtures in tests/golden/walk_hand_cases.yaml (including Fig. 1) and special
cases (K = 1, uniform scores, a planted chain).
"""
import itertools
import math
import os

import numpy as np
import pytest
import yaml
from scipy.special import logsumexp

import oracle


def _node_scores(S, S0, logp, lam, n, path):
    """z_t[k] for every slot t along `path` (float32, one rounding, as the walk decides)."""
    B = len(path)
    K = logp.shape[-1]
    zs = []
    for t in range(B):
        if t == 0:
            pair = S0[n] if S0 is not None else np.zeros(K, np.float32)
        else:
            pair = S[n, t - 1, path[t - 1]]
        z = (pair.astype(np.float64) + np.float64(lam) * logp[n, t].astype(np.float64)).astype(np.float32)
        zs.append(z)
    return zs


def _brute_force_greedy(S, S0, logp, n, lam=0.0):
    """Greedy path characterised without a sequential walk: among all K^B paths, the
    lexicographic maximum of ((z_0[c_0], -c_0), (z_1[c_1], -c_1), ...)."""
    K = logp.shape[-1]
    B = logp.shape[1]
    best, best_key = None, None
    for path in itertools.product(range(K), repeat=B):
        zs = _node_scores(S, S0, logp, lam, n, path)
        key = tuple(x for t in range(B) for x in (float(zs[t][path[t]]), -path[t]))
        if best_key is None or key > best_key:
            best, best_key = path, key
    return list(best)


@pytest.mark.parametrize("seed", range(12))
def test_greedy_equals_brute_force_lexicographic_max(seed):
    rng = np.random.default_rng(seed)
    N, B, K = 2, int(rng.integers(2, 6)), int(rng.integers(1, 5))
    # coarse values -> frequent exact ties
    S = rng.integers(-3, 4, size=(N, B - 1, K, K)).astype(np.float32) * 0.5
    S0 = rng.integers(-3, 4, size=(N, K)).astype(np.float32) if seed % 2 else None
    logp = -np.sort(rng.random((N, B, K)), axis=-1).astype(np.float32)
    ids = rng.integers(0, 1000, size=(N, B, K)).astype(np.int32)
    draft, choice, logq = oracle.greedy_walk(S, S0, logp, ids)
    for n in range(N):
        assert choice[n].tolist() == _brute_force_greedy(S, S0, logp, n)
        np.testing.assert_array_equal(draft[n], ids[n, np.arange(B), choice[n]])


@pytest.mark.parametrize("seed", range(4))
def test_logq_is_the_local_log_softmax(seed):
    rng = np.random.default_rng(100 + seed)
    N, B, K = 3, 6, 5
    S = (rng.standard_normal((N, B - 1, K, K)) * 3).astype(np.float32)
    S0 = (rng.standard_normal((N, K)) * 3).astype(np.float32)
    logp = -rng.random((N, B, K)).astype(np.float32)
    ids = rng.integers(0, 50, size=(N, B, K)).astype(np.int32)
    draft, choice, logq = oracle.greedy_walk(S, S0, logp, ids)
    for n in range(N):
        zs = _node_scores(S, S0, logp, 0.0, n, choice[n])
        for t in range(B):
            z = zs[t].astype(np.float64)
            assert choice[n, t] == int(np.argmax(z))
            np.testing.assert_allclose(logq[n, t], z[choice[n, t]] - logsumexp(z), atol=1e-6)


def test_hand_cases(golden_dir):
    cases = yaml.safe_load(open(os.path.join(golden_dir, "walk_hand_cases.yaml")))["cases"]
    for c in cases:
        S = np.array(c["S"], np.float32)[None]
        B = S.shape[1] + 1
        K = S.shape[-1]
        S0 = None if c["S0"] is None else np.array(c["S0"], np.float32)[None]
        ids = np.array(c.get("ids", np.arange(B * K).reshape(B, K)), np.int32)[None]
        logp = np.zeros((1, B, K), np.float32)
        draft, choice, logq = oracle.greedy_walk(S, S0, logp, ids)
        assert choice[0].tolist() == c["choice"], c["name"]
        if "draft" in c:
            assert draft[0].tolist() == c["draft"], c["name"]
        if "logq" in c:
            np.testing.assert_allclose(logq[0], c["logq"], rtol=0, atol=1e-7, err_msg=c["name"])
        if "logq0" in c:
            np.testing.assert_allclose(logq[0, 0], c["logq0"], rtol=0, atol=1e-7, err_msg=c["name"])
        if "g_greedy" in c:
            path = choice[0]
            g = float(S0[0, path[0]]) + sum(float(S[0, t - 1, path[t - 1], path[t]]) for t in range(1, B))
            assert abs(g - c["g_greedy"]) < 1e-6
            # the best-scoring path is strictly better, and greedy did not find it
            best = max(itertools.product(range(K), repeat=B),
                       key=lambda p: float(S0[0, p[0]]) + sum(float(S[0, t - 1, p[t - 1], p[t]]) for t in range(1, B)))
            gb = float(S0[0, best[0]]) + sum(float(S[0, t - 1, best[t - 1], best[t]]) for t in range(1, B))
            assert list(best) == c["best_path"] and abs(gb - c["g_best"]) < 1e-6 and gb > g


def test_single_candidate_and_uniform_scores_reduce_to_drafter_argmax():
    rng = np.random.default_rng(5)
    N, B = 3, 7
    ids = rng.integers(0, 100, size=(N, B, 1)).astype(np.int32)
    draft, choice, logq = oracle.greedy_walk(np.zeros((N, B - 1, 1, 1), np.float32), None,
                                             np.zeros((N, B, 1), np.float32), ids)
    np.testing.assert_array_equal(draft, ids[..., 0])
    assert (logq == 0).all()
    K = 6
    ids = rng.integers(0, 100, size=(N, B, K)).astype(np.int32)
    S = np.full((N, B - 1, K, K), 2.5, np.float32)
    draft, choice, logq = oracle.greedy_walk(S, None, np.zeros((N, B, K), np.float32), ids)
    np.testing.assert_array_equal(draft, ids[..., 0])  # vanilla per-slot argmax
    np.testing.assert_allclose(logq, -math.log(K), atol=1e-7)


def test_planted_chain_is_recovered():
    rng = np.random.default_rng(6)
    N, B, K = 4, 9, 8
    chain = rng.integers(0, K, size=(N, B))
    S = rng.uniform(-8, 7, size=(N, B - 1, K, K)).astype(np.float32)
    S0 = rng.uniform(-8, 7, size=(N, K)).astype(np.float32)
    for n in range(N):
        S0[n, chain[n, 0]] = 8.0
        for t in range(B - 1):
            S[n, t, chain[n, t], chain[n, t + 1]] = 8.0
    ids = rng.integers(0, 1000, size=(N, B, K)).astype(np.int32)
    draft, choice, logq = oracle.greedy_walk(S, S0, np.zeros((N, B, K), np.float32), ids)
    np.testing.assert_array_equal(choice, chain)


def test_missing_anchor_equals_zero_anchor():
    rng = np.random.default_rng(7)
    N, B, K = 2, 5, 4
    S = rng.standard_normal((N, B - 1, K, K)).astype(np.float32)
    logp = -rng.random((N, B, K)).astype(np.float32)
    ids = rng.integers(0, 9, size=(N, B, K)).astype(np.int32)
    a = oracle.greedy_walk(S, None, logp, ids, logp_weight=0.7)
    b = oracle.greedy_walk(S, np.zeros((N, K), np.float32), logp, ids, logp_weight=0.7)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


def test_logp_weight_enters_node_scores():
    # lambda = 1 with dyadic values (exact in float): z = S + logp decides
    N, B, K = 1, 2, 3
    S = np.array([[[[1.0, 1.25, 1.5], [0, 0, 0], [0, 0, 0]]]], np.float32)
    logp = np.array([[[0.0, -1.0, -2.0], [-0.5, -0.5, -0.75]]], np.float32)
    ids = np.arange(6, dtype=np.int32).reshape(1, 2, 3)
    _, choice, _ = oracle.greedy_walk(S, None, logp, ids, logp_weight=0.0)
    assert choice[0].tolist() == [0, 2]
    _, choice, logq = oracle.greedy_walk(S, None, logp, ids, logp_weight=1.0)
    assert choice[0].tolist() == [0, 1]  # z = [0.5, 0.75, 0.75] -> tie to the lower index
    np.testing.assert_allclose(logq[0, 1], 0.75 - logsumexp([0.5, 0.75, 0.75]), atol=1e-7)
