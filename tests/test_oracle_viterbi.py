"""Pins for the oracle's exact max-path decode (decode-rule appendix, Eq. pathscore), CPU only.

The path score g(c) sums the matching terms of adjacent slots (plus the anchor term); the exact
decode returns its maximiser, found by dynamic programming. Checked against enumeration of all
K^B paths (with the tie rule: among maximising paths, the smallest read from the last slot
backwards), the hand-worked greedy-versus-best example of tests/golden/walk_hand_cases.yaml,
the greedy walk (never better), and special cases (B = 1, K = 1, a planted chain, no anchor
equals an all-zero anchor). logq along the path is checked against scipy's logsumexp.
"""
import itertools
import os

import numpy as np
import pytest
import yaml
from scipy.special import logsumexp

import oracle


def _g(S, S0, logp, lam, n, path):
    """Path score in fp64."""
    K = logp.shape[-1]
    g = float(S0[n, path[0]]) if S0 is not None else 0.0
    g += lam * float(logp[n, 0, path[0]])
    for t in range(1, len(path)):
        g += float(S[n, t - 1, path[t - 1], path[t]]) + lam * float(logp[n, t, path[t]])
    return g


def _brute_force(S, S0, logp, lam, n):
    """Every path scored exactly; the maximisers, and the one the tie rule selects."""
    B, K = logp.shape[1], logp.shape[2]
    scored = [(_g(S, S0, logp, lam, n, p), p) for p in itertools.product(range(K), repeat=B)]
    gmax = max(g for g, _ in scored)
    best = [p for g, p in scored if g == gmax]
    return gmax, min(best, key=lambda p: tuple(reversed(p))), scored


def _inputs(rng, N, B, K, anchor, coarse):
    if coarse:  # small integers: exact in float and double, frequent exact ties
        S = rng.integers(-3, 4, size=(N, B - 1, K, K)).astype(np.float32)
        S0 = rng.integers(-3, 4, size=(N, K)).astype(np.float32) if anchor else None
        logp = -rng.integers(0, 4, size=(N, B, K)).astype(np.float32)
    else:
        S = (rng.standard_normal((N, B - 1, K, K)) * 3).astype(np.float32)
        S0 = rng.standard_normal((N, K)).astype(np.float32) if anchor else None
        logp = -np.sort(rng.random((N, B, K)) * 4, axis=-1).astype(np.float32)
    ids = rng.integers(0, 10 ** 5, size=(N, B, K)).astype(np.int32)
    return S, S0, logp, ids


@pytest.mark.parametrize("seed", range(16))
def test_exact_decode_equals_brute_force_with_ties(seed):
    rng = np.random.default_rng(100 + seed)
    N, B, K = 2, int(rng.integers(1, 6)), int(rng.integers(1, 5))
    lam = 1.0 if seed % 4 == 3 else 0.0
    S, S0, logp, ids = _inputs(rng, N, B, K, anchor=seed % 2 == 1, coarse=True)
    draft, choice, logq, score = oracle.viterbi_walk(S, S0, logp, ids, lam)
    for n in range(N):
        gmax, path, _ = _brute_force(S, S0, logp, lam, n)
        assert tuple(choice[n]) == path, (seed, n, choice[n], path)
        assert float(score[n]) == gmax
        assert list(draft[n]) == [ids[n, t, c] for t, c in enumerate(path)]


@pytest.mark.parametrize("seed", range(8))
def test_exact_decode_real_scores(seed):
    rng = np.random.default_rng(200 + seed)
    N, B, K = 3, int(rng.integers(2, 6)), int(rng.integers(2, 5))
    S, S0, logp, ids = _inputs(rng, N, B, K, anchor=seed % 2 == 0, coarse=False)
    draft, choice, logq, score = oracle.viterbi_walk(S, S0, logp, ids)
    for n in range(N):
        gmax, path, scored = _brute_force(S, S0, logp, 0.0, n)
        assert abs(float(score[n]) - gmax) <= 1e-5 * max(1.0, abs(gmax))
        assert abs(_g(S, S0, logp, 0.0, n, tuple(choice[n])) - gmax) <= 1e-5 * max(1.0, abs(gmax))
        margin = gmax - max([g for g, p in scored if p != path], default=-np.inf)
        if margin > 1e-4:  # no float near-tie: the path itself is unique
            assert tuple(choice[n]) == path


@pytest.mark.parametrize("seed", range(6))
def test_greedy_never_beats_exact(seed):
    rng = np.random.default_rng(300 + seed)
    N, B, K = 4, 6, 4
    S, S0, logp, ids = _inputs(rng, N, B, K, anchor=True, coarse=False)
    _, gc, _ = oracle.greedy_walk(S, S0, logp, ids)
    _, vc, _, score = oracle.viterbi_walk(S, S0, logp, ids)
    for n in range(N):
        assert _g(S, S0, logp, 0.0, n, gc[n]) <= _g(S, S0, logp, 0.0, n, vc[n]) + 1e-5


def test_hand_case_greedy_versus_best(golden_dir):
    cases = yaml.safe_load(open(os.path.join(golden_dir, "walk_hand_cases.yaml")))["cases"]
    c = next(c for c in cases if "best_path" in c)
    S = np.array(c["S"], np.float32)[None]
    S0 = np.array(c["S0"], np.float32)[None]
    B, K = S.shape[1] + 1, S.shape[-1]
    ids = np.arange(B * K, dtype=np.int32).reshape(1, B, K)
    logp = np.zeros((1, B, K), np.float32)
    _, gchoice, _ = oracle.greedy_walk(S, S0, logp, ids)
    _, choice, _, score = oracle.viterbi_walk(S, S0, logp, ids)
    assert gchoice[0].tolist() == c["choice"]
    assert choice[0].tolist() == c["best_path"]
    assert abs(float(score[0]) - c["g_best"]) < 1e-6
    assert abs(_g(S, S0, logp, 0.0, 0, gchoice[0]) - c["g_greedy"]) < 1e-6


def test_logq_along_the_path():
    rng = np.random.default_rng(7)
    N, B, K = 3, 5, 6
    S, S0, logp, ids = _inputs(rng, N, B, K, anchor=True, coarse=False)
    lam = 0.5
    _, choice, logq, _ = oracle.viterbi_walk(S, S0, logp, ids, lam)
    for n in range(N):
        for t in range(B):
            pair = S0[n] if t == 0 else S[n, t - 1, choice[n, t - 1]]
            # node scores in float (the product of two floats is exact in double)
            z = (np.float64(lam) * logp[n, t].astype(np.float64) + pair.astype(np.float64))
            z = z.astype(np.float32).astype(np.float64)
            expect = z[choice[n, t]] - logsumexp(z)
            assert abs(logq[n, t] - expect) <= 1e-5 * max(1.0, abs(expect))


def test_special_cases():
    rng = np.random.default_rng(11)
    # B = 1: slot 0 alone, decided by the anchor scores (all zero without an anchor -> 0)
    S = np.zeros((2, 0, 3, 3), np.float32)
    S0 = np.array([[0.1, 0.7, 0.7], [-1.0, -2.0, -0.5]], np.float32)
    logp = np.zeros((2, 1, 3), np.float32)
    ids = np.arange(6, dtype=np.int32).reshape(2, 1, 3)
    assert oracle.viterbi_walk(S, S0, logp, ids)[1][:, 0].tolist() == [1, 2]
    assert oracle.viterbi_walk(S, None, logp, ids)[1][:, 0].tolist() == [0, 0]
    # K = 1: the only path
    S1, S01, logp1, ids1 = _inputs(rng, 2, 5, 1, anchor=True, coarse=False)
    assert (oracle.viterbi_walk(S1, S01, logp1, ids1)[1] == 0).all()
    # a planted chain with the top score on every one of its links is the best path
    N, B, K = 2, 7, 5
    S, _, logp, ids = _inputs(rng, N, B, K, anchor=False, coarse=False)
    S = np.clip(S, -7.0, 7.0)
    chain = rng.integers(0, K, size=(N, B))
    for n in range(N):
        for t in range(B - 1):
            S[n, t, chain[n, t], chain[n, t + 1]] = 8.0
    assert (oracle.viterbi_walk(S, None, logp, ids)[1] == chain).all()
    # no anchor is the same as an all-zero anchor
    S, S0, logp, ids = _inputs(rng, 3, 4, 3, anchor=True, coarse=True)
    a = oracle.viterbi_walk(S, None, logp, ids)
    b = oracle.viterbi_walk(S, np.zeros_like(S0), logp, ids)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
