"""Pins for the oracle's exact max-path decode (decode-rule appendix, Eq. pathscore), CPU only.

The path score g(c) sums the matching terms of adjacent slots (plus the anchor term); the exact
decode returns its maximiser, found by dynamic programming. Checked against enumeration of all
K^B paths scored in exact rational arithmetic (with the tie rule: among maximising paths, the
smallest read from the last slot backwards), on integer lattices full of exact ties, on
real-valued lattices, and on real-valued lattices with planted near-ties: two paths whose exact
scores differ by about one float ulp, which a float dynamic program (written out in the test)
decides wrongly in many of the cases. Also: the hand-worked greedy-versus-best example of
tests/golden/walk_hand_cases.yaml, the greedy walk (never better), and special cases (B = 1,
K = 1, a planted chain, no anchor equals an all-zero anchor). logq along the path is checked
against scipy's logsumexp.
"""
import itertools
import os
from fractions import Fraction

import numpy as np
import pytest
import yaml
from scipy.special import logsumexp

import oracle


def _g(S, S0, logp, lam, n, path):
    """Path score in exact rational arithmetic (every float term converts exactly)."""
    F = lambda x: Fraction(float(x))
    lam = F(np.float32(lam))
    g = F(S0[n, path[0]]) if S0 is not None else Fraction(0)
    g += lam * F(logp[n, 0, path[0]])
    for t in range(1, len(path)):
        g += F(S[n, t - 1, path[t - 1], path[t]]) + lam * F(logp[n, t, path[t]])
    return g


def _brute_force(S, S0, logp, lam, n):
    """Every path scored exactly; the maximisers, and the one the tie rule selects."""
    B, K = logp.shape[1], logp.shape[2]
    scored = [(_g(S, S0, logp, lam, n, p), p) for p in itertools.product(range(K), repeat=B)]
    gmax = max(g for g, _ in scored)
    best = [p for g, p in scored if g == gmax]
    return gmax, min(best, key=lambda p: tuple(reversed(p))), scored


def _float_dp(S, S0, n, B, K):
    """A float32 dynamic program (one float rounding per addition): what a decode that sums its
    path scores in float would return. Used only to show that the planted near-ties matter."""
    f = np.float32
    best = [f(S0[n, k]) if S0 is not None else f(0) for k in range(K)]
    frm = np.zeros((B, K), np.int64)
    for t in range(1, B):
        nxt = []
        for k in range(K):
            bv, bp = f(best[0] + S[n, t - 1, 0, k]), 0
            for p in range(1, K):
                v = f(best[p] + S[n, t - 1, p, k])
                if v > bv:
                    bv, bp = v, p
            nxt.append(bv)
            frm[t, k] = bp
        best = nxt
    c = int(np.argmax(best))
    path = [c]
    for t in range(B - 1, 0, -1):
        c = int(frm[t, c])
        path.append(c)
    return tuple(reversed(path))


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
    lam = 0.75 if seed % 4 == 1 else 0.0
    S, S0, logp, ids = _inputs(rng, N, B, K, anchor=seed % 2 == 0, coarse=False)
    draft, choice, logq, score = oracle.viterbi_walk(S, S0, logp, ids, lam)
    for n in range(N):
        gmax, path, scored = _brute_force(S, S0, logp, lam, n)
        assert tuple(choice[n]) == path
        assert float(score[n]) == float(np.float32(float(gmax)))


def _plant_near_tie(rng, S, S0, n, B, K):
    """Make a runner-up path q beat the best path p* by a sliver: one link of q that p* does not
    use is set to the float that puts g(q) just above g(p*) (about one float ulp of the link).
    Returns the exact gap g(q) - g(p*) after planting, or None when no positive gap was found."""
    _, p, scored = _brute_force(S, S0, np.zeros((S.shape[0], B, K), np.float32), 0.0, n)
    gp = dict((pp, g) for g, pp in scored)[p]
    others = sorted((g, pp) for g, pp in scored if pp != p)
    q = others[-1 - int(rng.integers(0, min(3, len(others))))][1]
    links = [t for t in range(1, B) if (q[t - 1], q[t]) != (p[t - 1], p[t])]
    t = links[int(rng.integers(0, len(links)))]
    a, b = q[t - 1], q[t]
    base = S[n, t - 1, a, b]
    gq = _g(S, S0, np.zeros((S.shape[0], B, K), np.float32), 0.0, n, q)
    target = float(gp - gq) + float(base)
    best = None
    for step in range(-4, 5):
        cand = np.float32(target)
        cand = np.nextafter(cand, np.float32(np.inf if step > 0 else -np.inf)) if step else cand
        for _ in range(abs(step) - 1):
            cand = np.nextafter(cand, np.float32(np.inf if step > 0 else -np.inf))
        S[n, t - 1, a, b] = cand
        gap = _g(S, S0, np.zeros((S.shape[0], B, K), np.float32), 0.0, n, q) - gp
        if gap > 0 and (best is None or gap < best[0]):
            best = (gap, cand)
    if best is None:
        S[n, t - 1, a, b] = base
        return None
    S[n, t - 1, a, b] = best[1]
    return best[0]


@pytest.mark.parametrize("seed", range(6))
def test_exact_decode_planted_near_ties(seed):
    """Near-ties of about one float ulp: the decode must return the exact maximiser (a float
    dynamic program gets a good share of these wrong: next test)."""
    rng = np.random.default_rng(400 + seed)
    N, B, K = 8, int(rng.integers(3, 6)), int(rng.integers(2, 5))
    S, S0, logp, ids = _inputs(rng, N, B, K, anchor=seed % 2 == 0, coarse=False)
    S *= np.float32(4.0)  # path sums of tens: the float grid there is coarser than the gap
    logp[:] = 0.0
    gaps = [_plant_near_tie(rng, S, S0, n, B, K) for n in range(N)]
    assert all(g is not None for g in gaps)
    draft, choice, logq, score = oracle.viterbi_walk(S, S0, logp, ids)
    for n in range(N):
        gmax, path, scored = _brute_force(S, S0, logp, 0.0, n)
        assert tuple(choice[n]) == path, (seed, n, gaps[n])


def test_planted_near_ties_defeat_float_sums():
    """Over the planted cases above (48 lattices), a float32 decode returns a different path in
    at least one case in eight (12 of the 48 as seeded): the pin separates a double decode from a
    float one."""
    total = 0
    for seed in range(6):
        rng = np.random.default_rng(400 + seed)
        N, B, K = 8, int(rng.integers(3, 6)), int(rng.integers(2, 5))
        S, S0, logp, ids = _inputs(rng, N, B, K, anchor=seed % 2 == 0, coarse=False)
        S *= np.float32(4.0)
        for n in range(N):
            _plant_near_tie(rng, S, S0, n, B, K)
        for n in range(N):
            _, path, _ = _brute_force(S, S0, np.zeros_like(logp), 0.0, n)
            total += _float_dp(S, S0, n, B, K) != path
    assert total >= 6, total


@pytest.mark.parametrize("seed", range(6))
def test_greedy_never_beats_exact(seed):
    rng = np.random.default_rng(300 + seed)
    N, B, K = 4, 6, 4
    S, S0, logp, ids = _inputs(rng, N, B, K, anchor=True, coarse=False)
    _, gc, _ = oracle.greedy_walk(S, S0, logp, ids)
    _, vc, _, score = oracle.viterbi_walk(S, S0, logp, ids)
    for n in range(N):
        assert _g(S, S0, logp, 0.0, n, gc[n]) <= _g(S, S0, logp, 0.0, n, vc[n])


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
    assert abs(float(_g(S, S0, logp, 0.0, 0, gchoice[0])) - c["g_greedy"]) < 1e-6


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
