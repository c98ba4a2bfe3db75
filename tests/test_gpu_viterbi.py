"""GPU parity of lilicorr_viterbi_walk (exact max-path decode, Eq. pathscore) against the oracle.

Both sum path scores in double, each fp32 term widened exactly and each partial sum rounded once
in the same order, so on identical S / S0 / logp the path (choice, draft) is bit-exact, and logq
and the path score within 1e-5 * max(1, |oracle|). Cases: coarse scores full of exact ties, real
scores, anchor or not, lambda != 0, K from 1 to 64, B up to 1000 (matrices too large to stage in
LDS), the hand-worked greedy-versus-best example, planted near-ties of about one float ulp
(checked against enumeration in exact rational arithmetic: a float32 decode gets a share of them
wrong), and the oracle chain's own pair scores at the workloads' shapes (every request).
"""
import itertools
import os
from fractions import Fraction

import numpy as np
import pytest
import torch
import yaml

import oracle
from parity import assert_close, assert_equal, to_np

pytestmark = pytest.mark.gpu


def _gpu(lib, S, S0, logp, ids, lam=0.0):
    c = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
    out = lib.viterbi_walk(c(S), c(S0), c(logp), c(ids), lam)
    torch.cuda.synchronize()
    return [to_np(o) for o in out]


def _compare(g, r, what):
    gd, gc, gq, gs = g
    rd, rc, rq, rs = r
    assert_equal(gc, rc, f"{what} choice")
    assert_equal(gd, rd, f"{what} draft")
    assert_close(gq, rq, f"{what} logq")
    assert_close(gs, rs, f"{what} score")


@pytest.mark.parametrize("N,B,K,anchor,lam,coarse", [
    (1, 1, 1, False, 0.0, False), (3, 1, 5, True, 0.0, True), (4, 2, 2, True, 0.0, True),
    (8, 16, 16, False, 0.0, True), (8, 16, 16, True, 0.0, False), (5, 16, 32, False, 0.0, False),
    (3, 9, 64, True, 0.0, True), (2, 30, 17, True, 1.0, False), (6, 6, 3, False, -0.5, True),
    (2, 200, 8, True, 0.0, False), (2, 1000, 64, False, 0.0, False),
])
def test_viterbi_random(lib, N, B, K, anchor, lam, coarse):
    print(f"viterbi N={N} B={B} K={K} anchor={anchor} lam={lam} coarse={coarse}", flush=True)
    rng = np.random.default_rng(N * 1009 + B * 13 + K)
    if coarse:
        S = rng.integers(-3, 4, size=(N, B - 1, K, K)).astype(np.float32)
        S0 = rng.integers(-3, 4, size=(N, K)).astype(np.float32) if anchor else None
        logp = -rng.integers(0, 4, size=(N, B, K)).astype(np.float32)
    else:
        S = (rng.standard_normal((N, B - 1, K, K)) * 3).astype(np.float32)
        S0 = rng.standard_normal((N, K)).astype(np.float32) if anchor else None
        logp = -np.sort(rng.random((N, B, K)) * 4, axis=-1).astype(np.float32)
    ids = rng.integers(0, 150000, size=(N, B, K)).astype(np.int32)
    _compare(_gpu(lib, S, S0, logp, ids, lam), oracle.viterbi_walk(S, S0, logp, ids, lam),
             f"N={N} B={B} K={K}")


def test_viterbi_hand_case(lib, golden_dir):
    cases = yaml.safe_load(open(os.path.join(golden_dir, "walk_hand_cases.yaml")))["cases"]
    c = next(c for c in cases if "best_path" in c)
    S = np.array(c["S"], np.float32)[None]
    S0 = np.array(c["S0"], np.float32)[None]
    B, K = S.shape[1] + 1, S.shape[-1]
    ids = np.arange(B * K, dtype=np.int32).reshape(1, B, K)
    gd, gc, gq, gs = _gpu(lib, S, S0, np.zeros((1, B, K), np.float32), ids)
    assert gc[0].tolist() == c["best_path"]
    assert abs(float(gs[0]) - c["g_best"]) < 1e-6


def _exact_best(S, S0, n, B, K):
    """Among all K^B paths, the exact maximiser of the path score (rational arithmetic), with the
    tie rule: the smallest path read from the last slot backwards."""
    F = lambda x: Fraction(float(x))
    best = None
    for p in itertools.product(range(K), repeat=B):
        g = (F(S0[n, p[0]]) if S0 is not None else Fraction(0)) + sum(
            (F(S[n, t - 1, p[t - 1], p[t]]) for t in range(1, B)), Fraction(0))
        key = (g, tuple(-c for c in reversed(p)))
        if best is None or key > best[0]:
            best = (key, p)
    return best[1]


@pytest.mark.parametrize("seed", range(4))
def test_viterbi_planted_near_ties(lib, seed):
    """Links set so that a runner-up path beats the best by about one float ulp; the decode must
    return the exact maximiser (the planting is the oracle pins' own, on the CPU)."""
    import test_oracle_viterbi as pins

    rng = np.random.default_rng(900 + seed)
    N, B, K = 12, int(rng.integers(3, 6)), int(rng.integers(2, 5))
    S, S0, logp, ids = pins._inputs(rng, N, B, K, anchor=seed % 2 == 0, coarse=False)
    S *= np.float32(4.0)
    logp[:] = 0.0
    for n in range(N):
        pins._plant_near_tie(rng, S, S0, n, B, K)
    g = _gpu(lib, S, S0, logp, ids)
    _compare(g, oracle.viterbi_walk(S, S0, logp, ids), f"planted seed {seed}")
    for n in range(N):
        assert tuple(g[1][n]) == _exact_best(S, S0, n, B, K), (seed, n)


@pytest.mark.parametrize("cfg_index", [1, 2, 3, 4])
def test_viterbi_on_oracle_chain_scores(lib, oracle_chain, cfg_index):
    """The exact decode over the oracle chain's own pair scores, every request: bit-exact paths
    against the oracle chain's exact decode."""
    r = oracle_chain(cfg_index)
    print(f"viterbi on the oracle chain of config {cfg_index}", flush=True)
    g = _gpu(lib, r["S"], None, r["logp"], r["ids"])
    _compare(g, (r["vdraft"], r["vchoice"], r["vlogq"], r["vscore"]), f"config {cfg_index}")


@pytest.mark.parametrize("cfg_index", [1, 3])
def test_viterbi_on_chain_scores(lib, cfg_inputs, cfg_index):
    """The exact decode over the GPU chain's own pair scores (the GPU's S fed to both sides)."""
    cfg, inp = cfg_inputs(cfg_index)
    print(f"viterbi on config {cfg_index} {cfg.name}", flush=True)
    ids, logp = lib.topk(inp["logits"].cuda(), cfg.K)
    packed = lib.pack_weights(inp["W_in"].cuda(), inp["W_out"].cuda())
    S, _ = lib.pair_scores(*lib.candidate_vectors(ids, inp["E"].cuda(), packed))
    g = lib.viterbi_walk(S, None, logp, ids)
    torch.cuda.synchronize()
    g = [to_np(x) for x in g]
    r = oracle.viterbi_walk(to_np(S), None, to_np(logp), to_np(ids))
    _compare(g, r, f"config {cfg_index}")
    # the exact decode never scores below the greedy walk on the same lattice
    gd, gch, _ = lib.greedy_walk(S, None, logp, ids)
    torch.cuda.synchronize()
    Sn, gch = to_np(S).astype(np.float64), to_np(gch)
    for n in range(cfg.N):
        greedy_g = sum(Sn[n, t - 1, gch[n, t - 1], gch[n, t]] for t in range(1, cfg.B))
        assert greedy_g <= float(g[3][n]) + 1e-5 * max(1.0, abs(greedy_g))
