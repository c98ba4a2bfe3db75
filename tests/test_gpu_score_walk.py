"""GPU parity of lilicorr_score_walk (steps 2-4 in one pass) against the oracle.

On the same ids / logp the fused pass must give the oracle's draft and choice bit-exactly, its
logq and (when asked for) its pair scores S / S0 within 1e-5 * max(1, |oracle|): the oracle
chain is candidate_vectors -> pair_scores -> greedy_walk in fp64. Shapes cover one and several
pairs per workgroup, K not a multiple of 16, K = 64, padded d, B = 1, many pair groups, the
anchor workgroup, lambda != 0, ids outside the table, and repeated calls on one workspace.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from parity import assert_close, assert_equal, greedy_gap, path_gap, to_np

pytestmark = pytest.mark.gpu


def _oracle(ids, logp, E_np, W_in, W_out, anchor=None, lam=0.0):
    # the library maps ids outside [0, V) to zero vectors (a memory-safety rule, not the
    # paper's); the oracle takes valid ids only, so such ids point at an appended zero row
    V = E_np.shape[0]
    valid = (ids >= 0) & (ids < V)
    ids_o = np.where(valid, ids, V).astype(np.int32)
    E_o = np.concatenate([E_np, np.zeros_like(E_np[:1])])
    iv, ov = oracle.candidate_vectors(ids_o, E_o, W_in, W_out)
    S, S0 = oracle.pair_scores(iv, ov, anchor, 8.0)
    _, choice, logq = oracle.greedy_walk(S, S0, logp, ids_o, lam)
    draft = np.take_along_axis(ids, choice[..., None].astype(np.int64), -1)[..., 0]
    return dict(S=S, S0=S0, draft=draft, choice=choice, logq=logq)


def _check(g, r, what, B):
    assert_equal(g["choice"], r["choice"], f"{what} choice")
    assert_equal(g["draft"], r["draft"], f"{what} draft")
    assert_close(g["logq"], r["logq"], f"{what} logq")
    if B > 1:
        assert_close(g["S"], r["S"], f"{what} S")
    if r["S0"] is not None:
        assert_close(g["S0"], r["S0"], f"{what} S0")


def _run(lib, ids, logp, E, packed, anchor=None, lam=0.0, workspace=None):
    c = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
    draft, choice, logq, S, S0 = lib.score_walk(c(ids), c(logp), E, packed, c(anchor), 8.0, lam,
                                                scores=True, workspace=workspace)
    torch.cuda.synchronize()
    return dict(draft=to_np(draft), choice=to_np(choice), logq=to_np(logq),
                S=to_np(S) if S is not None else None, S0=to_np(S0) if S0 is not None else None)


@pytest.mark.parametrize("N,B,K,d,anchor,lam", [
    (1, 1, 1, 16, False, 0.0), (1, 1, 4, 64, True, 0.0), (2, 2, 3, 48, True, 0.0),
    (3, 5, 5, 80, False, 0.0), (2, 17, 16, 256, True, 0.0), (1, 9, 32, 128, False, 0.0),
    (2, 4, 64, 256, True, 0.0), (4, 30, 8, 64, False, 1.0), (1, 300, 16, 32, False, 0.0),
    (2, 16, 17, 96, True, -0.5), (3, 7, 2, 256, True, 0.0),
])
def test_score_walk_shapes(lib, N, B, K, d, anchor, lam):
    print(f"score_walk N={N} B={B} K={K} d={d} anchor={anchor} lam={lam}", flush=True)
    rng = np.random.default_rng(N * 7919 + B * 31 + K)
    V = 500
    E = torch.from_numpy((rng.standard_normal((V, d)) * 0.05).astype(np.float32)).to(torch.bfloat16)
    W_in = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    W_out = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    ids = rng.integers(0, V, size=(N, B, K)).astype(np.int32)
    ids.reshape(-1)[::11] = -3       # outside the table: zero vectors, cosine 0
    ids.reshape(-1)[5::13] = V + 2
    logp = -np.sort(rng.random((N, B, K)) * 4, axis=-1).astype(np.float32)
    ao = rng.standard_normal((N, d)).astype(np.float32) if anchor else None
    packed = lib.pack_weights(torch.from_numpy(W_in).cuda(), torch.from_numpy(W_out).cuda())
    g = _run(lib, ids, logp, E.cuda(), packed, ao, lam)
    r = _oracle(ids, logp, to_np(E), W_in, W_out, ao, lam)
    _check(g, r, f"N={N} B={B} K={K} d={d}", B)


@pytest.mark.parametrize("cfg_index", [1, 2, 3])
def test_score_walk_configs(lib, cfg_inputs, oracle_chain, cfg_index):
    """Every request of the workloads' own shapes, from the oracle's own top-K, against the
    oracle chain (fp64 vectors and scores, greedy walk)."""
    cfg, inp = cfg_inputs(cfg_index)
    print(f"score_walk config {cfg_index} {cfg.name}", flush=True)
    r = oracle_chain(cfg_index)
    ids, logp = torch.from_numpy(r["ids"]).cuda(), torch.from_numpy(r["logp"]).cuda()
    E = inp["E"].cuda()
    packed = lib.pack_weights(inp["W_in"].cuda(), inp["W_out"].cuda())
    draft, choice, logq, S, _ = lib.score_walk(ids, logp, E, packed, scores=True)
    torch.cuda.synchronize()
    g = dict(draft=to_np(draft), choice=to_np(choice), logq=to_np(logq), S=to_np(S), S0=None)
    what = f"cfg{cfg_index} ({cfg.N} requests)"
    assert_close(g["S"], r["S"], f"{what} S")
    bad = np.argwhere((g["choice"] != r["choice"]).any(axis=1))
    if bad.size:
        n = int(bad[0, 0])
        t = int(np.argmax(g["choice"][n] != r["choice"][n]))
        raise AssertionError(f"{what}: drafts differ in {bad.size} requests; request {n} slot {t}: "
                             f"oracle top-2 gap {greedy_gap(r['S'], None, r['choice'], n, t):.3e}")
    assert_equal(g["draft"], r["draft"], f"{what} draft")
    assert_close(g["logq"], r["logq"], f"{what} logq")
    # the separate calls give the same drafts
    d4, c4, _ = lib.greedy_walk(*lib.pair_scores(*lib.candidate_vectors(ids, E, packed)), logp, ids)
    torch.cuda.synchronize()
    assert_equal(g["draft"], to_np(d4), f"cfg{cfg_index} fused vs separate calls")


def test_score_walk_with_anchor_config(lib, cfg_inputs):
    cfg, inp = cfg_inputs(1)
    anchor = to_np(workloads.make_anchor(cfg))
    ids, logp = lib.topk(inp["logits"].cuda(), cfg.K)
    packed = lib.pack_weights(inp["W_in"].cuda(), inp["W_out"].cuda())
    g = _run(lib, to_np(ids), to_np(logp), inp["E"].cuda(), packed, anchor)
    r = _oracle(to_np(ids), to_np(logp), to_np(inp["E"]), to_np(inp["W_in"]), to_np(inp["W_out"]),
                anchor)
    _check(g, r, "config 1 with anchor", cfg.B)


def test_score_walk_reuses_workspace(lib):
    """Every call leaves the workspace ready for the next: three calls, then a smaller batch."""
    rng = np.random.default_rng(3)
    N, B, K, d, V = 8, 16, 16, 128, 400
    E = torch.from_numpy((rng.standard_normal((V, d)) * 0.05).astype(np.float32)).to(torch.bfloat16)
    W_in = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    W_out = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    packed = lib.pack_weights(torch.from_numpy(W_in).cuda(), torch.from_numpy(W_out).cuda())
    ws = lib.score_walk_workspace(N, B, K)
    for call, n in enumerate([N, N, N, 3]):
        ids = rng.integers(0, V, size=(n, B, K)).astype(np.int32)
        logp = -np.sort(rng.random((n, B, K)) * 4, axis=-1).astype(np.float32)
        g = _run(lib, ids, logp, E.cuda(), packed, workspace=ws)
        r = _oracle(ids, logp, to_np(E), W_in, W_out)
        _check(g, r, f"call {call}", B)
    assert int(ws[: 4 * N].view(torch.int32).abs().sum().item()) == 0  # counters back at zero


# ---- the same pass with the exact max-path decode (lilicorr_score_viterbi) ---------------------

def _run_exact(lib, ids, logp, E, packed, anchor=None, lam=0.0, workspace=None):
    c = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()
    d, ch, q, g, S, S0 = lib.score_viterbi(c(ids), c(logp), E, packed, c(anchor), 8.0, lam,
                                           scores=True, workspace=workspace)
    torch.cuda.synchronize()
    return dict(draft=to_np(d), choice=to_np(ch), logq=to_np(q), score=to_np(g),
                S=to_np(S) if S is not None else None, S0=to_np(S0) if S0 is not None else None)


def _check_exact(g, ids, logp, E_np, W_in, W_out, anchor, lam, what):
    """Scores against the oracle's fp64 chain; the decode (1) against the oracle's exact decode
    on the oracle's own scores (the end-to-end result), and (2) against the oracle's exact decode
    on the very scores the pass produced (both sum paths in double in the same order, so on
    identical scores the path is bit-exact whatever the margins). For (1) a request whose best
    and second-best oracle path scores lie within twice the largest possible drift of a path sum
    (B times the largest fp32 score error) is a tie at the pass's precision: its path may
    differ, and is counted rather than failed (the workloads' own tests allow none)."""
    B = ids.shape[1]
    r = _oracle(ids, logp, E_np, W_in, W_out, anchor, lam)
    if B > 1:
        assert_close(g["S"], r["S"], f"{what} S")
    if anchor is not None:
        assert_close(g["S0"], r["S0"], f"{what} S0")
    ids_ok = np.clip(ids, 0, None)
    empty = np.zeros((ids.shape[0], 0, ids.shape[2], ids.shape[2]), np.float32)
    S_r = r["S"] if B > 1 else empty
    S_g = g["S"] if B > 1 else empty
    err = float(np.abs(S_g.astype(np.float64) - S_r).max()) if B > 1 else 0.0
    if anchor is not None:
        err = max(err, float(np.abs(g["S0"].astype(np.float64) - r["S0"]).max()))
    ties = _check_exact_path(g, oracle.viterbi_walk(S_r, r["S0"], logp, ids_ok, lam), ids, S_r,
                             r["S0"], f"{what} (oracle scores)", tie_band=2 * B * err,
                             logp=logp, lam=lam)
    if ties:
        print(f"{what}: {ties} request(s) tied within the fp32 score error", flush=True)
    _check_exact_path(g, oracle.viterbi_walk(S_g, g["S0"], logp, ids_ok, lam), ids, S_g, g["S0"],
                      f"{what} (the pass's scores)")


def _check_exact_path(g, ref, ids, S, S0, what, tie_band=0.0, logp=None, lam=0.0):
    """Path (choice, draft) bit-exact, logq and score within tolerance, per request; a request
    whose paths differ passes only when the reference's best and second-best path scores are
    within tie_band. Returns the number of such requests."""
    vd, vc, vq, vs = ref
    differ = (g["choice"] != vc).any(axis=1)
    for n in np.argwhere(differ)[:, 0]:
        gap = path_gap(S, S0, int(n), logp, lam)
        if not gap <= tie_band:
            raise AssertionError(f"{what}: paths differ in {int(differ.sum())} requests; request "
                                 f"{int(n)}: best-to-second path gap {gap:.3e}")
    keep = ~differ
    draft_ref = np.take_along_axis(ids, vc[..., None].astype(np.int64), -1)[..., 0]
    assert_equal(g["draft"][keep], draft_ref[keep], f"{what} draft")
    assert_close(g["logq"][keep], vq[keep], f"{what} logq")
    assert_close(g["score"][keep], vs[keep], f"{what} score")
    return int(differ.sum())


@pytest.mark.parametrize("N,B,K,d,anchor,lam", [
    (1, 1, 1, 16, False, 0.0), (1, 1, 4, 64, True, 0.0), (2, 2, 3, 48, True, 0.0),
    (3, 5, 5, 80, False, 0.0), (2, 17, 16, 256, True, 0.0), (1, 9, 32, 128, False, 0.0),
    (2, 4, 64, 256, True, 0.0), (4, 30, 8, 64, False, 1.0), (1, 300, 16, 32, False, 0.0),
    (2, 16, 17, 96, True, -0.5), (2, 200, 64, 32, False, 0.0),
])
def test_score_viterbi_shapes(lib, N, B, K, d, anchor, lam):
    print(f"score_viterbi N={N} B={B} K={K} d={d} anchor={anchor} lam={lam}", flush=True)
    rng = np.random.default_rng(N * 7919 + B * 31 + K + 1)
    V = 500
    E = torch.from_numpy((rng.standard_normal((V, d)) * 0.05).astype(np.float32)).to(torch.bfloat16)
    W_in = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    W_out = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    ids = rng.integers(0, V, size=(N, B, K)).astype(np.int32)
    ids.reshape(-1)[::11] = -3
    logp = -np.sort(rng.random((N, B, K)) * 4, axis=-1).astype(np.float32)
    ao = rng.standard_normal((N, d)).astype(np.float32) if anchor else None
    packed = lib.pack_weights(torch.from_numpy(W_in).cuda(), torch.from_numpy(W_out).cuda())
    g = _run_exact(lib, ids, logp, E.cuda(), packed, ao, lam)
    _check_exact(g, ids, logp, to_np(E), W_in, W_out, ao, lam, f"N={N} B={B} K={K} d={d}")


@pytest.mark.parametrize("cfg_index", [1, 2, 3])
def test_score_viterbi_configs(lib, cfg_inputs, oracle_chain, cfg_index):
    """Every request, from the oracle's own top-K, against the oracle chain's exact decode on the
    oracle's own scores; and on the pass's scores (bit-exact decisions on identical scores)."""
    cfg, inp = cfg_inputs(cfg_index)
    print(f"score_viterbi config {cfg_index} {cfg.name}", flush=True)
    r = oracle_chain(cfg_index)
    packed = lib.pack_weights(inp["W_in"].cuda(), inp["W_out"].cuda())
    g = _run_exact(lib, r["ids"], r["logp"], inp["E"].cuda(), packed)
    what = f"cfg{cfg_index} ({cfg.N} requests)"
    assert_close(g["S"], r["S"], f"{what} S")
    _check_exact_path(g, (r["vdraft"], r["vchoice"], r["vlogq"], r["vscore"]), r["ids"], r["S"],
                      None, f"{what} (oracle chain)")
    _check_exact_path(g, oracle.viterbi_walk(g["S"], None, r["logp"], r["ids"]), r["ids"], g["S"],
                      None, f"{what} (the pass's scores)")


def test_score_viterbi_reuses_workspace(lib):
    rng = np.random.default_rng(5)
    N, B, K, d, V = 8, 16, 16, 64, 300
    E = torch.from_numpy((rng.standard_normal((V, d)) * 0.05).astype(np.float32)).to(torch.bfloat16)
    W_in = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    W_out = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    packed = lib.pack_weights(torch.from_numpy(W_in).cuda(), torch.from_numpy(W_out).cuda())
    ws = lib.score_viterbi_workspace(N, B, K)
    for call, n in enumerate([N, N, 2]):
        ids = rng.integers(0, V, size=(n, B, K)).astype(np.int32)
        logp = -np.sort(rng.random((n, B, K)) * 4, axis=-1).astype(np.float32)
        g = _run_exact(lib, ids, logp, E.cuda(), packed, workspace=ws)
        _check_exact(g, ids, logp, to_np(E), W_in, W_out, None, 0.0, f"call {call}")
    assert int(ws[: 4 * N].view(torch.int32).abs().sum().item()) == 0
