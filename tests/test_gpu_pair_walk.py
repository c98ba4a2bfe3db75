"""GPU parity of steps 3-4 in one pass over precomputed vectors (lilicorr_pair_walk,
lilicorr_pair_walk_certified, lilicorr_pair_viterbi), the one-pass decode for widths above the
fused projection pass (the stress workload's d = 512).

Bars:
  * against the separate calls on the same vectors (lilicorr_pair_scores -> lilicorr_greedy_walk
    or lilicorr_viterbi_walk), whose parity with the oracle the other tests establish: S, S0,
    draft, choice, logq and score bit for bit, at widths 16-1024, K 1-64, B = 1, with and without
    an anchor and a lambda term;
  * against the oracle chain on every request of every workload, the GPU's vectors fed to the
    pass: greedy and exact drafts bit-exact, logq / score within 1e-5 * max(1, |oracle|);
  * certified: the bars of the fused certified pass (draft and choice bit-exact against the oracle,
    re-scored contenders' pair scores equal to the oracle's bit for bit), on random shapes up to
    d = 512, on planted twin ties at d = 128 and 512, and on the workloads of configs 1-4 with the
    certificate's premise checked (every fp32 pair score within margin / 2 of the oracle's).
"""
import numpy as np
import pytest
import torch

from parity import assert_close, assert_equal, to_np
from test_gpu_certified import MARGIN, _check as _check_cert, _random_case, _twin_case
from test_gpu_score_walk import _oracle

pytestmark = pytest.mark.gpu


def _t(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _vectors(lib, ids, E, W_in, W_out):
    packed = lib.pack_weights(_t(W_in), _t(W_out))
    iv, ov = lib.candidate_vectors(_t(ids), E.cuda(), packed)
    return iv, ov, packed


def _np(d):
    return {k: (to_np(v) if v is not None else None) for k, v in d.items()}


@pytest.mark.parametrize("N,B,K,d,anchor,lam", [
    (1, 1, 1, 16, False, 0.0), (1, 1, 8, 128, True, 0.0), (2, 2, 3, 48, True, 0.0),
    (3, 5, 5, 80, False, 0.0), (2, 17, 16, 256, True, 0.0), (2, 16, 32, 512, False, 0.0),
    (2, 9, 33, 512, True, 0.5), (1, 6, 64, 1024, True, 0.0), (2, 5, 64, 96, False, -0.5),
    (4, 30, 8, 64, False, 1.0), (1, 300, 16, 32, False, 0.0), (3, 16, 32, 1024, False, 0.0),
])
def test_pair_walk_matches_separate_calls(lib, N, B, K, d, anchor, lam):
    print(f"pair_walk N={N} B={B} K={K} d={d} anchor={anchor} lam={lam}", flush=True)
    rng = np.random.default_rng(N * 7919 + B * 31 + K + d)
    iv = _t(rng.standard_normal((N, B, K, d)).astype(np.float32))
    ov = _t(rng.standard_normal((N, B, K, d)).astype(np.float32))
    iv[0, 0, 0] = 0.0    # a zero vector scores 0
    ids = _t(rng.integers(0, 1000, size=(N, B, K)).astype(np.int32))
    logp = _t(-np.sort(rng.random((N, B, K)) * 4, axis=-1).astype(np.float32))
    ao = _t(rng.standard_normal((N, d)).astype(np.float32)) if anchor else None

    S, S0 = lib.pair_scores(iv, ov, ao, 8.0)
    want = dict(zip(("draft", "choice", "logq"), lib.greedy_walk(S, S0, logp, ids, lam)))
    want_x = dict(zip(("draft", "choice", "logq", "score"), lib.viterbi_walk(S, S0, logp, ids, lam)))
    got = dict(zip(("draft", "choice", "logq", "S", "S0"),
                   lib.pair_walk(iv, ov, logp, ids, ao, 8.0, lam, scores=True)))
    got_x = dict(zip(("draft", "choice", "logq", "score", "S", "S0"),
                     lib.pair_viterbi(iv, ov, logp, ids, ao, 8.0, lam, scores=True)))
    torch.cuda.synchronize()
    want, want_x, got, got_x = _np(want), _np(want_x), _np(got), _np(got_x)
    what = f"N={N} B={B} K={K} d={d}"
    for g in (got, got_x):
        if B > 1:
            assert_equal(g["S"].view(np.uint32), to_np(S).view(np.uint32), f"{what} S")
        if anchor:
            assert_equal(g["S0"].view(np.uint32), to_np(S0).view(np.uint32), f"{what} S0")
    for k in ("draft", "choice"):
        assert_equal(got[k], want[k], f"{what} greedy {k}")
        assert_equal(got_x[k], want_x[k], f"{what} exact {k}")
    assert_equal(got["logq"].view(np.uint32), want["logq"].view(np.uint32), f"{what} greedy logq")
    for k in ("logq", "score"):
        assert_equal(got_x[k].view(np.uint32), want_x[k].view(np.uint32), f"{what} exact {k}")


@pytest.mark.parametrize("cfg_index", [0, 1, 2, 3, 4])
def test_pair_walk_chain_configs(lib, cfg_inputs, oracle_chain, cfg_index):
    """topk -> candidate_vectors -> the one-pass decode, every request, against the oracle chain's
    greedy walk and exact decode (each on its own scores)."""
    cfg, inp = cfg_inputs(cfg_index)
    print(f"pair_walk chain config {cfg_index} {cfg.name}", flush=True)
    ids, logp = lib.topk(inp["logits"].cuda(), cfg.K)
    packed = lib.pack_weights(inp["W_in"].cuda(), inp["W_out"].cuda())
    iv, ov = lib.candidate_vectors(ids, inp["E"].cuda(), packed)
    d, c, q, S, _ = lib.pair_walk(iv, ov, logp, ids, scores=True)
    vd, vc, vq, vs = lib.pair_viterbi(iv, ov, logp, ids)
    torch.cuda.synchronize()
    del iv, ov
    r = oracle_chain(cfg_index)
    what = f"cfg{cfg_index} ({cfg.N} requests)"
    assert_close(to_np(S), r["S"], f"{what} S")
    assert_equal(to_np(c), r["choice"], f"{what} greedy choice")
    assert_equal(to_np(d), r["draft"], f"{what} greedy draft")
    assert_close(to_np(q), r["logq"], f"{what} greedy logq")
    assert_equal(to_np(vc), r["vchoice"], f"{what} exact choice")
    assert_equal(to_np(vd), r["vdraft"], f"{what} exact draft")
    assert_close(to_np(vq), r["vlogq"], f"{what} exact logq")
    assert_close(to_np(vs), r["vscore"], f"{what} exact score")


def _run(lib, iv, ov, ids, logp, E, packed, ao, lam, margin=None, workspace=None):
    if margin is None:
        out = lib.pair_walk(iv, ov, _t(logp), _t(ids), _t(ao), 8.0, lam, scores=True,
                            workspace=workspace)
        keys = ("draft", "choice", "logq", "S", "S0")
    else:
        out = lib.pair_walk_certified(iv, ov, _t(logp), _t(ids), E, packed, _t(ao), 8.0, lam,
                                      margin, scores=True, workspace=workspace)
        keys = ("draft", "choice", "logq", "rescored", "S", "S0")
    torch.cuda.synchronize()
    return _np(dict(zip(keys, out)))


@pytest.mark.parametrize("margin", [MARGIN, 0.0, 1e3])
@pytest.mark.parametrize("N,B,K,d,anchor,lam", [
    (1, 1, 1, 16, False, 0.0), (2, 2, 3, 48, True, 0.0), (2, 17, 16, 256, True, 0.0),
    (2, 16, 32, 512, False, 0.0), (2, 5, 33, 512, True, 1.0), (1, 4, 64, 320, False, 0.0),
])
def test_pair_walk_certified_shapes(lib, N, B, K, d, anchor, lam, margin):
    print(f"pair_walk certified N={N} B={B} K={K} d={d} anchor={anchor} lam={lam} "
          f"margin={margin}", flush=True)
    E, W_in, W_out, ids, logp, ao = _random_case(N * 7919 + B * 31 + K, N, B, K, d, anchor)
    iv, ov, packed = _vectors(lib, ids, E, W_in, W_out)
    g = _run(lib, iv, ov, ids, logp, E.cuda(), packed, ao, lam, margin)
    plain = _run(lib, iv, ov, ids, logp, E.cuda(), packed, ao, lam)
    r = _oracle(ids, logp, to_np(E), W_in, W_out, ao, lam)
    touched = _check_cert(g, plain, r, logp, lam, margin, f"N={N} B={B} K={K} d={d} m={margin}")
    if margin > 100 and K > 1:
        first = 0 if anchor else 1
        assert (g["rescored"][:, first:] > 0).all()
        assert touched == N * (B - first)


@pytest.mark.parametrize("N,B,K,d,anchor", [(32, 8, 4, 128, False), (16, 16, 32, 512, True),
                                           (16, 16, 16, 512, False)])
def test_pair_walk_certified_planted_ties(lib, N, B, K, d, anchor):
    print(f"pair_walk certified twins N={N} B={B} K={K} d={d} anchor={anchor}", flush=True)
    E, W_in, W_out, ids, logp, ao = _twin_case(N, B, K, d, anchor=anchor)
    iv, ov, packed = _vectors(lib, ids, E, W_in, W_out)
    g = _run(lib, iv, ov, ids, logp, E.cuda(), packed, ao, 0.0, MARGIN)
    plain = _run(lib, iv, ov, ids, logp, E.cuda(), packed, ao, 0.0)
    r = _oracle(ids, logp, to_np(E), W_in, W_out, ao)
    first = 0 if anchor else 1
    assert (g["rescored"][:, first:] > 0).all()
    _check_cert(g, plain, r, logp, 0.0, MARGIN, f"twins N={N} B={B} K={K} d={d}")
    wrong = int((plain["choice"] != r["choice"]).any(axis=1).sum())
    changed = int((g["rescored"] == 2).sum())
    print(f"  requests the fp32 pass decides differently from the oracle: {wrong} of {N}; "
          f"decisions changed by the re-scoring: {changed}", flush=True)
    assert wrong > 0 and changed > 0, "the planted ties no longer separate the two passes"


@pytest.mark.parametrize("cfg_index", [1, 2, 3, 4])
def test_pair_walk_certified_configs(lib, cfg_inputs, oracle_chain, cfg_index):
    """The workloads on the oracle's top-K: the oracle's drafts, and the certificate's premise."""
    cfg, inp = cfg_inputs(cfg_index)
    print(f"pair_walk certified config {cfg_index} {cfg.name}", flush=True)
    r = oracle_chain(cfg_index)
    E = inp["E"].cuda()
    packed = lib.pack_weights(inp["W_in"].cuda(), inp["W_out"].cuda())
    iv, ov = lib.candidate_vectors(_t(r["ids"]), E, packed)
    g = _run(lib, iv, ov, r["ids"], r["logp"], E, packed, None, 0.0, MARGIN)
    plain = _run(lib, iv, ov, r["ids"], r["logp"], E, packed, None, 0.0)
    del iv, ov
    rr = dict(S=r["S"], S0=None, draft=r["draft"], choice=r["choice"], logq=r["logq"])
    _check_cert(g, plain, rr, r["logp"], 0.0, MARGIN, f"cfg{cfg_index}")
    err = float(np.abs(plain["S"].astype(np.float64) - r["S"]).max())
    print(f"  max |S fp32 - S oracle| = {err:.3g}; re-scored decisions: "
          f"{int((g['rescored'] > 0).sum())} of {g['rescored'].size}", flush=True)
    assert err <= MARGIN / 2


def test_pair_walk_reuses_workspace(lib):
    """Every call leaves its workspace ready for the next: three calls, then a smaller batch, for
    each decode rule."""
    N, B, K, d = 8, 16, 32, 512
    ws = {"greedy": lib.score_walk_workspace(N, B, K),
          "exact": lib.score_viterbi_workspace(N, B, K),
          "certified": lib.score_walk_certified_workspace(N, B, K)}
    for call, n in enumerate([N, N, N, 3]):
        rng = np.random.default_rng(call)
        iv = _t(rng.standard_normal((n, B, K, d)).astype(np.float32))
        ov = _t(rng.standard_normal((n, B, K, d)).astype(np.float32))
        ids = _t(rng.integers(0, 1000, size=(n, B, K)).astype(np.int32))
        logp = _t(-np.sort(rng.random((n, B, K)) * 4, axis=-1).astype(np.float32))
        S, _ = lib.pair_scores(iv, ov)
        want = lib.greedy_walk(S, None, logp, ids)
        want_x = lib.viterbi_walk(S, None, logp, ids)
        got = lib.pair_walk(iv, ov, logp, ids, workspace=ws["greedy"])
        got_x = lib.pair_viterbi(iv, ov, logp, ids, workspace=ws["exact"])
        torch.cuda.synchronize()
        for a, b, k in zip(got + got_x, want + want_x, ("draft", "choice", "logq") * 2 + ("score",)):
            assert_equal(to_np(a).view(np.uint32), to_np(b).view(np.uint32), f"call {call} {k}")
    E, W_in, W_out, ids, logp, ao = _twin_case(N, B, K, d)
    iv, ov, packed = _vectors(lib, ids, E, W_in, W_out)
    r = _oracle(ids, logp, to_np(E), W_in, W_out)
    for call in range(2):
        g = _run(lib, iv, ov, ids, logp, E.cuda(), packed, None, 0.0, MARGIN,
                 workspace=ws["certified"])
        assert_equal(g["draft"], r["draft"], f"certified call {call} draft")
    for w in ws.values():
        assert int(w[:256].view(torch.int32)[:N].abs().sum()) == 0, "counters back at zero"
