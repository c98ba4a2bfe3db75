"""GPU parity of lilicorr_score_walk_certified (the fused greedy pass with near-tied decisions
decided again in fp64) against the oracle chain candidate_vectors -> pair_scores -> greedy_walk.

Bars: draft and choice bit-exact; logq and S within 1e-5 * max(1, |oracle|); and, for every
re-scored decision, the contenders' pair scores equal the oracle's bit for bit (the re-scoring
repeats the oracle's double-precision operations in the oracle's order). Inputs:
  * random shapes (as for the plain pass), with the default margin, margin 0 (exact fp32 ties
    only) and a margin above every score gap (every decision re-scored, all K contenders);
  * planted ties: each slot's candidates come in twin pairs whose pair scores are equal in exact
    arithmetic (the out vectors are symmetric in two coordinates and the twins' in vectors swap
    them), so every decision is a tie that fp32 rounding order may break either way;
  * the workloads of configs 1-3, where the premise of the certificate is checked too: every
    fp32 pair score within margin / 2 of the oracle's.
"""
import numpy as np
import pytest
import torch

from parity import assert_close, assert_equal, to_np
from test_gpu_score_walk import _oracle, _run as _run_plain

pytestmark = pytest.mark.gpu

MARGIN = 2.0 ** -14


def _t(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _run_cert(lib, ids, logp, E, packed, anchor=None, lam=0.0, margin=MARGIN, workspace=None):
    draft, choice, logq, resc, S, S0 = lib.score_walk_certified(
        _t(ids), _t(logp), E, packed, _t(anchor), 8.0, lam, margin, scores=True,
        workspace=workspace)
    torch.cuda.synchronize()
    return dict(draft=to_np(draft), choice=to_np(choice), logq=to_np(logq), rescored=to_np(resc),
                S=to_np(S) if S is not None else None, S0=to_np(S0) if S0 is not None else None)


def _node_scores(row, lp, lam):
    if lam == 0.0:
        return row.astype(np.float32)
    return (np.float64(lam) * lp.astype(np.float64) + row.astype(np.float64)).astype(np.float32)


def _check(g, plain, r, logp, lam, margin, what):
    """g: certified pass, plain: the fp32 pass on the same inputs, r: the oracle chain."""
    assert_equal(g["choice"], r["choice"], f"{what} choice")
    assert_equal(g["draft"], r["draft"], f"{what} draft")
    assert_close(g["logq"], r["logq"], f"{what} logq")
    assert set(np.unique(g["rescored"])) <= {0, 1, 2}
    N, B = g["draft"].shape
    if B > 1:
        assert_close(g["S"], r["S"], f"{what} S")
    if r["S0"] is not None:
        assert_close(g["S0"], r["S0"], f"{what} S0")
    touched = 0
    mask = np.zeros(g["S"].shape if B > 1 else (0,), bool)
    for n in range(N):
        for t in range(B):
            if g["rescored"][n, t] == 0:
                continue
            if t == 0:
                assert r["S0"] is not None, "slot 0 re-scored without an anchor"
                row_p, row_g, row_r = plain["S0"][n], g["S0"][n], r["S0"][n]
            else:
                c = g["choice"][n, t - 1]
                row_p, row_g, row_r = plain["S"][n, t - 1, c], g["S"][n, t - 1, c], r["S"][n, t - 1, c]
            # the kernel's contenders: fp32 node scores within the margin of the row's maximum
            # (lambda is a power of two in these tests, so the double evaluation is exact)
            z = _node_scores(row_p, logp[n, t], lam)
            cont = z >= np.float32(z.max()) - np.float32(margin)
            assert cont.sum() >= 2, f"{what}: n={n} t={t} re-scored with one contender"
            assert np.array_equal(row_g[cont].view(np.uint32), row_r[cont].view(np.uint32)), (
                f"{what}: n={n} t={t} re-scored pair scores differ from the oracle's: "
                f"{row_g[cont]} vs {row_r[cont]}")
            if t > 0:
                mask[n, t - 1, c] = cont
            touched += 1
    if B > 1:  # every other entry is the fp32 pass's own
        assert np.array_equal(g["S"][~mask].view(np.uint32), plain["S"][~mask].view(np.uint32))
    return touched


def _random_case(seed, N, B, K, d, anchor, V=500):
    rng = np.random.default_rng(seed)
    E = torch.from_numpy((rng.standard_normal((V, d)) * 0.05).astype(np.float32)).to(torch.bfloat16)
    W_in = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    W_out = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    ids = rng.integers(0, V, size=(N, B, K)).astype(np.int32)
    ids.reshape(-1)[::11] = -3       # outside the table: zero vectors, cosine 0
    logp = -np.sort(rng.random((N, B, K)) * 4, axis=-1).astype(np.float32)
    ao = rng.standard_normal((N, d)).astype(np.float32) if anchor else None
    return E, W_in, W_out, ids, logp, ao


@pytest.mark.parametrize("margin", [MARGIN, 0.0, 1e3])
@pytest.mark.parametrize("N,B,K,d,anchor,lam", [
    (1, 1, 1, 16, False, 0.0), (2, 2, 3, 48, True, 0.0), (3, 5, 5, 80, False, 0.0),
    (2, 17, 16, 256, True, 0.0), (1, 9, 32, 128, False, 0.0), (2, 4, 64, 256, True, 0.0),
    (4, 30, 8, 64, False, 1.0), (2, 16, 17, 96, True, -0.5),
])
def test_certified_shapes(lib, N, B, K, d, anchor, lam, margin):
    print(f"certified N={N} B={B} K={K} d={d} anchor={anchor} lam={lam} margin={margin}",
          flush=True)
    E, W_in, W_out, ids, logp, ao = _random_case(N * 7919 + B * 31 + K, N, B, K, d, anchor)
    packed = lib.pack_weights(torch.from_numpy(W_in).cuda(), torch.from_numpy(W_out).cuda())
    g = _run_cert(lib, ids, logp, E.cuda(), packed, ao, lam, margin)
    plain = _run_plain(lib, ids, logp, E.cuda(), packed, ao, lam)
    r = _oracle(ids, logp, to_np(E), W_in, W_out, ao, lam)
    touched = _check(g, plain, r, logp, lam, margin, f"N={N} B={B} K={K} d={d} m={margin}")
    if margin > 100 and K > 1:
        # every decision with scores to compare is re-scored, over all K candidates
        first = 0 if anchor else 1
        assert (g["rescored"][:, first:] > 0).all()
        assert touched == N * (B - first)
    if (g["rescored"] == 0).all():
        assert_equal(g["draft"], plain["draft"], "nothing re-scored: the fp32 pass's draft")


def _twin_case(N, B, K, d=64, anchor=False, seed=5):
    """Candidates in twin pairs (2m, 2m+1) whose pair scores tie in exact arithmetic.

    W_out = I makes the out vector e / ||e||; every embedding row has e[0] = e[37], so every out
    vector (and the anchor, when given) is symmetric in coordinates 0 and 37. W_in is the cyclic
    shift u[j] = e[(j - 2) mod d], so an in vector's coordinates 0 and 37 are e[d-2] and e[35]; a
    twin swaps e[d-2] and e[35]: same norm, and the same dot product with any symmetric out vector.
    """
    assert K % 2 == 0
    rng = np.random.default_rng(seed)
    M = N * B * K
    base = (rng.standard_normal((M // 2, d)) * 0.05).astype(np.float32)
    base[:, 37] = base[:, 0]
    base[:, d - 2] = base[:, 35] + 0.03 + np.abs(base[:, d - 2])  # the twins differ
    e = torch.from_numpy(base).to(torch.bfloat16)
    twin = e.clone()
    twin[:, [35, d - 2]] = e[:, [d - 2, 35]]
    E = torch.stack([e, twin], 1).reshape(M, d).contiguous()
    W_out = np.eye(d, dtype=np.float32)
    W_in = np.zeros((d, d), np.float32)
    W_in[np.arange(d), (np.arange(d) + 2) % d] = 1.0   # u[j] = e[(j - 2) mod d]
    ids = np.arange(M, dtype=np.int32).reshape(N, B, K)
    lp = -np.sort(rng.random((N, B, K // 2)) * 4, axis=-1).astype(np.float32)
    logp = np.repeat(lp, 2, axis=-1)                    # twins share their log-probability
    ao = None
    if anchor:
        ao = rng.standard_normal((N, d)).astype(np.float32)
        ao[:, 37] = ao[:, 0]
    return E, W_in, W_out, ids, logp, ao


@pytest.mark.parametrize("N,B,K,anchor,lam", [(64, 8, 4, False, 0.0), (32, 16, 16, True, 0.0),
                                             (32, 6, 8, True, 0.5)])
def test_certified_planted_ties(lib, N, B, K, anchor, lam):
    print(f"certified twins N={N} B={B} K={K} anchor={anchor} lam={lam}", flush=True)
    E, W_in, W_out, ids, logp, ao = _twin_case(N, B, K, anchor=anchor)
    packed = lib.pack_weights(torch.from_numpy(W_in).cuda(), torch.from_numpy(W_out).cuda())
    g = _run_cert(lib, ids, logp, E.cuda(), packed, ao, lam)
    plain = _run_plain(lib, ids, logp, E.cuda(), packed, ao, lam)
    r = _oracle(ids, logp, to_np(E), W_in, W_out, ao, lam)
    # every decision with pair scores is a tie between twins, so every one of them is re-scored
    first = 0 if anchor else 1
    assert (g["rescored"][:, first:] > 0).all()
    _check(g, plain, r, logp, lam, MARGIN, f"twins N={N} B={B} K={K}")
    wrong = int((plain["choice"] != r["choice"]).any(axis=1).sum())
    changed = int((g["rescored"] == 2).sum())
    print(f"  requests the fp32 pass decides differently from the oracle: {wrong} of {N}; "
          f"decisions changed by the re-scoring: {changed}", flush=True)
    assert wrong > 0 and changed > 0, "the planted ties no longer separate the two passes"


@pytest.mark.parametrize("cfg_index", [1, 2, 3])
def test_certified_configs(lib, cfg_inputs, cfg_index):
    """The workloads, on the GPU's top-K: the oracle's drafts, and the certificate's premise."""
    cfg, inp = cfg_inputs(cfg_index)
    print(f"certified config {cfg_index} {cfg.name}", flush=True)
    ids, logp = lib.topk(inp["logits"].cuda(), cfg.K)
    E = inp["E"].cuda()
    packed = lib.pack_weights(inp["W_in"].cuda(), inp["W_out"].cuda())
    ids_np, logp_np = to_np(ids), to_np(logp)
    g = _run_cert(lib, ids_np, logp_np, E, packed)
    plain = _run_plain(lib, ids_np, logp_np, E, packed)
    r = _oracle(ids_np, logp_np, to_np(inp["E"]), to_np(inp["W_in"]), to_np(inp["W_out"]))
    _check(g, plain, r, logp_np, 0.0, MARGIN, f"cfg{cfg_index}")
    err = float(np.abs(plain["S"].astype(np.float64) - r["S"]).max())
    print(f"  max |S fp32 - S oracle| = {err:.3g}; re-scored decisions: "
          f"{int((g['rescored'] > 0).sum())} of {g['rescored'].size}", flush=True)
    assert err <= MARGIN / 2


def test_certified_reuses_workspace(lib):
    """Every call leaves the workspace ready for the next: three calls, then a smaller batch."""
    N, B, K, d = 8, 16, 16, 64
    ws = lib.score_walk_certified_workspace(N, B, K)
    for call, n in enumerate([N, N, N, 3]):
        E, W_in, W_out, ids, logp, ao = _twin_case(n, B, K, d, anchor=call % 2 == 1, seed=call)
        packed = lib.pack_weights(torch.from_numpy(W_in).cuda(), torch.from_numpy(W_out).cuda())
        g = _run_cert(lib, ids, logp, E.cuda(), packed, ao, workspace=ws)
        r = _oracle(ids, logp, to_np(E), W_in, W_out, ao)
        assert_equal(g["draft"], r["draft"], f"call {call} draft")
        assert_close(g["logq"], r["logq"], f"call {call} logq")
    assert int(ws[:256].view(torch.int32)[:N].abs().sum()) == 0, "counters back at zero"
