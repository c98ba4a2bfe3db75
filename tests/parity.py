"""Comparison helpers for GPU-vs-oracle parity tests (test infrastructure)."""
import numpy as np
import torch

# spec tolerance for fp32 outputs (log-probs, scores, log-likelihoods):
#   |gpu - oracle| <= 1e-5 * max(1, |oracle|)
RTOL = 1e-5


def to_np(t):
    if isinstance(t, torch.Tensor):
        t = t.detach().cpu()
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).numpy().view(np.uint16)
        return t.numpy()
    return np.asarray(t)


def assert_close(gpu, ref, what, tol=RTOL):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, f"{what}: shape {gpu.shape} vs {ref.shape}"
    both_inf = np.isinf(gpu) & np.isinf(ref) & (np.sign(gpu) == np.sign(ref))
    with np.errstate(invalid="ignore"):
        err = np.where(both_inf, 0.0, np.abs(gpu - ref))
    bound = tol * np.maximum(1.0, np.where(np.isinf(ref), 1.0, np.abs(ref)))
    bad = ~(err <= bound)
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} outside tolerance; first at "
                             f"{tuple(i)}: gpu {gpu[tuple(i)]!r} oracle {ref[tuple(i)]!r}; "
                             f"max err {np.nanmax(err):.3e}")


def assert_equal(gpu, ref, what):
    gpu = np.asarray(gpu)
    ref = np.asarray(ref)
    assert gpu.shape == ref.shape, f"{what}: shape {gpu.shape} vs {ref.shape}"
    bad = gpu != ref
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} differ; first at {tuple(i)}: "
                             f"gpu {gpu[tuple(i)]!r} oracle {ref[tuple(i)]!r}")


def oracle_threads() -> int:
    """Worker threads for the oracle (its C routines release the interpreter lock)."""
    import os

    return max(1, min(16, len(os.sched_getaffinity(0))))


def oracle_chain_all(cfg, inp, threads=None):
    """The oracle chain of every request of a workload, one request per task on a thread pool:
    top-K, candidate vectors, pair scores, then both decode rules on the oracle's own scores
    (greedy walk; exact max-path decode) and the confidence features of its top-K. Returns
    numpy arrays over all N requests."""
    import concurrent.futures

    import oracle

    lg, E = to_np(inp["logits"]), to_np(inp["E"])
    W_in, W_out = to_np(inp["W_in"]), to_np(inp["W_out"])
    N, B, K = cfg.N, cfg.B, cfg.K
    out = dict(ids=np.zeros((N, B, K), np.int32), logp=np.zeros((N, B, K), np.float32),
               S=np.zeros((N, B - 1, K, K), np.float32), draft=np.zeros((N, B), np.int32),
               choice=np.zeros((N, B), np.int32), logq=np.zeros((N, B), np.float32),
               vdraft=np.zeros((N, B), np.int32), vchoice=np.zeros((N, B), np.int32),
               vlogq=np.zeros((N, B), np.float32), vscore=np.zeros((N,), np.float32),
               feat=np.zeros((N, B, K, 5), np.float32))

    def one(n):
        ids, logp = oracle.topk(lg[n:n + 1], K)
        iv, ov = oracle.candidate_vectors(ids, E, W_in, W_out)
        S, S0 = oracle.pair_scores(iv, ov, None, 8.0)
        d, c, q = oracle.greedy_walk(S, S0, logp, ids)
        vd, vc, vq, vs = oracle.viterbi_walk(S, S0, logp, ids)
        for key, val in (("ids", ids), ("logp", logp), ("S", S), ("draft", d), ("choice", c),
                         ("logq", q), ("vdraft", vd), ("vchoice", vc), ("vlogq", vq),
                         ("vscore", vs), ("feat", oracle.candidate_features(logp))):
            out[key][n] = val[0]

    with concurrent.futures.ThreadPoolExecutor(threads or oracle_threads()) as ex:
        list(ex.map(one, range(N)))
    return out


def greedy_gap(S, S0, choice, n, t):
    """The top-2 gap of the greedy walk's node scores (lambda = 0) at request n, slot t, on the
    scores S / S0 along `choice`: how near that decision is to a tie."""
    if t == 0:
        z = S0[n] if S0 is not None else np.zeros(S.shape[-1])
    else:
        z = S[n, t - 1, choice[n, t - 1]]
    top = np.sort(np.asarray(z, np.float64))[::-1]
    return float(top[0] - top[1]) if top.size > 1 else float("inf")


def path_gap(S, S0, n, logp=None, lam=0.0):
    """The gap between the best and the second-best path score of Eq. (pathscore) of request n
    (with lambda * logp node terms when lam != 0), by a two-best dynamic program in double: how
    near the exact decode is to a tie."""
    Sn = np.asarray(S[n], np.float64)
    K = S.shape[-1]
    node = (lambda t: lam * np.asarray(logp[n, t], np.float64)) if lam else (lambda t: 0.0)
    first = (np.asarray(S0[n], np.float64) if S0 is not None else np.zeros(K)) + node(0)
    second = np.full(K, -np.inf)
    for t in range(Sn.shape[0]):
        cand = np.concatenate([first[:, None] + Sn[t], second[:, None] + Sn[t]], axis=0)
        cand = np.sort(cand, axis=0)[::-1]
        first, second = cand[0] + node(t + 1), cand[1] + node(t + 1)
    allv = np.sort(np.concatenate([first, second]))[::-1]
    return float(allv[0] - allv[1])
