"""GPU parity of step 1 (lilicorr_topk) against the oracle: ids bit-exact, logp within 1e-5.

Every row of every workload: configs 0-2 directly, configs 3-4 (full size, the benchmark's
launch configuration) against the oracle chain of every request, computed on a thread pool.
Edge cases: ragged and tiny vocabularies, K = 1 and K = 64, exact ties, signed zeros, -inf, rows
split over several workgroups, fp32 and bf16 logits. Also: forced expiry of the kernel's bounded
waits (reported, never silent), bit-identical repeated calls, and the vocabulary-sharded layout
(per-shard top-K merged on the host) against the unsharded result.
"""
import numpy as np
import pytest
import torch

import oracle
from parity import assert_close, assert_equal, to_np

pytestmark = pytest.mark.gpu


def _run(lib, logits_cpu, K):
    x = logits_cpu.cuda()
    ids, logp = lib.topk(x, K)
    torch.cuda.synchronize()
    return to_np(ids), to_np(logp)


def _check_rows(lib, logits_cpu, K, rows=None, what=""):
    gi, gl = _run(lib, logits_cpu, K)
    N, B, V = logits_cpu.shape
    x = to_np(logits_cpu).reshape(N * B, V)
    gi = gi.reshape(N * B, K)
    gl = gl.reshape(N * B, K)
    rows = range(N * B) if rows is None else rows
    for r in rows:
        ri, rl = oracle.topk(x[r][None, None], K)
        assert_equal(gi[r], ri[0, 0], f"{what} ids row {r}")
        assert_close(gl[r], rl[0, 0], f"{what} logp row {r}")


@pytest.mark.parametrize("cfg_index", [0, 1, 2])
def test_topk_configs_full(lib, cfg_inputs, cfg_index):
    cfg, inp = cfg_inputs(cfg_index)
    print(f"topk config {cfg_index} {cfg.name}", flush=True)
    gi, gl = _run(lib, inp["logits"], cfg.K)
    ri, rl = oracle.topk(to_np(inp["logits"]), cfg.K)
    assert_equal(gi, ri, f"cfg{cfg_index} ids")
    assert_close(gl, rl, f"cfg{cfg_index} logp")


@pytest.mark.parametrize("cfg_index", [3, 4])
def test_topk_full_size_all_rows(lib, cfg_inputs, oracle_chain, cfg_index):
    cfg, inp = cfg_inputs(cfg_index)
    print(f"topk config {cfg_index} {cfg.name}", flush=True)
    gi, gl = _run(lib, inp["logits"], cfg.K)
    r = oracle_chain(cfg_index)
    assert_equal(gi, r["ids"], f"cfg{cfg_index} ids ({cfg.N * cfg.B} rows)")
    assert_close(gl, r["logp"], f"cfg{cfg_index} logp")


def _bf16(x):
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16)


EDGE = [
    # (N, B, V, K, kind)
    (1, 1, 1, 1, "normal"),
    (1, 2, 7, 7, "normal"),
    (2, 3, 63, 5, "normal"),
    (1, 4, 1000, 64, "normal"),
    (2, 2, 32001, 16, "normal"),
    (1, 3, 32001, 1, "normal"),
    (3, 5, 70001, 33, "ties"),
    (1, 2, 5000, 8, "equal"),
    (1, 2, 3000, 20, "zeros"),
    (2, 2, 4099, 10, "neginf"),
    (1, 16, 151936, 8, "normal"),  # few rows: short segments of 8192 + merge kernel
    (1, 1, 262144, 64, "ties"),
    # short segments with exact ties at the threshold (lane maxima all equal: the id search)
    (1, 2, 20000, 8, "equal"),
    (1, 2, 20000, 20, "zeros"),
    (2, 2, 20001, 10, "neginf"),
    (1, 3, 30000, 12, "maskblock"),  # whole segments at -inf next to finite ones
    (1, 1, 20000, 64, "ties"),
    # a split that leaves rows*segments above one round: streaming segments + merge
    (2, 16, 151936, 16, "normal"),
    # more than 2048 partial keys per row: the merge kernel's list-merging path
    (1, 1, 300000, 64, "normal"),
    # the most rows the short-segment path takes (256 rows of two segments)
    (1, 256, 10000, 4, "normal"),
]


def _edge_logits(N, B, V, kind, seed):
    rng = np.random.default_rng(seed)
    if kind == "normal":
        x = rng.standard_normal((N, B, V)) * 2
    elif kind == "ties":
        x = rng.integers(-20, 21, size=(N, B, V)) * 0.25
    elif kind == "equal":
        x = np.full((N, B, V), 1.5)
    elif kind == "zeros":
        x = rng.choice([-0.0, 0.0, -1.0], size=(N, B, V))
    elif kind == "maskblock":
        x = rng.standard_normal((N, B, V))
        x[..., : V // 2] = -np.inf
        x[..., -1] = 3.0
    elif kind == "neginf":
        x = rng.standard_normal((N, B, V))
        x[rng.random((N, B, V)) < 0.9] = -np.inf
        x[..., 0] = 0.5
    return x.astype(np.float32)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("case", range(len(EDGE)))
def test_topk_edge_cases(lib, case, dtype):
    N, B, V, K, kind = EDGE[case]
    print(f"topk edge {EDGE[case]} {dtype}", flush=True)
    x = _edge_logits(N, B, V, kind, case)
    t = _bf16(x) if dtype == "bf16" else torch.from_numpy(x)
    _check_rows(lib, t, K, None, f"edge{case}-{dtype}")


def test_topk_workspace_shared_across_paths(lib):
    """One zero-filled workspace through short-segment, streaming split and whole-row calls in
    turn: every call matches the same call on a fresh workspace bit for bit."""
    shapes = [(1, 16, 151936, 8), (2, 16, 151936, 16), (1, 256, 10000, 4), (4, 16, 151936, 16),
              (1, 16, 151936, 8), (1, 3, 30000, 12)]
    need = max(lib.lilicorr_topk_workspace_bytes(N, B, V, K) for N, B, V, K in shapes)
    ws = torch.zeros((need + 15) // 16 * 16, dtype=torch.uint8, device="cuda")
    rng = np.random.default_rng(17)
    for i, (N, B, V, K) in enumerate(shapes):
        print(f"topk shared workspace call {i}: N={N} B={B} V={V} K={K}", flush=True)
        x = _bf16(rng.standard_normal((N, B, V)) * 2).cuda()
        ids, logp = lib.topk(x, K, workspace=ws)
        ids0, logp0 = lib.topk(x, K)
        torch.cuda.synchronize()
        assert_equal(to_np(ids), to_np(ids0), f"call {i} ids")
        assert_equal(to_np(logp), to_np(logp0), f"call {i} logp")
    assert lib.topk_wait_status(ws) == 0


def test_topk_sparse_finite_row(lib):
    # fewer than K finite logits: the -inf candidates follow by id
    x = np.full((1, 2, 600), -np.inf, np.float32)
    x[0, 0, [5, 400]] = [1.0, 2.0]
    x[0, 1, 599] = -3.0
    _check_rows(lib, torch.from_numpy(x), 4, None, "sparse")


def test_topk_rejects_bad_arguments(lib):
    x = torch.zeros(1, 1, 10, device="cuda", dtype=torch.bfloat16)
    with pytest.raises(lib.LilicorrError):
        lib.topk(x, 11)
    with pytest.raises(lib.LilicorrError):
        lib.topk(x, 65)
    with pytest.raises(lib.LilicorrError):
        lib.topk(x, 0)


# ---- confidence features from the same pass (lilicorr_topk_features) ---------------------------

def _features(lib, logits_cpu, K):
    ids, logp, feat = lib.topk(logits_cpu.cuda(), K, features=True)
    torch.cuda.synchronize()
    return to_np(ids), to_np(logp), to_np(feat)


@pytest.mark.parametrize("cfg_index", [0, 1, 2, 3, 4])
def test_topk_features_configs(lib, cfg_inputs, oracle_chain, cfg_index):
    """ids / logp as lilicorr_topk gives them; features against the oracle's from its own top-K
    (configs 0-1 split each row over several workgroups: the merge kernel writes them)."""
    cfg, inp = cfg_inputs(cfg_index)
    print(f"features config {cfg_index} {cfg.name}", flush=True)
    gi, gl, gf = _features(lib, inp["logits"], cfg.K)
    ri, rl = lib.topk(inp["logits"].cuda(), cfg.K)
    torch.cuda.synchronize()
    assert_equal(gi, to_np(ri), "ids with and without features")
    assert_equal(gl, to_np(rl), "logp with and without features")
    if cfg.N <= 16:
        oi, ol = oracle.topk(to_np(inp["logits"]), cfg.K)
        of = oracle.candidate_features(ol)
    else:  # every request, from the session's oracle chain
        r = oracle_chain(cfg_index)
        oi, of = r["ids"], r["feat"]
    assert_equal(gi, oi, "ids")
    assert_close(gf, of, "features")


@pytest.mark.parametrize("K", [1, 3, 64])
def test_topk_features_ties_and_small_k(lib, K):
    g = torch.Generator().manual_seed(K)
    x = torch.randn(2, 5, 3000, generator=g) * 3
    x[:, :, 10:20] = x.max(-1, keepdim=True).values + 1.0  # ten-way tie at the top
    xb = x.to(torch.bfloat16)
    gi, gl, gf = _features(lib, xb, K)
    oi, ol = oracle.topk(to_np(xb), K)
    assert_equal(gi, oi, "ids")
    assert_close(gf, oracle.candidate_features(ol), "features")
    assert (gf[..., :min(K, 10), 2] == 0).all()  # tied with the top: zero gap


# ---- bounded waits: expiry is reported, never silent ---------------------------------------------

def test_topk_wait_expiry_is_reported(lib):
    """With the spin limit forced to 0 from the host, the streaming kernel's consumer gives up at
    once (every wave still runs to the kernel's end) and the workspace's status word reports it;
    the query clears the word, and with the default limit the same call is correct and clean."""
    N, B, V, K = 64, 16, 24576, 16  # 1024 rows, one workgroup per row: the streaming kernel
    g = torch.Generator().manual_seed(5)
    x = (torch.randn(N, B, V, generator=g) * 2).to(torch.bfloat16)
    xd = x.cuda()
    ws = lib.topk_workspace(N, B, V, K)
    assert lib.topk_wait_status(ws) == 0
    lib.lilicorr_set_wait_limit(0)
    try:
        lib.topk(xd, K, workspace=ws)
        torch.cuda.synchronize()
    finally:
        lib.lilicorr_set_wait_limit(-1)
    assert lib.topk_wait_status(ws) == -6
    assert lib.topk_wait_status(ws) == 0
    gi, gl = lib.topk(xd, K, workspace=ws)
    assert lib.topk_wait_status(ws) == 0
    ri, rl = oracle.topk(to_np(x), K)
    assert_equal(to_np(gi), ri, "ids after the forced expiry")
    assert_close(to_np(gl), rl, "logp after the forced expiry")


def test_topk_logp_is_deterministic(lib, cfg_inputs):
    """The exp sums' reference depends on each producer's own tiles only, so repeated calls give
    bit-identical log-probabilities (stress workload: planted peaks move the threshold early)."""
    cfg, inp = cfg_inputs(4)
    x = inp["logits"].cuda()
    a = [to_np(t) for t in lib.topk(x, cfg.K)]
    for _ in range(3):
        b = [to_np(t) for t in lib.topk(x, cfg.K)]
        assert_equal(b[0], a[0], "ids of repeated calls")
        assert_equal(b[1], a[1], "logp of repeated calls")


# ---- the vocabulary-sharded layout on one GPU ----------------------------------------------------

def test_topk_vocabulary_shards_merge(lib, cfg_inputs, oracle_chain):
    """What a tensor-parallel LM head over 8 GPUs would hand this path: each shard holds V/8 =
    18,992 columns of every slot. Each shard's lilicorr_topk runs on its own slice; the exchange
    the sharded design needs per slot is the shard's K (id + base, logit) keys and its
    log-sum-exp (recovered here from the shard's top key: lse_shard = x[id_0] - logp_shard[0]).
    Merged (keys by value desc, global id asc; lse = logsumexp over shards), they must equal the
    unsharded result of the oracle chain: ids bit-exact, logp within tolerance."""
    cfg, inp = cfg_inputs(3)
    x = inp["logits"]  # [64, 16, 151936] bf16
    N, B, V, K = cfg.N, cfg.B, cfg.V, cfg.K
    P = 8
    w = V // P
    assert w * P == V
    xb = to_np(x)  # bf16 bit patterns

    def values(gid):  # the logits at global ids, widened exactly
        bits = np.take_along_axis(xb, gid, axis=-1).astype(np.uint32) << 16
        return bits.view(np.float32).astype(np.float64)

    keys_v, keys_id, lses = [], [], []
    for p in range(P):
        sl = x[:, :, p * w:(p + 1) * w].contiguous()
        gi, gl = _run(lib, sl, K)
        gid = gi.astype(np.int64) + p * w
        xv = values(gid)
        keys_v.append(xv)
        keys_id.append(gid)
        lses.append(xv[..., 0] - gl[..., 0].astype(np.float64))
    kv = np.concatenate(keys_v, -1)
    ki = np.concatenate(keys_id, -1)
    order = np.lexsort((ki, -kv), axis=-1)[..., :K]
    ids = np.take_along_axis(ki, order, -1).astype(np.int32)
    lse = np.logaddexp.reduce(np.stack(lses, -1), axis=-1)
    logp = (np.take_along_axis(kv, order, -1) - lse[..., None]).astype(np.float32)
    r = oracle_chain(3)
    assert_equal(ids, r["ids"], "merged shard ids")
    assert_close(logp, r["logp"], "merged shard logp")
