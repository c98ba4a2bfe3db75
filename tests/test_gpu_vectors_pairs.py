"""GPU parity of steps 2-3 (candidate vectors, pair scores) against the oracle.

Each GPU call gets exactly the oracle's inputs: the candidate ids for step 2, the oracle's own
unit vectors for step 3. Vectors: |gpu - oracle| <= 1e-5 per component (components are at most 1
in magnitude; fp32 accumulation of d bf16-exact products). Scores: 1e-5 * max(1, |S|).
"""
import numpy as np
import pytest
import torch

import oracle
from parity import assert_close, to_np

pytestmark = pytest.mark.gpu


def _gpu_vectors(lib, ids_np, E_cpu, W_in, W_out):
    packed = lib.pack_weights(W_in.cuda(), W_out.cuda())
    iv, ov = lib.candidate_vectors(torch.from_numpy(ids_np).cuda(), E_cpu.cuda(), packed)
    torch.cuda.synchronize()
    return to_np(iv), to_np(ov)


@pytest.mark.parametrize("cfg_index", [0, 1, 2, 3, 4])
def test_vectors_configs(lib, cfg_inputs, cfg_index):
    cfg, inp = cfg_inputs(cfg_index)
    print(f"vectors config {cfg_index} {cfg.name}", flush=True)
    rng = np.random.default_rng(cfg_index)
    # candidate ids of the config's shape (the parity of the ids themselves is step 1's test)
    ids = rng.integers(0, cfg.V, size=(cfg.N, cfg.B, cfg.K)).astype(np.int32)
    giv, gov = _gpu_vectors(lib, ids, inp["E"], inp["W_in"], inp["W_out"])
    E = to_np(inp["E"])
    W_in, W_out = to_np(inp["W_in"]), to_np(inp["W_out"])
    M = cfg.N * cfg.B * cfg.K
    flat = ids.reshape(M)
    sample = np.arange(M) if M <= 4096 else np.unique(
        np.concatenate([[0, M - 1], rng.choice(M, 1500, replace=False)]))
    riv, rov = oracle.candidate_vectors(flat[sample][None, None], E, W_in, W_out)
    d = cfg.d
    assert_close(giv.reshape(M, d)[sample], riv.reshape(-1, d), f"cfg{cfg_index} in_vec")
    assert_close(gov.reshape(M, d)[sample], rov.reshape(-1, d), f"cfg{cfg_index} out_vec")


@pytest.mark.parametrize("d,K,N,B,e_dtype", [
    (16, 1, 1, 1, "bf16"), (48, 5, 2, 3, "bf16"), (64, 7, 3, 5, "bf16"), (1024, 3, 2, 4, "bf16"),
    (512, 32, 1, 9, "bf16"), (96, 4, 2, 2, "f32"), (1024, 2, 1, 3, "f32"), (16, 3, 1, 2, "f32"),
    # padded column groups and k-blocks: d = 80 (5 -> 8 column blocks, 3 -> 4 k-blocks),
    # d = 272 (17 -> 20, 9 -> 10), d = 1008 (63 -> 64, 32)
    (80, 9, 3, 7, "bf16"), (272, 16, 2, 5, "bf16"), (1008, 4, 2, 3, "bf16"),
    # enough rows for the 128-row tiles (M = 131072)
    (64, 32, 64, 64, "bf16"),
])
def test_vectors_shapes(lib, d, K, N, B, e_dtype):
    print(f"vectors d={d} K={K} N={N} B={B} {e_dtype}", flush=True)
    rng = np.random.default_rng(d + K)
    V = 300
    E32 = (rng.standard_normal((V, d)) * 0.05).astype(np.float32)
    E32[7] = 0.0  # a zero embedding maps to a zero vector
    W_in = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    W_out = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    ids = rng.integers(0, V, size=(N, B, K)).astype(np.int32)
    ids.reshape(-1)[0] = 7
    E = torch.from_numpy(E32).to(torch.bfloat16) if e_dtype == "bf16" else torch.from_numpy(E32)
    giv, gov = _gpu_vectors(lib, ids, E, torch.from_numpy(W_in), torch.from_numpy(W_out))
    riv, rov = oracle.candidate_vectors(ids, to_np(E), W_in, W_out)
    assert_close(giv, riv, "in_vec")
    assert_close(gov, rov, "out_vec")
    assert (giv.reshape(-1, d)[0] == 0).all()


@pytest.mark.parametrize("d,N,B,K", [(512, 40, 31, 33), (496, 40, 31, 33),
                                     (512, 70, 31, 31), (464, 70, 31, 31), (512, 64, 32, 32),
                                     (512, 16, 32, 32)])
def test_vectors_persistent_tiles(lib, d, N, B, K):
    """The persistent kernel at 448 < d <= 512, which copies the next tile's rows into LDS while
    the current tile's products run (128-row tiles, each side a tile of its own): 40 x 31 x 33
    rows give 640 tiles (a ragged last tile of 88 rows), 70 x 31 x 31 rows 1052 (a ragged last
    tile of 70), 64 x 32 x 32 rows exactly 1024 (four per compute unit) and 16 x 32 x 32 rows 256
    (one per compute unit, the fewest that take this kernel). d = 496 and 464 leave the end of
    every row copy outside the row. Ids outside [0, V) give zero vectors, in the
    first tiles (whose ids are read before the loop) and in late ones (whose ids are copied while
    an earlier tile runs); the oracle takes the in-range rows."""
    V = 3000
    print(f"vectors persistent d={d} M={N * B * K}", flush=True)
    rng = np.random.default_rng(d + N)
    E32 = (rng.standard_normal((V, d)) * 0.05).astype(np.float32)
    E32[7] = 0.0
    W_in = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    W_out = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    ids = rng.integers(0, V, size=(N, B, K)).astype(np.int32)
    M = N * B * K
    flat = ids.reshape(M)
    flat[0], flat[M - 1], flat[5000], flat[M - 30], flat[M - 200] = 7, 7, -1, V, -5
    E = torch.from_numpy(E32).to(torch.bfloat16)
    giv, gov = _gpu_vectors(lib, ids, E, torch.from_numpy(W_in), torch.from_numpy(W_out))
    giv, gov = giv.reshape(M, d), gov.reshape(M, d)
    for r in (5000, M - 30, M - 200):
        assert (giv[r] == 0).all() and (gov[r] == 0).all(), f"row {r} of an out-of-range id"
    sample = np.unique(np.concatenate([np.arange(64), np.arange(M - 64, M),
                                       rng.choice(M, 700, replace=False)]))
    sample = sample[(flat[sample] >= 0) & (flat[sample] < V)]
    riv, rov = oracle.candidate_vectors(flat[sample][None, None], to_np(E), W_in, W_out)
    assert_close(giv[sample], riv.reshape(-1, d), f"d={d} in_vec")
    assert_close(gov[sample], rov.reshape(-1, d), f"d={d} out_vec")
    assert (giv[0] == 0).all() and (giv[M - 1] == 0).all()


def test_vectors_identity_weights(lib):
    d, V = 64, 50
    rng = np.random.default_rng(9)
    E = torch.from_numpy((rng.standard_normal((V, d))).astype(np.float32)).to(torch.bfloat16)
    eye = torch.eye(d)
    ids = np.arange(V, dtype=np.int32).reshape(1, 5, 10)
    giv, gov = _gpu_vectors(lib, ids, E, eye, eye)
    Ef = to_np(E.float()).astype(np.float64)
    expect = Ef / np.linalg.norm(Ef, axis=1, keepdims=True)
    assert_close(giv.reshape(V, d), expect, "identity in")
    assert_close(gov.reshape(V, d), expect, "identity out")


@pytest.mark.parametrize("N,B,K,d,anchor", [
    (1, 2, 1, 16, False), (2, 3, 3, 48, True), (4, 16, 16, 256, True), (2, 16, 32, 512, False),
    (1, 5, 64, 1024, True), (3, 1, 8, 64, True), (2, 4, 17, 144, True),
    (2, 3, 40, 80, True), (1, 3, 64, 1008, False), (3, 4, 33, 208, False),
])
def test_pair_scores_shapes(lib, N, B, K, d, anchor):
    print(f"pairs N={N} B={B} K={K} d={d} anchor={anchor}", flush=True)
    rng = np.random.default_rng(N * 1000 + K)
    iv = rng.standard_normal((N, B, K, d)).astype(np.float32)
    ov = rng.standard_normal((N, B, K, d)).astype(np.float32)
    iv /= np.linalg.norm(iv, axis=-1, keepdims=True)
    ov /= np.linalg.norm(ov, axis=-1, keepdims=True)
    iv[0, 0, 0] = 0.0  # a zero vector scores 0
    ao = rng.standard_normal((N, d)).astype(np.float32) if anchor else None
    S, S0 = lib.pair_scores(torch.from_numpy(iv).cuda(), torch.from_numpy(ov).cuda(),
                            torch.from_numpy(ao).cuda() if anchor else None, 8.0)
    torch.cuda.synchronize()
    rS, rS0 = oracle.pair_scores(iv, ov, ao, 8.0)
    if B > 1:
        assert_close(to_np(S), rS, "S")
        assert np.abs(to_np(S)).max() <= 8.0 * (1 + 4 * 2.0 ** -24)
    if anchor:
        assert_close(to_np(S0), rS0, "S0")
        assert to_np(S0)[0, 0] == 0.0


@pytest.mark.parametrize("cfg_index", [1, 3, 4])
def test_pair_scores_configs(lib, cfg_inputs, cfg_index):
    cfg, inp = cfg_inputs(cfg_index)
    N = min(cfg.N, 8)
    print(f"pairs config {cfg_index} on {N} requests", flush=True)
    rng = np.random.default_rng(cfg_index)
    ids = rng.integers(0, cfg.V, size=(N, cfg.B, cfg.K)).astype(np.int32)
    iv, ov = oracle.candidate_vectors(ids, to_np(inp["E"]), to_np(inp["W_in"]), to_np(inp["W_out"]))
    S, _ = lib.pair_scores(torch.from_numpy(iv).cuda(), torch.from_numpy(ov).cuda(), None, 8.0)
    torch.cuda.synchronize()
    rS, _ = oracle.pair_scores(iv, ov, None, 8.0)
    assert_close(to_np(S), rS, f"cfg{cfg_index} S")
