"""GPU parity of step 1 (lilicorr_topk) against the oracle: ids bit-exact, logp within 1e-5.

Full-row comparison at configs 0-2; at configs 3-4 (full size, the benchmark's launch
configuration) every row is computed on the GPU and a deterministic sample of rows is compared
with the oracle one row at a time. Edge cases: ragged and tiny vocabularies, K = 1 and K = 64,
exact ties, signed zeros, -inf, rows split over several workgroups, fp32 and bf16 logits.
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
def test_topk_full_size_sampled_rows(lib, cfg_inputs, cfg_index):
    cfg, inp = cfg_inputs(cfg_index)
    print(f"topk config {cfg_index} {cfg.name}", flush=True)
    R = cfg.N * cfg.B
    rng = np.random.default_rng(cfg_index)
    rows = sorted(set([0, 1, 2, R - 1] + rng.choice(R, 28, replace=False).tolist()))
    _check_rows(lib, inp["logits"], cfg.K, rows, f"cfg{cfg_index}")


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
    (1, 16, 151936, 8, "normal"),  # few rows: split over many workgroups + merge kernel
    (1, 1, 262144, 64, "ties"),
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
