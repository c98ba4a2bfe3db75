"""GPU parity of the scoring-Transformer stand-in (lilicorr_scorer_pack / lilicorr_scorer_forward)
against the fp64 oracle (oracle/scorer.py) on the same seeded inputs.

Tolerances. Every matrix-core input is rounded to bf16 on both sides, but the GPU forms the
values it rounds in fp32, so a value within its fp32 error of a bf16 rounding boundary rounds the
other way (one bf16 ulp, 2^-8 relative), and each such flip perturbs everything downstream,
where more values cross boundaries. An fp32 emulation of the same rounding points (fp32 sums in a
different order) against the oracle, on these shapes, gives at most:
    attention block alone (w_2 = 0, one layer):  max |err| 1.9e-3, mean 2.5e-5
    feed-forward block alone (w_o = 0):          max |err| 2.3e-3, mean 6.3e-6
    two full layers:                             max |err| 1.03e-2, mean 1.46e-3
for outputs up to ~7 in magnitude. The bounds below allow a few times that; the block-alone mean
bounds also sit well under the mean effect of leaving out the rounding points (>= 4.4e-4 and
>= 1.07e-3), so a missing or extra rounding point fails them. Plumbing cases (no layers, zero
output maps) are bit-exact.
"""
import numpy as np
import pytest
import torch

import workloads
from oracle import scorer as osc

pytestmark = pytest.mark.gpu

TOL = {"attn": (8e-3, 1.5e-4), "ffn": (8e-3, 5e-5), "full": (4e-2, 3e-3)}

CASES = [
    # several GEMM row tiles with a ragged tail (M = 105), small width
    workloads.ScorerConfig(N=3, S=5, K=7, H=256, heads=2, F=384),
    # the paper's widths, K = 16 (M = 480: 3 full row tiles + a 96-row tail)
    workloads.ScorerConfig(N=2, S=15, K=16),
    # the paper's K = 8
    workloads.ScorerConfig(N=4, S=15, K=8),
    # the largest lattice one workgroup holds (L = 256)
    workloads.ScorerConfig(N=2, S=16, K=16),
    # one node per request (L = 1), and one slot of several candidates
    workloads.ScorerConfig(N=3, S=1, K=1, H=512, heads=4, F=256),
    workloads.ScorerConfig(N=2, S=1, K=9, H=256, heads=2, F=128),
]


def _bits(t):
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def _oracle_layers(layers):
    return [osc.layer_from_arrays(_bits(l["w_qkv"]), _bits(l["w_o"]), _bits(l["w_1"]),
                                  _bits(l["w_2"]), l["g_attn"].numpy(), l["g_ffn"].numpy(),
                                  l["dist_bias"].numpy(), l["same_bias"].numpy()) for l in layers]


def _variant(layers, mode):
    if mode == "attn":
        return [dict(layers[0], w_2=torch.zeros_like(layers[0]["w_2"]))]
    if mode == "ffn":
        return [dict(layers[0], w_o=torch.zeros_like(layers[0]["w_o"]))]
    return layers


def _gpu(lib, X, layers, sc):
    dev = [{k: v.cuda() for k, v in l.items()} for l in layers]
    packed = lib.scorer_pack(dev, sc.S)
    Xg = X.cuda().clone()
    lib.scorer_forward(Xg, packed, sc.S, sc.K, sc.heads, sc.F, len(layers))
    torch.cuda.synchronize()
    return Xg.cpu().numpy().astype(np.float64)


def _check(g, r, mode, what):
    tmax, tmean = TOL[mode]
    d = np.abs(g - r)
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    assert d.max() <= tmax, f"{what}: max |err| {d.max():.3e} > {tmax}"
    assert d.mean() <= tmean, f"{what}: mean |err| {d.mean():.3e} > {tmean}"


@pytest.mark.parametrize("mode", ["attn", "ffn", "full"])
@pytest.mark.parametrize("sc", CASES, ids=lambda s: f"N{s.N}S{s.S}K{s.K}H{s.H}F{s.F}")
def test_scorer_matches_oracle(lib, sc, mode):
    print(f"scorer {mode} N={sc.N} S={sc.S} K={sc.K} H={sc.H} F={sc.F}", flush=True)
    inp = workloads.make_scorer_inputs(sc)
    layers = _variant(inp["layers"], mode)
    g = _gpu(lib, inp["X"], layers, sc)
    r = osc.scorer_forward(inp["X"].numpy(), _oracle_layers(layers), sc.S, sc.K, sc.heads)
    _check(g, r, mode, f"{mode} {sc}")


def test_scorer_headline_all_requests(lib):
    """The headline shape (64 requests of 15 x 16 candidates, width 1024, two layers) in one call,
    every request checked against the oracle (run eight requests at a time)."""
    sc = workloads.SCORER_HEADLINE
    print(f"scorer headline {sc}", flush=True)
    inp = workloads.make_scorer_inputs(sc)
    g = _gpu(lib, inp["X"], inp["layers"], sc)
    ol = _oracle_layers(inp["layers"])
    r = np.concatenate([osc.scorer_forward(inp["X"][n:n + 8].numpy(), ol, sc.S, sc.K, sc.heads)
                        for n in range(0, sc.N, 8)])
    _check(g, r, "full", "headline, all 64 requests")


def test_scorer_plumbing_exact(lib):
    sc = workloads.ScorerConfig(N=2, S=3, K=5, H=256, heads=2, F=256)
    inp = workloads.make_scorer_inputs(sc)
    X = inp["X"].numpy().astype(np.float64)
    # no layers: X untouched
    dev = [{k: v.cuda() for k, v in l.items()} for l in inp["layers"]]
    packed = lib.scorer_pack(dev, sc.S)
    Xg = inp["X"].cuda().clone()
    lib.scorer_forward(Xg, packed, sc.S, sc.K, sc.heads, sc.F, 0)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(Xg.cpu().numpy(), inp["X"].numpy())
    # zero output maps: both residual updates add exact zeros
    zero = [dict(l, w_o=torch.zeros_like(l["w_o"]), w_2=torch.zeros_like(l["w_2"]))
            for l in inp["layers"]]
    np.testing.assert_array_equal(_gpu(lib, inp["X"], zero, sc), X)


def test_scorer_within_slot_permutation(lib):
    """Permuting candidates within their slots permutes the outputs (up to the bf16 noise of a
    different summation order over keys)."""
    sc = workloads.ScorerConfig(N=2, S=15, K=16)
    inp = workloads.make_scorer_inputs(sc)
    rng = np.random.default_rng(9)
    perm = torch.from_numpy(np.concatenate([s * sc.K + rng.permutation(sc.K) for s in range(sc.S)]))
    a = _gpu(lib, inp["X"], inp["layers"], sc)[:, perm.numpy()]
    b = _gpu(lib, inp["X"][:, perm].contiguous(), inp["layers"], sc)
    _check(a, b, "full", "within-slot permutation")


def test_scorer_rejects_bad_sizes(lib):
    sc = workloads.ScorerConfig(N=1, S=3, K=4, H=256, heads=2, F=256)
    inp = workloads.make_scorer_inputs(sc)
    dev = [{k: v.cuda() for k, v in l.items()} for l in inp["layers"]]
    packed = lib.scorer_pack(dev, sc.S)
    X = inp["X"].cuda()
    with pytest.raises(lib.LilicorrError):  # L = S * K above 256
        lib.scorer_forward(torch.zeros(1, 3 * 100, 256, device="cuda"), packed, 3, 100, 2, 256, 2)
    with pytest.raises(lib.LilicorrError):  # heads * 128 != H
        lib.scorer_forward(X, packed, sc.S, sc.K, 4, sc.F, 2)
    with pytest.raises(lib.LilicorrError):  # workspace too small
        lib.scorer_forward(X, packed, sc.S, sc.K, sc.heads, sc.F, 2,
                           workspace=torch.empty(16, dtype=torch.uint8, device="cuda"))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(X.cpu().numpy(), inp["X"].numpy())
