"""Pins of the scoring-Transformer oracle (oracle/scorer.py) to things other than itself:
library routines (torch's bf16 conversion, rms_norm, silu, scaled_dot_product_attention, all in
fp64), brute-force loops on tiny inputs, exact invariants of the layer (residual identity,
permutation equivariance within a slot, mirror symmetry of the slot-distance bias, per-head
column ownership) and the error bound of the bf16 rounding points."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as TF

import workloads
from oracle import scorer as osc


def _bits(t):
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def _layers(sc):
    inp = workloads.make_scorer_inputs(sc)
    layers = [osc.layer_from_arrays(_bits(l["w_qkv"]), _bits(l["w_o"]), _bits(l["w_1"]),
                                    _bits(l["w_2"]), l["g_attn"].numpy(), l["g_ffn"].numpy(),
                                    l["dist_bias"].numpy(), l["same_bias"].numpy())
              for l in inp["layers"]]
    return inp["X"].numpy().astype(np.float64), layers


SMALL = workloads.ScorerConfig(N=2, S=3, K=4, H=64, heads=4, F=96, layers=2, seed=3)


def test_bf16_round_matches_torch_on_fp32_values():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))).astype(np.float32)
    # exact ties: low 16 bits 0x8000, both mantissa parities
    ties = (rng.integers(0x3f000000, 0x41000000, 2000, dtype=np.uint32) & 0xFFFF0000) | 0x8000
    x = np.concatenate([x, ties.view(np.float32), -ties.view(np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(osc.bf16_round(x.astype(np.float64)), ref)


def test_bf16_round_directly_from_fp64():
    # ties go to the even 8-bit significand; a value just above a tie rounds up even where an fp32
    # intermediate would have lost the excess and rounded down
    assert osc.bf16_round(np.float64(1 + 2 ** -8)) == 1.0
    assert osc.bf16_round(np.float64(1 + 3 * 2 ** -8)) == 1 + 2 ** -6
    assert osc.bf16_round(np.float64(1 + 2 ** -8 + 2 ** -40)) == 1 + 2 ** -7
    assert osc.bf16_round(np.float64(-(1 + 2 ** -8 + 2 ** -40))) == -(1 + 2 ** -7)
    assert osc.bf16_round(np.float64(0.0)) == 0.0
    assert osc.bf16_round(np.float64(255.5)) == 256.0


def test_bf16_bits_to_f64():
    v = np.array([1.0, -2.5, 0.1, 3e-20, 7e30], np.float32)
    bits = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(osc.bf16_bits_to_f64(bits), ref)


def test_rms_norm_and_silu_match_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 64)) * 3
    g = 1 + 0.1 * rng.standard_normal(64)
    ref = TF.rms_norm(torch.from_numpy(x), (64,), torch.from_numpy(g), eps=osc.EPS).numpy()
    np.testing.assert_allclose(osc.rms_norm(x, g), ref, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(osc.silu(x), TF.silu(torch.from_numpy(x)).numpy(),
                               rtol=1e-13, atol=1e-13)


def _bias_loops(S, K, dist, same):
    L = S * K
    b = np.zeros((L, L))
    for i in range(L):
        for j in range(L):
            si, sj = i // K, j // K
            b[i, j] = dist[si - sj + S - 1] + (same if si == sj else 0.0)
    return b


def test_lattice_bias_brute_force():
    rng = np.random.default_rng(2)
    for S, K in [(1, 1), (3, 2), (5, 3), (15, 4)]:
        dist = rng.standard_normal(2 * S - 1)
        same = float(rng.standard_normal())
        np.testing.assert_array_equal(osc.lattice_bias(S, K, dist, same),
                                      _bias_loops(S, K, dist, same))


def test_attention_matches_sdpa():
    rng = np.random.default_rng(3)
    S, K, dh = 5, 4, 16
    L = S * K
    q, k, v = (rng.standard_normal((L, dh)) for _ in range(3))
    dist = rng.standard_normal(2 * S - 1)
    same = 0.7
    out = osc.lattice_attention(q, k, v, S, K, dist, same, exact=True)
    t = lambda a: torch.from_numpy(a)[None, None]
    ref = TF.scaled_dot_product_attention(t(q), t(k), t(v),
                                          attn_mask=t(_bias_loops(S, K, dist, same)))[0, 0]
    np.testing.assert_allclose(out, ref.numpy(), rtol=1e-12, atol=1e-12)


def test_attention_brute_force_loops():
    rng = np.random.default_rng(4)
    S, K, dh = 3, 2, 4
    L = S * K
    q, k, v = (rng.standard_normal((L, dh)) for _ in range(3))
    dist = [0.3, -1.1, 0.5, 0.9, -0.2]
    same = -0.4
    out = osc.lattice_attention(q, k, v, S, K, np.array(dist), same, exact=True)
    for i in range(L):
        w = []
        for j in range(L):
            dot = sum(q[i][c] * k[j][c] for c in range(dh)) / math.sqrt(dh)
            b = dist[i // K - j // K + S - 1] + (same if i // K == j // K else 0.0)
            w.append(math.exp(dot + b))
        tot = sum(w)
        for c in range(dh):
            assert abs(out[i][c] - sum(w[j] / tot * v[j][c] for j in range(L))) < 1e-12


def test_attention_rounding_point_within_bound():
    rng = np.random.default_rng(5)
    S, K, dh = 4, 4, 8
    L = S * K
    q, k, v = (rng.standard_normal((L, dh)) * 2 for _ in range(3))
    dist = rng.standard_normal(2 * S - 1)
    exact = osc.lattice_attention(q, k, v, S, K, dist, 0.2, exact=True)
    rounded = osc.lattice_attention(q, k, v, S, K, dist, 0.2, exact=False)
    z = q @ k.T / math.sqrt(dh) + _bias_loops(S, K, dist, 0.2)
    p = np.exp(z - z.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    bound = 2.0 ** -8 * (p @ np.abs(v)) + 1e-12
    assert np.all(np.abs(rounded - exact) <= bound)
    assert np.any(rounded != exact)


def _torch_layer(X, l, S, K, heads):
    """The same layer written with torch's fp64 library routines (no bf16 rounding)."""
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    X = t(X)
    N, L, H = X.shape
    dh = H // heads
    mask = torch.stack([t(_bias_loops(S, K, l["dist_bias"][h], float(l["same_bias"][h])))
                        for h in range(heads)])
    xn = TF.rms_norm(X, (H,), t(l["g_attn"]), eps=osc.EPS)
    qkv = xn @ t(l["w_qkv"])
    sp = lambda a: a.reshape(N, L, heads, dh).transpose(1, 2)
    q, k, v = sp(qkv[..., :H]), sp(qkv[..., H:2 * H]), sp(qkv[..., 2 * H:])
    o = TF.scaled_dot_product_attention(q, k, v, attn_mask=mask[None]).transpose(1, 2)
    X = X + o.reshape(N, L, H) @ t(l["w_o"])
    hn = TF.rms_norm(X, (H,), t(l["g_ffn"]), eps=osc.EPS)
    return (X + TF.silu(hn @ t(l["w_1"])) @ t(l["w_2"])).numpy()


def test_layer_matches_torch_composition():
    X, layers = _layers(SMALL)
    for l in layers:
        out = osc.scorer_layer(X, l, SMALL.S, SMALL.K, SMALL.heads, exact=True)
        np.testing.assert_allclose(out, _torch_layer(X, l, SMALL.S, SMALL.K, SMALL.heads),
                                   rtol=1e-11, atol=1e-11)
        X = out


def test_layer_rounding_points_move_little():
    X, layers = _layers(SMALL)
    a = osc.scorer_forward(X, layers, SMALL.S, SMALL.K, SMALL.heads, exact=True)
    b = osc.scorer_forward(X, layers, SMALL.S, SMALL.K, SMALL.heads)
    d = np.abs(a - b)
    assert d.max() < 0.05 and d.max() > 0


def test_zero_output_maps_are_identity():
    X, layers = _layers(SMALL)
    l = dict(layers[0], w_o=np.zeros_like(layers[0]["w_o"]), w_2=np.zeros_like(layers[0]["w_2"]))
    np.testing.assert_array_equal(osc.scorer_layer(X, l, SMALL.S, SMALL.K, SMALL.heads), X)


def test_within_slot_permutation_equivariance():
    X, layers = _layers(SMALL)
    S, K = SMALL.S, SMALL.K
    rng = np.random.default_rng(6)
    perm = np.concatenate([s * K + rng.permutation(K) for s in range(S)])
    a = osc.scorer_forward(X, layers, S, K, SMALL.heads)[:, perm]
    b = osc.scorer_forward(X[:, perm], layers, S, K, SMALL.heads)
    np.testing.assert_allclose(a, b, rtol=1e-9, atol=1e-9)


def test_slot_reversal_mirrors_distance_bias():
    X, layers = _layers(SMALL)
    S, K = SMALL.S, SMALL.K
    rev = np.concatenate([s * K + np.arange(K) for s in reversed(range(S))])
    mirrored = [dict(l, dist_bias=l["dist_bias"][:, ::-1].copy()) for l in layers]
    a = osc.scorer_forward(X, layers, S, K, SMALL.heads)[:, rev]
    b = osc.scorer_forward(X[:, rev], mirrored, S, K, SMALL.heads)
    np.testing.assert_allclose(a, b, rtol=1e-9, atol=1e-9)
    # and the bias is not symmetric, so the mirror is what makes them agree
    c = osc.scorer_forward(X[:, rev], layers, S, K, SMALL.heads)
    assert np.abs(a - c).max() > 1e-3


def test_head_owns_its_columns():
    X, layers = _layers(SMALL)
    H, heads = SMALL.H, SMALL.heads
    dh = H // heads
    l = dict(layers[0])
    w_qkv = l["w_qkv"].copy()
    w_qkv[:, 2 * H + dh:2 * H + 2 * dh] = 0.0           # head 1's value columns
    l.update(w_qkv=w_qkv, w_o=np.eye(H), w_2=np.zeros_like(l["w_2"]))
    delta = osc.scorer_layer(X, l, SMALL.S, SMALL.K, heads) - X
    assert np.all(delta[..., dh:2 * dh] == 0.0)
    assert np.all(np.abs(delta[..., :dh]).max(axis=-1) > 0)


@pytest.mark.parametrize("sc", [workloads.ScorerConfig(N=1, S=2, K=1, H=32, heads=2, F=32, layers=1),
                                workloads.ScorerConfig(N=1, S=1, K=3, H=32, heads=1, F=64, layers=1)])
def test_degenerate_lattices(sc):
    X, layers = _layers(sc)
    out = osc.scorer_forward(X, layers, sc.S, sc.K, sc.heads, exact=True)
    ref = X
    for l in layers:
        ref = _torch_layer(ref, l, sc.S, sc.K, sc.heads)
    np.testing.assert_allclose(out, ref, rtol=1e-11, atol=1e-11)
