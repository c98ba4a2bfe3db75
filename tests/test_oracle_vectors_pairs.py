"""Pins for the oracle's steps 2-3 (candidate vectors, pair scores), CPU only.

Step 2 stands in for the head's two linear heads, whose outputs are normalised to unit norm
(Sec. 3.2, implementation appendix): v = u / ||u||, u = E[id] W. Step 3 is Eq. (pair),
phi = sigma * cos(out_{s,k}, in_{s+1,k'}), with sigma = 8 (hyper-parameter table). Checked
against numpy fp64 matrix products, closed-form special cases, a hand-worked fixture and index
probes built from one-hot vectors.
"""
import os

import numpy as np
import pytest
import torch
import yaml

import oracle


def _bf16_bits(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).view(
        torch.int16).numpy().view(np.uint16)


def _bits_to_f32(b):
    return (b.astype(np.uint32) << 16).view(np.float32)


def _np_vectors(ids, E32, W):
    u = E32.astype(np.float64)[ids] @ W.astype(np.float64)
    n = np.linalg.norm(u, axis=-1, keepdims=True)
    return np.where(n > 0, u / np.where(n > 0, n, 1), 0.0)


@pytest.mark.parametrize("e_bf16", [False, True])
def test_vectors_match_numpy_fp64(e_bf16):
    rng = np.random.default_rng(0)
    V, d, N, B, K = 50, 48, 2, 3, 4
    E32 = rng.standard_normal((V, d)).astype(np.float32)
    W_in = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    W_out = (rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32)
    ids = rng.integers(0, V, size=(N, B, K)).astype(np.int32)
    E = _bf16_bits(E32) if e_bf16 else E32
    Ew = _bits_to_f32(E) if e_bf16 else E32
    iv, ov = oracle.candidate_vectors(ids, E, W_in, W_out)
    np.testing.assert_allclose(iv, _np_vectors(ids, Ew, W_in), rtol=0, atol=1e-7)
    np.testing.assert_allclose(ov, _np_vectors(ids, Ew, W_out), rtol=0, atol=1e-7)
    assert np.allclose(np.linalg.norm(iv.astype(np.float64), axis=-1), 1.0, atol=1e-6)


def test_vectors_identity_weight_and_orientation():
    rng = np.random.default_rng(1)
    V, d = 10, 16
    E = rng.standard_normal((V, d)).astype(np.float32)
    ids = np.arange(V, dtype=np.int32).reshape(1, 2, 5)
    eye = np.eye(d, dtype=np.float32)
    # W[i][j]: only input 0 feeds output 3, so u = (0, 0, 0, e_0, 0, ...)
    probe = np.zeros((d, d), np.float32)
    probe[0, 3] = 1.0
    iv, ov = oracle.candidate_vectors(ids, E, eye, probe)
    expect = E / np.linalg.norm(E.astype(np.float64), axis=1, keepdims=True)
    np.testing.assert_allclose(iv.reshape(V, d), expect, atol=1e-7)
    o = ov.reshape(V, d)
    assert (o[:, [j for j in range(d) if j != 3]] == 0).all()
    np.testing.assert_array_equal(o[:, 3], np.sign(E[:, 0]))


def test_vectors_zero_row_maps_to_zero():
    E = np.zeros((3, 16), np.float32)
    E[1] = 1.0
    W = np.eye(16, dtype=np.float32)
    iv, ov = oracle.candidate_vectors(np.array([[[0, 1]]], np.int32), E, W, W)
    assert (iv[0, 0, 0] == 0).all() and (ov[0, 0, 0] == 0).all()
    np.testing.assert_allclose(iv[0, 0, 1], 0.25, atol=1e-7)


def test_vectors_reject_out_of_range_id():
    E = np.ones((3, 16), np.float32)
    W = np.eye(16, dtype=np.float32)
    with pytest.raises(ValueError):
        oracle.candidate_vectors(np.array([[[0, 3]]], np.int32), E, W, W)


def test_pair_hand_fixture(golden_dir):
    g = yaml.safe_load(open(os.path.join(golden_dir, "walk_hand_cases.yaml")))["pair_2d"]
    out0 = np.array(g["out0"], np.float32)
    in1 = np.array(g["in1"], np.float32)
    K, d = out0.shape
    in_vec = np.zeros((1, 2, K, d), np.float32)
    out_vec = np.zeros((1, 2, K, d), np.float32)
    out_vec[0, 0] = out0
    in_vec[0, 1] = in1
    S, S0 = oracle.pair_scores(in_vec, out_vec, sigma=g["sigma"])
    assert S0 is None
    np.testing.assert_allclose(S[0, 0], np.array(g["S"]), rtol=0, atol=1e-6)


def test_pair_special_cases_and_bound():
    rng = np.random.default_rng(2)
    d = 32
    a = rng.standard_normal(d).astype(np.float32)
    b = rng.standard_normal(d).astype(np.float32)
    b_perp = (b - a * (a @ b) / (a @ a)).astype(np.float32)
    out_vec = np.zeros((1, 2, 3, d), np.float32)
    in_vec = np.zeros((1, 2, 3, d), np.float32)
    out_vec[0, 0, 0] = a
    in_vec[0, 1] = np.stack([3 * a, -0.5 * a, b_perp])
    S, _ = oracle.pair_scores(in_vec, out_vec)
    np.testing.assert_allclose(S[0, 0, 0], [8.0, -8.0, 0.0], atol=1e-5)
    # zero out vectors score 0
    assert (S[0, 0, 1:] == 0).all()
    # random vectors stay inside [-sigma, sigma] and match a numpy cosine
    N, B, K = 2, 5, 6
    iv = rng.standard_normal((N, B, K, d)).astype(np.float32)
    ov = rng.standard_normal((N, B, K, d)).astype(np.float32)
    S, _ = oracle.pair_scores(iv, ov, sigma=8.0)
    assert np.abs(S).max() <= 8.0
    o = ov[:, :-1].astype(np.float64)
    i = iv[:, 1:].astype(np.float64)
    o /= np.linalg.norm(o, axis=-1, keepdims=True)
    i /= np.linalg.norm(i, axis=-1, keepdims=True)
    ref = 8.0 * np.einsum("ntkd,ntjd->ntkj", o, i)
    np.testing.assert_allclose(S, ref, atol=2e-6)


def test_pair_indexing_with_one_hot_probes():
    # out[n][t][k] = e_{code(n,t,k)}, in[n][t][k'] = e_{code'(n,t,k')}: S is sigma exactly where
    # the codes agree, so any slip in n, t, k or k' indexing moves the ones
    N, B, K = 2, 4, 3
    d = 64
    rng = np.random.default_rng(3)
    oc = rng.integers(0, 6, size=(N, B, K))
    ic = rng.integers(0, 6, size=(N, B, K))
    ov = np.eye(d, dtype=np.float32)[oc]
    iv = np.eye(d, dtype=np.float32)[ic]
    anchor_code = rng.integers(0, 6, size=N)
    anchor = np.eye(d, dtype=np.float32)[anchor_code]
    S, S0 = oracle.pair_scores(iv, ov, anchor)
    for n in range(N):
        for t in range(B - 1):
            for k in range(K):
                for kk in range(K):
                    assert S[n, t, k, kk] == (8.0 if oc[n, t, k] == ic[n, t + 1, kk] else 0.0)
        for kk in range(K):
            assert S0[n, kk] == (8.0 if anchor_code[n] == ic[n, 0, kk] else 0.0)


def test_pair_single_slot_block_has_no_pairs():
    iv = np.ones((2, 1, 3, 16), np.float32)
    S, S0 = oracle.pair_scores(iv, iv, np.ones((2, 16), np.float32))
    assert S.shape == (2, 0, 3, 3)
    np.testing.assert_allclose(S0, 8.0, atol=1e-6)
