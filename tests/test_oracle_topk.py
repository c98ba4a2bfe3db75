"""Pins for the oracle's step 1 (vocabulary log-normalisation + top-K), CPU only.

The oracle sorts every index by (value desc, id asc) with qsort and sums exp in a plain loop;
these tests check it against independent routines (numpy lexsort, scipy logsumexp) and against
invariants the definitions fix (Sec. 3.2 candidate pool; implementation appendix, vocabulary-wide
normalisation fused with the top-K extraction).
"""
import numpy as np
import pytest
import torch
from scipy.special import logsumexp

import oracle
import workloads


def _bf16_bits(x: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).view(
        torch.int16).numpy().view(np.uint16)


def _bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


def _lexsort_topk(x: np.ndarray, K: int) -> np.ndarray:
    v = np.arange(x.shape[-1])
    return np.lexsort((v, -x.astype(np.float64)))[:K]


@pytest.mark.parametrize("seed", range(6))
def test_topk_matches_lexsort_with_heavy_ties(seed):
    rng = np.random.default_rng(seed)
    N, B, V, K = 2, 3, 257, 9
    # few distinct values -> many exact ties, plus signed zeros and -inf
    x = rng.choice(np.array([-2.0, -0.0, 0.0, 0.5, 1.0, 1.5, -np.inf], np.float32), size=(N, B, V))
    x[..., 0] = 1.5  # at least one finite value per slot
    ids, logp = oracle.topk(x, K)
    for n in range(N):
        for b in range(B):
            np.testing.assert_array_equal(ids[n, b], _lexsort_topk(x[n, b], K))


def test_logsumexp_against_scipy():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal((3, 4, 5000)) * 3).astype(np.float32)
    ids, logp = oracle.topk(x, 5)
    for n in range(3):
        for b in range(4):
            lse = logsumexp(x[n, b].astype(np.float64))
            expect = x[n, b, ids[n, b]].astype(np.float64) - lse
            np.testing.assert_allclose(logp[n, b], expect, rtol=0, atol=2e-6)


def test_full_vocabulary_normalises_and_is_a_permutation():
    rng = np.random.default_rng(2)
    V = 300
    x = (rng.standard_normal((1, 2, V)) * 2).astype(np.float32)
    ids, logp = oracle.topk(x, V)
    for b in range(2):
        assert sorted(ids[0, b].tolist()) == list(range(V))
        assert abs(np.exp(logp[0, b].astype(np.float64)).sum() - 1.0) < 1e-5


def test_invariants_sorted_distinct_nonpositive():
    rng = np.random.default_rng(3)
    x = rng.integers(-4, 5, size=(2, 5, 1000)).astype(np.float32)  # integer values: many ties
    K = 16
    ids, logp = oracle.topk(x, K)
    for n in range(2):
        for b in range(5):
            vals = x[n, b, ids[n, b]]
            assert len(set(ids[n, b].tolist())) == K
            for k in range(K - 1):
                assert vals[k] > vals[k + 1] or (vals[k] == vals[k + 1] and ids[n, b, k] < ids[n, b, k + 1])
            assert (logp[n, b] <= 0).all()
            assert (np.diff(logp[n, b]) <= 0).all()
            # nothing left out ranks above the K-th entry
            kth = (vals[-1], -ids[n, b, -1])
            rest = np.setdiff1d(np.arange(1000), ids[n, b])
            for v in rest:
                assert (x[n, b, v], -v) < kth


def test_signed_zero_ties_break_by_id():
    x = np.array([[[-0.0, 0.0, -0.0, -1.0]]], np.float32)
    ids, logp = oracle.topk(x, 3)
    assert ids[0, 0].tolist() == [0, 1, 2]


def test_bf16_input_equals_float_input_of_same_values():
    rng = np.random.default_rng(4)
    x32 = (rng.standard_normal((2, 3, 4001)) * 2).astype(np.float32)
    bits = _bf16_bits(x32)
    ids_a, logp_a = oracle.topk(bits, 7)
    ids_b, logp_b = oracle.topk(_bits_to_f32(bits), 7)
    np.testing.assert_array_equal(ids_a, ids_b)
    np.testing.assert_array_equal(logp_a, logp_b)


def test_single_finite_value_and_minus_inf():
    x = np.full((1, 1, 50), -np.inf, np.float32)
    x[0, 0, 17] = 3.0
    ids, logp = oracle.topk(x, 3)
    assert ids[0, 0].tolist() == [17, 0, 1]
    assert logp[0, 0, 0] == 0.0
    assert np.isneginf(logp[0, 0, 1:]).all()


def test_all_minus_inf_slot_is_rejected():
    x = np.full((1, 1, 10), -np.inf, np.float32)
    with pytest.raises(ValueError):
        oracle.topk(x, 2)


def test_tiny_config_planted_peak_is_rank_zero():
    cfg = workloads.config(0)
    logits = workloads.make_logits(cfg).numpy()
    ids, logp = oracle.topk(logits, cfg.K)
    # +6 over N(0,1) noise in V = 32000: the planted id tops its slot (statistical, seed 0)
    top = logits.argmax(-1)
    np.testing.assert_array_equal(ids[..., 0], top)
    assert (logits.max(-1) > 5.0).all()
