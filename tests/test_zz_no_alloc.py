"""The allocation-free fused pass (lilicorr_score_walk_noalloc) against lilicorr_score_walk.

For callers that cannot allocate: the pass's counters and table live in the library's per-GPU
scratch array. Through the raw C ABI, two calls in a row (the second with a smaller batch, so the
scratch holds the first call's data) must give what lilicorr_score_walk gives on the same inputs:
draft and choice bit-exact, logq and S within 1e-5 * max(1, |ref|) (the same kernels run, so in
practice bit-identical). A call that needs more than the scratch holds is rejected.
"""
import numpy as np
import pytest
import torch

from parity import assert_close, assert_equal, to_np

pytestmark = pytest.mark.gpu


def _inputs(rng, N, B, K, d, V):
    E = torch.from_numpy((rng.standard_normal((V, d)) * 0.05).astype(np.float32)).to(torch.bfloat16)
    W_in = torch.from_numpy((rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32))
    W_out = torch.from_numpy((rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32))
    ids = torch.from_numpy(rng.integers(0, V, size=(N, B, K)).astype(np.int32))
    logp = torch.from_numpy(-np.sort(rng.random((N, B, K)) * 4, axis=-1).astype(np.float32))
    return E.cuda(), W_in.cuda(), W_out.cuda(), ids.cuda(), logp.cuda()


def _noalloc(lib, ids, logp, E, packed, lam=0.0):
    N, B, K = ids.shape
    V, d = E.shape
    draft = torch.full((N, B), -7, dtype=torch.int32, device="cuda")
    choice = torch.full((N, B), -7, dtype=torch.int32, device="cuda")
    logq = torch.full((N, B), float("nan"), dtype=torch.float32, device="cuda")
    S = torch.full((N, max(B - 1, 1), K, K), float("nan"), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    lib.lilicorr_score_walk_noalloc(ids.data_ptr(), logp.data_ptr(), E.data_ptr(), lib.BF16, V, d,
                                    packed.data_ptr(), None, N, B, K, 8.0, lam, S.data_ptr(), None,
                                    draft.data_ptr(), choice.data_ptr(), logq.data_ptr(), stream)
    torch.cuda.synchronize()
    return dict(draft=to_np(draft), choice=to_np(choice), logq=to_np(logq), S=to_np(S))


def test_noalloc_matches_workspace_pass_twice(lib):
    rng = np.random.default_rng(11)
    d, V = 256, 3000
    for call, (N, B, K, lam) in enumerate([(64, 16, 16, 0.0), (5, 9, 8, 0.5)]):
        print(f"noalloc call {call}: N={N} B={B} K={K}", flush=True)
        E, W_in, W_out, ids, logp = _inputs(rng, N, B, K, d, V)
        packed = lib.pack_weights(W_in, W_out)
        g = _noalloc(lib, ids, logp, E, packed, lam)
        d_ref, c_ref, q_ref, S_ref, _ = lib.score_walk(ids, logp, E, packed, None, 8.0, lam,
                                                       scores=True)
        torch.cuda.synchronize()
        assert_equal(g["choice"], to_np(c_ref), f"call {call} choice")
        assert_equal(g["draft"], to_np(d_ref), f"call {call} draft")
        assert_close(g["logq"], to_np(q_ref), f"call {call} logq")
        assert_close(g["S"], to_np(S_ref), f"call {call} S")


def test_noalloc_rejects_what_the_scratch_cannot_hold(lib):
    # 5000 requests of 16 x 16 need 5000 * 241 * 8 bytes of table: more than the 8 MiB scratch
    N, B, K = 5000, 16, 16
    assert lib.lilicorr_score_walk_workspace_bytes(N, B, K) > 8 << 20
    x = torch.zeros(16, dtype=torch.int32, device="cuda")
    rc = lib.load_library().lilicorr_score_walk_noalloc(
        x.data_ptr(), x.data_ptr(), x.data_ptr(), lib.BF16, 100, 256, x.data_ptr(), None, N, B,
        K, 8.0, 0.0, None, None, x.data_ptr(), None, None, torch.cuda.current_stream().cuda_stream)
    assert rc == -4
