"""GPU test: consecutive blocks on two streams.

The library keeps no state between calls beyond the caller's workspaces, so blocks of
independent batches may run concurrently on different streams, each with its own outputs and
workspaces (the benchmark's two-stream figure relies on this). Here four headline-shaped blocks
(the headline logits with their slots permuted) are launched alternately on two streams with no
synchronisation between them; every block's ids, log-probabilities and draft must equal, bit for
bit, what the same calls give one block at a time on one stream (whose parity with the oracle is
the other tests' subject).
"""
import numpy as np
import pytest
import torch

from parity import assert_equal, to_np

pytestmark = pytest.mark.gpu


def test_blocks_on_two_streams_match_one_stream(lib, cfg_inputs):
    cfg, inp = cfg_inputs(3)
    print("two streams, config 3, four blocks", flush=True)
    g = torch.Generator().manual_seed(5)
    E = inp["E"].cuda()
    packed = lib.pack_weights(inp["W_in"].cuda(), inp["W_out"].cuda())
    base = inp["logits"].reshape(cfg.N * cfg.B, -1)
    blocks = [base[torch.randperm(cfg.N * cfg.B, generator=g)].reshape(cfg.N, cfg.B, -1).cuda()
              for _ in range(4)]
    torch.cuda.synchronize()

    want = []
    for lg in blocks:
        ids, logp = lib.topk(lg, cfg.K)
        draft, choice, logq = lib.score_walk(ids, logp, E, packed)
        torch.cuda.synchronize()
        want.append([to_np(x) for x in (ids, logp, draft, choice, logq)])

    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    ws = [(lib.topk_workspace(cfg.N, cfg.B, cfg.V, cfg.K), lib.score_walk_workspace(cfg.N, cfg.B, cfg.K))
          for _ in streams]
    torch.cuda.synchronize()
    got = []
    for rep in range(2):  # the second round reuses each stream's workspaces
        got = []
        for b, lg in enumerate(blocks):
            s = streams[b % 2]
            tws, fws = ws[b % 2]
            with torch.cuda.stream(s):
                ids, logp = lib.topk(lg, cfg.K, workspace=tws)
                draft, choice, logq = lib.score_walk(ids, logp, E, packed, workspace=fws)
                got.append((ids, logp, draft, choice, logq))
        torch.cuda.synchronize()
        for b in range(len(blocks)):
            for name, w, x in zip(("ids", "logp", "draft", "choice", "logq"), want[b], got[b]):
                assert_equal(to_np(x), w, f"round {rep} block {b} {name}")
    for tws, _ in ws:
        assert lib.topk_wait_status(tws) == 0
