"""GPU tests of lilicorr_block_graph_* (top-K + one fused pass, or where that pass does not apply
the candidate vectors + the one-pass decode over them, recorded as one HIP graph).

Each graph is replayed several times, with the program's own eager work and synchronisations
between replays and new logits written into the captured buffer before each one; every replay
must give, bit for bit, what the eager calls give on the same logits (the same kernels run), and
the eager calls are themselves checked against the oracle by the other parity tests (the draft
is checked against the oracle here too, once).
"""
import ctypes

import numpy as np
import pytest
import torch

from parity import assert_equal, to_np
from test_gpu_score_walk import _oracle

pytestmark = pytest.mark.gpu

OUTS = {"greedy": ("draft", "choice", "logq"), "certified": ("draft", "choice", "logq", "rescored"),
        "exact": ("draft", "choice", "logq", "score")}


def _eager(lib, logits, K, E, packed, anchor, decode):
    ids, logp = lib.topk(logits, K)
    if decode == "greedy":
        d, c, q = lib.score_walk(ids, logp, E, packed, anchor)
        res = dict(draft=d, choice=c, logq=q)
    elif decode == "certified":
        d, c, q, r = lib.score_walk_certified(ids, logp, E, packed, anchor)
        res = dict(draft=d, choice=c, logq=q, rescored=r)
    else:
        d, c, q, s = lib.score_viterbi(ids, logp, E, packed, anchor)
        res = dict(draft=d, choice=c, logq=q, score=s)
    res.update(ids=ids, logp=logp)
    torch.cuda.synchronize()
    return {k: to_np(v) for k, v in res.items()}


@pytest.mark.parametrize("decode", ["greedy", "certified", "exact"])
@pytest.mark.parametrize("anchor", [False, True])
def test_block_graph_replays_match_eager(lib, cfg_inputs, decode, anchor):
    cfg, inp = cfg_inputs(2)
    print(f"graph decode={decode} anchor={anchor} config 2", flush=True)
    g = torch.Generator().manual_seed(11)
    E = inp["E"].cuda()
    packed = lib.pack_weights(inp["W_in"].cuda(), inp["W_out"].cuda())
    ao = (torch.randn(cfg.N, cfg.d, generator=g).cuda() if anchor else None)
    logits = inp["logits"].cuda()            # the captured buffer
    graph = lib.BlockGraph(logits, cfg.K, E, packed, ao, decode=decode)
    torch.cuda.synchronize()
    for rep in range(3):
        if rep > 0:  # new logits in the captured buffer: permute the slots of the batch
            perm = torch.randperm(cfg.N * cfg.B, generator=g)
            logits.copy_(inp["logits"].reshape(cfg.N * cfg.B, -1)[perm].reshape(logits.shape))
        want = _eager(lib, logits, cfg.K, E, packed, ao, decode)   # eager work between replays
        graph.launch()
        torch.cuda.synchronize()
        got = dict(ids=to_np(graph.ids), logp=to_np(graph.logp), draft=to_np(graph.draft),
                   choice=to_np(graph.choice), logq=to_np(graph.logq))
        if decode == "certified":
            got["rescored"] = to_np(graph.rescored)
        if decode == "exact":
            got["score"] = to_np(graph.score)
        for k in ("ids", "logp") + OUTS[decode]:
            assert np.array_equal(got[k].view(np.uint8), want[k].view(np.uint8)), \
                f"replay {rep}: {k} differs from the eager calls"
        if rep == 0 and decode != "exact":
            r = _oracle(want["ids"], want["logp"], to_np(inp["E"]), to_np(inp["W_in"]),
                        to_np(inp["W_out"]), to_np(ao) if anchor else None)
            assert_equal(got["draft"], r["draft"], "graph draft against the oracle")
    graph.close()


def _eager_vectors(lib, logits, K, E, packed, anchor, decode):
    """The block through the candidate vectors and the one-pass decode over them (the calls the
    graph records where the fused pass does not apply)."""
    ids, logp = lib.topk(logits, K)
    iv, ov = lib.candidate_vectors(ids, E, packed)
    if decode == "greedy":
        res = dict(zip(OUTS[decode], lib.pair_walk(iv, ov, logp, ids, anchor)))
    elif decode == "certified":
        res = dict(zip(OUTS[decode], lib.pair_walk_certified(iv, ov, logp, ids, E, packed, anchor)))
    else:
        res = dict(zip(OUTS[decode], lib.pair_viterbi(iv, ov, logp, ids, anchor)))
    res.update(ids=ids, logp=logp)
    torch.cuda.synchronize()
    return {k: to_np(v) for k, v in res.items()}


@pytest.mark.parametrize("cfg_index,decode", [(4, "greedy"), (4, "certified"), (4, "exact"),
                                              (0, "greedy"), (0, "exact")])
def test_block_graph_wide_path_replays_match_eager(lib, cfg_inputs, cfg_index, decode):
    """Where the fused pass does not apply (d = 512 at the stress workload, fp32 E at config 0)
    the graph holds the candidate vectors and the one-pass decode over them; its replays equal
    those eager calls bit for bit (the stress workload's first 8 requests)."""
    cfg, inp = cfg_inputs(cfg_index)
    n = min(cfg.N, 8)
    print(f"graph wide path decode={decode} config {cfg_index} ({n} requests)", flush=True)
    g = torch.Generator().manual_seed(13)
    E = inp["E"].cuda()
    packed = lib.pack_weights(inp["W_in"].cuda(), inp["W_out"].cuda())
    ao = torch.randn(n, cfg.d, generator=g).cuda()
    base = inp["logits"][:n].contiguous()
    logits = base.cuda()
    graph = lib.BlockGraph(logits, cfg.K, E, packed, ao, decode=decode)
    assert graph.in_vec is not None
    torch.cuda.synchronize()
    for rep in range(3):
        if rep > 0:
            perm = torch.randperm(n * cfg.B, generator=g)
            logits.copy_(base.reshape(n * cfg.B, -1)[perm].reshape(logits.shape))
        want = _eager_vectors(lib, logits, cfg.K, E, packed, ao, decode)
        graph.launch()
        torch.cuda.synchronize()
        got = dict(ids=to_np(graph.ids), logp=to_np(graph.logp))
        got.update({k: to_np(getattr(graph, k)) for k in OUTS[decode]})
        for k in ("ids", "logp") + OUTS[decode]:
            assert np.array_equal(got[k].view(np.uint8), want[k].view(np.uint8)), \
                f"replay {rep}: {k} differs from the eager calls"
        if rep == 0 and decode == "greedy":
            r = _oracle(want["ids"], want["logp"], to_np(inp["E"]), to_np(inp["W_in"]),
                        to_np(inp["W_out"]), to_np(ao))
            assert_equal(got["draft"], r["draft"], "graph draft against the oracle")
    graph.close()


def test_block_graph_wide_path_needs_vector_buffers(lib, cfg_inputs):
    """The wide path records into caller-given vector buffers: without them create fails with no
    graph; the certified rule re-scores from bf16 rows only (fp32 E: unsupported)."""
    cfg, inp = cfg_inputs(0)
    logits = inp["logits"].cuda()
    E = inp["E"].cuda()
    packed = lib.pack_weights(inp["W_in"].cuda(), inp["W_out"].cuda())
    graph = lib.BlockGraph(logits, cfg.K, E, packed)
    a = graph.args
    handle = ctypes.c_void_p(1)
    a.in_vec = None
    rc = lib.load_library().lilicorr_block_graph_create(ctypes.byref(a), ctypes.byref(handle))
    assert rc == -1 and handle.value is None
    graph.close()
    with pytest.raises(lib.LilicorrError):
        lib.BlockGraph(logits, cfg.K, E, packed, decode="certified")


def test_block_graph_rejects_bad_arguments(lib, cfg_inputs):
    """Argument errors of the recorded calls come back from create, with no graph."""
    cfg, inp = cfg_inputs(1)
    logits = inp["logits"].cuda()
    E = inp["E"].cuda()
    packed = lib.pack_weights(inp["W_in"].cuda(), inp["W_out"].cuda())
    graph = lib.BlockGraph(logits, cfg.K, E, packed)
    a = graph.args
    saved = a.fused_workspace_bytes
    a.fused_workspace_bytes = 8          # too small
    handle = ctypes.c_void_p(1)
    rc = lib.load_library().lilicorr_block_graph_create(ctypes.byref(a), ctypes.byref(handle))
    assert rc == -4 and handle.value is None
    a.fused_workspace_bytes = saved
    a.K = 65                             # above the top-K limit
    rc = lib.load_library().lilicorr_block_graph_create(ctypes.byref(a), ctypes.byref(handle))
    assert rc == -2 and handle.value is None
    graph.close()
    graph.close()                        # a second close is a no-op
    with pytest.raises(lib.LilicorrError):
        graph.launch()
