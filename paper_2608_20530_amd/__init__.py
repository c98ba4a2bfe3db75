"""LiLiCorr draft-correlation hot path on MI355X (gfx950): Python binding of liblilicorr.so.

The four steps run in hand-written HIP kernels behind a C ABI (include/lilicorr.h):

  lilicorr_topk               logits [N,B,V] -> ids, logp [N,B,K]       (Sec. 3.2; serving appendix)
  lilicorr_topk_features      ... plus the five confidence scalars      (implementation appendix)
  lilicorr_topk_wait_status   reads and clears a top-K workspace's wait status word
  lilicorr_pack_weights       W_in, W_out [d,d] -> matrix-core layout   (once per weight set)
  lilicorr_candidate_vectors  ids, E -> in_vec, out_vec [N,B,K,d]       (Sec. 3.2 unit-norm heads)
  lilicorr_pair_scores        in/out -> S [N,B-1,K,K] (+ S0 [N,K])      (Eq. pair)
  lilicorr_greedy_walk        S, S0, logp, ids -> draft, choice, logq   (Sec. 3.5, Eq. localar)
  lilicorr_viterbi_walk       S, S0, logp, ids -> best path, logq, g    (Eq. pathscore)
  lilicorr_score_walk         ids, logp, E -> draft, choice, logq       (steps 2-4 in one pass)
  lilicorr_score_walk_noalloc the same pass with no workspace (library-held device scratch)
  lilicorr_score_walk_certified  the same pass, near-tied decisions decided again in fp64
  lilicorr_score_viterbi      the same pass with the exact max-path decode
  lilicorr_block_graph_*      top-K + one fused pass recorded as one HIP graph, replayed per block
  lilicorr_scorer_*           scoring-Transformer stand-in over the candidate lattice (cost only)

This module only marshals arguments: torch supplies device memory and the current HIP stream,
and every step of the path runs in the library's kernels. There is no fallback: if the library
is missing or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "LIB_PATH", "load_library", "LilicorrError", "SIGMA",
    "lilicorr_topk", "lilicorr_topk_features", "lilicorr_topk_workspace_bytes",
    "lilicorr_topk_wait_status", "lilicorr_set_wait_limit", "lilicorr_packed_weight_bytes",
    "lilicorr_pack_weights", "lilicorr_candidate_vectors", "lilicorr_pair_scores",
    "lilicorr_greedy_walk", "lilicorr_viterbi_walk", "lilicorr_score_walk", "lilicorr_score_walk_workspace_bytes",
    "lilicorr_score_walk_noalloc",
    "lilicorr_score_walk_certified", "lilicorr_score_walk_certified_workspace_bytes",
    "lilicorr_score_viterbi", "lilicorr_score_viterbi_workspace_bytes",
    "lilicorr_block_graph_create", "lilicorr_block_graph_launch", "lilicorr_block_graph_destroy",
    "BlockArgs", "BlockGraph", "lilicorr_status_string",
    "topk", "topk_workspace", "topk_wait_status", "pack_weights", "candidate_vectors", "pair_scores", "greedy_walk", "viterbi_walk", "score_walk", "score_viterbi",
    "score_walk_certified", "score_walk_certified_workspace", "CERT_MARGIN", "draft_block",
    "ScorerLayer", "lilicorr_scorer_packed_bytes", "lilicorr_scorer_pack",
    "lilicorr_scorer_workspace_bytes", "lilicorr_scorer_forward", "scorer_pack", "scorer_workspace",
    "scorer_forward",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liblilicorr.so")
SIGMA = 8.0  # cosine scale of Eq. (pair), hyper-parameter table of the implementation appendix
# fp32 score gap at or below which score_walk_certified decides again in fp64; the certificate
# holds while every fp32 node score is within CERT_MARGIN / 2 (3.1e-5) of its double-precision
# value, and the fused pass's fp32 pair scores measure within 1.8e-6 of it on the workloads
CERT_MARGIN = 2.0 ** -14

F32, BF16 = 0, 1
DECODE = {"greedy": 0, "certified": 1, "exact": 2}

_lib = None


class LilicorrError(RuntimeError):
    pass


class BlockArgs(ctypes.Structure):
    """lilicorr_block_args of include/lilicorr.h, field for field."""
    _fields_ = [
        ("logits", ctypes.c_void_p), ("logits_dtype", ctypes.c_int),
        ("N", ctypes.c_int64), ("B", ctypes.c_int64), ("V", ctypes.c_int64), ("K", ctypes.c_int),
        ("ids", ctypes.c_void_p), ("logp", ctypes.c_void_p), ("topk_workspace", ctypes.c_void_p),
        ("topk_workspace_bytes", ctypes.c_size_t),
        ("E", ctypes.c_void_p), ("e_dtype", ctypes.c_int), ("e_rows", ctypes.c_int64),
        ("d", ctypes.c_int), ("packed_w", ctypes.c_void_p), ("anchor_out", ctypes.c_void_p),
        ("sigma", ctypes.c_float), ("logp_weight", ctypes.c_float), ("decode", ctypes.c_int),
        ("margin", ctypes.c_float), ("S", ctypes.c_void_p), ("S0", ctypes.c_void_p),
        ("draft", ctypes.c_void_p), ("choice", ctypes.c_void_p), ("logq", ctypes.c_void_p),
        ("score", ctypes.c_void_p), ("rescored", ctypes.c_void_p),
        ("fused_workspace", ctypes.c_void_p), ("fused_workspace_bytes", ctypes.c_size_t),
        ("in_vec", ctypes.c_void_p), ("out_vec", ctypes.c_void_p),
    ]


class ScorerLayer(ctypes.Structure):
    """lilicorr_scorer_layer of include/lilicorr.h, field for field (device pointers)."""
    _fields_ = [(name, ctypes.c_void_p) for name in
                ("w_qkv", "w_o", "w_1", "w_2", "g_attn", "g_ffn", "dist_bias", "same_bias")]


def load_library() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise LilicorrError(f"{LIB_PATH} is not built (run __graft_entry__.build() or "
                            "python paper_2608_20530_amd/build.py); there is no fallback path")
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, I, SZ, F = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t,
                        ctypes.c_float)
    sig = {
        "lilicorr_topk_workspace_bytes": ([I64, I64, I64, I], SZ),
        "lilicorr_topk": ([P, I, I64, I64, I64, I, P, P, P, SZ, P], I),
        "lilicorr_topk_features": ([P, I, I64, I64, I64, I, P, P, P, P, SZ, P], I),
        "lilicorr_topk_wait_status": ([P, P], I),
        "lilicorr_set_wait_limit": ([I64], None),
        "lilicorr_packed_weight_bytes": ([I], SZ),
        "lilicorr_pack_weights": ([P, P, I, P, P], I),
        "lilicorr_candidate_vectors": ([P, P, I, I64, I, P, I64, I64, I, P, P, P], I),
        "lilicorr_pair_scores": ([P, P, P, I64, I64, I, I, F, P, P, P], I),
        "lilicorr_greedy_walk": ([P, P, P, P, I64, I64, I, F, P, P, P, P], I),
        "lilicorr_viterbi_walk": ([P, P, P, P, I64, I64, I, F, P, P, P, P, P], I),
        "lilicorr_score_walk_workspace_bytes": ([I64, I64, I], SZ),
        "lilicorr_score_walk": ([P, P, P, I, I64, I, P, P, I64, I64, I, F, F, P, P, P, P, P, P, SZ,
                                 P], I),
        "lilicorr_score_walk_noalloc": ([P, P, P, I, I64, I, P, P, I64, I64, I, F, F, P, P, P, P, P,
                                         P], I),
        "lilicorr_score_walk_certified_workspace_bytes": ([I64, I64, I], SZ),
        "lilicorr_score_walk_certified": ([P, P, P, I, I64, I, P, P, I64, I64, I, F, F, F, P, P, P,
                                           P, P, P, P, SZ, P], I),
        "lilicorr_score_viterbi_workspace_bytes": ([I64, I64, I], SZ),
        "lilicorr_score_viterbi": ([P, P, P, I, I64, I, P, P, I64, I64, I, F, F, P, P, P, P, P, P, P,
                                    SZ, P], I),
        "lilicorr_pair_walk": ([P, P, P, P, P, I64, I64, I, I, F, F, P, P, P, P, P, P, SZ, P], I),
        "lilicorr_pair_walk_certified": ([P, P, P, P, P, P, I, I64, P, I64, I64, I, I, F, F, F, P,
                                          P, P, P, P, P, P, SZ, P], I),
        "lilicorr_pair_viterbi": ([P, P, P, P, P, I64, I64, I, I, F, F, P, P, P, P, P, P, P, SZ,
                                   P], I),
        "lilicorr_block_graph_create": ([ctypes.POINTER(BlockArgs), ctypes.POINTER(P)], I),
        "lilicorr_block_graph_launch": ([P, P], I),
        "lilicorr_block_graph_destroy": ([P], None),
        "lilicorr_scorer_packed_bytes": ([I, I, I, I64], SZ),
        "lilicorr_scorer_pack": ([ctypes.POINTER(ScorerLayer), I, I, I, I64, P, P], I),
        "lilicorr_scorer_workspace_bytes": ([I64, I64, I, I, I], SZ),
        "lilicorr_scorer_forward": ([P, I64, I64, I, I, I, I, I, P, P, SZ, P], I),
        "lilicorr_status_string": ([I], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


# ---- raw C ABI (same names and argument order as include/lilicorr.h) ----------------------------

def lilicorr_status_string(status: int) -> str:
    return load_library().lilicorr_status_string(status).decode()


def _call(name: str, *args) -> int:
    rc = getattr(load_library(), name)(*args)
    if rc != 0:
        raise LilicorrError(f"{name}: {lilicorr_status_string(rc)} (status {rc})")
    return rc


def lilicorr_topk_workspace_bytes(N: int, B: int, V: int, K: int) -> int:
    return int(load_library().lilicorr_topk_workspace_bytes(N, B, V, K))


def lilicorr_topk_wait_status(workspace, stream) -> int:
    """Returns the status (0, or LILICORR_ERR_TIMEOUT = -6 when a wait gave up); raises only when
    the query itself fails."""
    rc = load_library().lilicorr_topk_wait_status(workspace, stream)
    if rc not in (0, -6):
        raise LilicorrError(f"lilicorr_topk_wait_status: {lilicorr_status_string(rc)} (status {rc})")
    return rc


def lilicorr_set_wait_limit(spins: int) -> None:
    load_library().lilicorr_set_wait_limit(spins)


def lilicorr_packed_weight_bytes(d: int) -> int:
    return int(load_library().lilicorr_packed_weight_bytes(d))


def lilicorr_topk(logits, dtype, N, B, V, K, ids, logp, workspace, workspace_bytes, stream):
    return _call("lilicorr_topk", logits, dtype, N, B, V, K, ids, logp, workspace,
                 workspace_bytes, stream)


def lilicorr_topk_features(logits, dtype, N, B, V, K, ids, logp, feat, workspace, workspace_bytes,
                           stream):
    return _call("lilicorr_topk_features", logits, dtype, N, B, V, K, ids, logp, feat, workspace,
                 workspace_bytes, stream)


def lilicorr_pack_weights(W_in, W_out, d, packed, stream):
    return _call("lilicorr_pack_weights", W_in, W_out, d, packed, stream)


def lilicorr_candidate_vectors(ids, E, e_dtype, V, d, packed_w, N, B, K, in_vec, out_vec, stream):
    return _call("lilicorr_candidate_vectors", ids, E, e_dtype, V, d, packed_w, N, B, K, in_vec,
                 out_vec, stream)


def lilicorr_pair_scores(in_vec, out_vec, anchor_out, N, B, K, d, sigma, S, S0, stream):
    return _call("lilicorr_pair_scores", in_vec, out_vec, anchor_out, N, B, K, d, sigma, S, S0,
                 stream)


def lilicorr_greedy_walk(S, S0, logp, ids, N, B, K, logp_weight, draft, choice, logq, stream):
    return _call("lilicorr_greedy_walk", S, S0, logp, ids, N, B, K, logp_weight, draft, choice,
                 logq, stream)


def lilicorr_viterbi_walk(S, S0, logp, ids, N, B, K, logp_weight, draft, choice, logq, score,
                          stream):
    return _call("lilicorr_viterbi_walk", S, S0, logp, ids, N, B, K, logp_weight, draft, choice,
                 logq, score, stream)


def lilicorr_score_walk_workspace_bytes(N: int, B: int, K: int) -> int:
    return int(load_library().lilicorr_score_walk_workspace_bytes(N, B, K))


def lilicorr_score_walk(ids, logp, E, e_dtype, V, d, packed_w, anchor_out, N, B, K, sigma,
                        logp_weight, S, S0, draft, choice, logq, workspace, workspace_bytes, stream):
    return _call("lilicorr_score_walk", ids, logp, E, e_dtype, V, d, packed_w, anchor_out, N, B,
                 K, sigma, logp_weight, S, S0, draft, choice, logq, workspace, workspace_bytes,
                 stream)


def lilicorr_score_walk_noalloc(ids, logp, E, e_dtype, V, d, packed_w, anchor_out, N, B, K,
                                sigma, logp_weight, S, S0, draft, choice, logq, stream):
    return _call("lilicorr_score_walk_noalloc", ids, logp, E, e_dtype, V, d, packed_w, anchor_out,
                 N, B, K, sigma, logp_weight, S, S0, draft, choice, logq, stream)


def lilicorr_score_walk_certified_workspace_bytes(N: int, B: int, K: int) -> int:
    return int(load_library().lilicorr_score_walk_certified_workspace_bytes(N, B, K))


def lilicorr_score_walk_certified(ids, logp, E, e_dtype, V, d, packed_w, anchor_out, N, B, K,
                                  sigma, logp_weight, margin, S, S0, draft, choice, logq, rescored,
                                  workspace, workspace_bytes, stream):
    return _call("lilicorr_score_walk_certified", ids, logp, E, e_dtype, V, d, packed_w,
                 anchor_out, N, B, K, sigma, logp_weight, margin, S, S0, draft, choice, logq,
                 rescored, workspace, workspace_bytes, stream)


def lilicorr_score_viterbi_workspace_bytes(N: int, B: int, K: int) -> int:
    return int(load_library().lilicorr_score_viterbi_workspace_bytes(N, B, K))


def lilicorr_score_viterbi(ids, logp, E, e_dtype, V, d, packed_w, anchor_out, N, B, K, sigma,
                           logp_weight, S, S0, draft, choice, logq, score, workspace,
                           workspace_bytes, stream):
    return _call("lilicorr_score_viterbi", ids, logp, E, e_dtype, V, d, packed_w, anchor_out, N,
                 B, K, sigma, logp_weight, S, S0, draft, choice, logq, score, workspace,
                 workspace_bytes, stream)


def lilicorr_pair_walk(in_vec, out_vec, anchor_out, logp, ids, N, B, K, d, sigma, logp_weight, S,
                       S0, draft, choice, logq, workspace, workspace_bytes, stream):
    return _call("lilicorr_pair_walk", in_vec, out_vec, anchor_out, logp, ids, N, B, K, d, sigma,
                 logp_weight, S, S0, draft, choice, logq, workspace, workspace_bytes, stream)


def lilicorr_pair_walk_certified(in_vec, out_vec, anchor_out, logp, ids, E, e_dtype, V, packed_w,
                                 N, B, K, d, sigma, logp_weight, margin, S, S0, draft, choice,
                                 logq, rescored, workspace, workspace_bytes, stream):
    return _call("lilicorr_pair_walk_certified", in_vec, out_vec, anchor_out, logp, ids, E,
                 e_dtype, V, packed_w, N, B, K, d, sigma, logp_weight, margin, S, S0, draft,
                 choice, logq, rescored, workspace, workspace_bytes, stream)


def lilicorr_pair_viterbi(in_vec, out_vec, anchor_out, logp, ids, N, B, K, d, sigma, logp_weight,
                          S, S0, draft, choice, logq, score, workspace, workspace_bytes, stream):
    return _call("lilicorr_pair_viterbi", in_vec, out_vec, anchor_out, logp, ids, N, B, K, d,
                 sigma, logp_weight, S, S0, draft, choice, logq, score, workspace,
                 workspace_bytes, stream)


def lilicorr_block_graph_create(args: BlockArgs) -> int:
    """-> the graph handle (an integer address); raises on a non-zero status."""
    handle = ctypes.c_void_p()
    _call("lilicorr_block_graph_create", ctypes.byref(args), ctypes.byref(handle))
    return handle.value


def lilicorr_block_graph_launch(graph, stream):
    return _call("lilicorr_block_graph_launch", graph, stream)


def lilicorr_block_graph_destroy(graph) -> None:
    load_library().lilicorr_block_graph_destroy(graph)


# ---- torch conveniences (marshalling only) -----------------------------------------------------

def _dev(t: torch.Tensor | None, name: str, dtypes=None):
    if t is None:
        return None
    if not t.is_cuda:
        raise LilicorrError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise LilicorrError(f"{name} must be contiguous")
    if dtypes is not None and t.dtype not in dtypes:
        raise LilicorrError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    return t.data_ptr()


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _dtype_code(t: torch.Tensor) -> int:
    return BF16 if t.dtype == torch.bfloat16 else F32


def topk_workspace(N: int, B: int, V: int, K: int, device="cuda") -> torch.Tensor:
    """A zero-filled top-K workspace (its status word must start at zero)."""
    need = lilicorr_topk_workspace_bytes(N, B, V, K)
    if need == 0:
        raise LilicorrError(f"topk does not support N={N}, B={B}, V={V}, K={K}")
    return torch.zeros(need, dtype=torch.uint8, device=device)


def topk_wait_status(workspace: torch.Tensor) -> int:
    """0 if every bounded wait of the top-K calls on `workspace` finished, -6
    (LILICORR_ERR_TIMEOUT) if one gave up; clears the word. Waits for the current stream."""
    return lilicorr_topk_wait_status(_dev(workspace, "workspace"), _stream())


def topk(logits: torch.Tensor, K: int, *, out=None, workspace=None, features: bool = False):
    """logits [N,B,V] bf16/fp32 -> (ids [N,B,K] int32, logp [N,B,K] fp32[, feat [N,B,K,5] fp32
    when features=True])."""
    N, B, V = logits.shape
    dev = logits.device
    if out is None:
        out = (torch.empty(N, B, K, dtype=torch.int32, device=dev),
               torch.empty(N, B, K, dtype=torch.float32, device=dev))
        if features:
            out = out + (torch.empty(N, B, K, 5, dtype=torch.float32, device=dev),)
    ids, logp = out[0], out[1]
    if workspace is None:
        workspace = topk_workspace(N, B, V, K, dev)
    args = (_dev(logits, "logits", (torch.bfloat16, torch.float32)), _dtype_code(logits), N, B, V,
            K, _dev(ids, "ids", (torch.int32,)), _dev(logp, "logp", (torch.float32,)))
    if features:
        feat = out[2]
        lilicorr_topk_features(*args, _dev(feat, "feat", (torch.float32,)),
                               _dev(workspace, "workspace"), workspace.numel(), _stream())
        return ids, logp, feat
    lilicorr_topk(*args, _dev(workspace, "workspace"), workspace.numel(), _stream())
    return ids, logp


def pack_weights(W_in: torch.Tensor, W_out: torch.Tensor, *, out=None) -> torch.Tensor:
    d = W_in.shape[0]
    need = lilicorr_packed_weight_bytes(d)
    packed = out if out is not None else torch.empty(max(need, 16), dtype=torch.uint8, device=W_in.device)
    lilicorr_pack_weights(_dev(W_in, "W_in", (torch.float32,)), _dev(W_out, "W_out", (torch.float32,)),
                          d, _dev(packed, "packed"), _stream())
    return packed


def candidate_vectors(ids: torch.Tensor, E: torch.Tensor, packed: torch.Tensor, *, out=None):
    """ids [N,B,K] int32, E [V,d] bf16/fp32 -> (in_vec, out_vec) [N,B,K,d] fp32."""
    N, B, K = ids.shape
    V, d = E.shape
    if out is None:
        out = (torch.empty(N, B, K, d, dtype=torch.float32, device=ids.device),
               torch.empty(N, B, K, d, dtype=torch.float32, device=ids.device))
    in_vec, out_vec = out
    lilicorr_candidate_vectors(_dev(ids, "ids", (torch.int32,)),
                               _dev(E, "E", (torch.bfloat16, torch.float32)), _dtype_code(E), V, d,
                               _dev(packed, "packed"), N, B, K,
                               _dev(in_vec, "in_vec", (torch.float32,)),
                               _dev(out_vec, "out_vec", (torch.float32,)), _stream())
    return in_vec, out_vec


def pair_scores(in_vec: torch.Tensor, out_vec: torch.Tensor, anchor_out=None, sigma: float = SIGMA,
                *, out=None):
    """-> (S [N,B-1,K,K] fp32, S0 [N,K] fp32 or None)."""
    N, B, K, d = in_vec.shape
    if out is None:
        S = torch.empty(N, max(B - 1, 0), K, K, dtype=torch.float32, device=in_vec.device)
        S0 = (torch.empty(N, K, dtype=torch.float32, device=in_vec.device)
              if anchor_out is not None else None)
    else:
        S, S0 = out
    lilicorr_pair_scores(_dev(in_vec, "in_vec", (torch.float32,)),
                         _dev(out_vec, "out_vec", (torch.float32,)),
                         _dev(anchor_out, "anchor_out", (torch.float32,)), N, B, K, d, float(sigma),
                         _dev(S, "S", (torch.float32,)) if B > 1 else None,
                         _dev(S0, "S0", (torch.float32,)), _stream())
    return S, S0


def greedy_walk(S: torch.Tensor, S0, logp: torch.Tensor, ids: torch.Tensor,
                logp_weight: float = 0.0, *, out=None):
    """-> (draft [N,B] int32, choice [N,B] int32, logq [N,B] fp32)."""
    N, B, K = ids.shape
    if out is None:
        out = (torch.empty(N, B, dtype=torch.int32, device=ids.device),
               torch.empty(N, B, dtype=torch.int32, device=ids.device),
               torch.empty(N, B, dtype=torch.float32, device=ids.device))
    draft, choice, logq = out
    lilicorr_greedy_walk(_dev(S, "S", (torch.float32,)) if B > 1 else None,
                         _dev(S0, "S0", (torch.float32,)), _dev(logp, "logp", (torch.float32,)),
                         _dev(ids, "ids", (torch.int32,)), N, B, K, float(logp_weight),
                         _dev(draft, "draft", (torch.int32,)), _dev(choice, "choice", (torch.int32,)),
                         _dev(logq, "logq", (torch.float32,)), _stream())
    return draft, choice, logq


def viterbi_walk(S: torch.Tensor, S0, logp: torch.Tensor, ids: torch.Tensor,
                 logp_weight: float = 0.0, *, out=None):
    """Exact max-path decode -> (draft [N,B] int32, choice [N,B] int32, logq [N,B] fp32,
    score [N] fp32)."""
    N, B, K = ids.shape
    if out is None:
        out = (torch.empty(N, B, dtype=torch.int32, device=ids.device),
               torch.empty(N, B, dtype=torch.int32, device=ids.device),
               torch.empty(N, B, dtype=torch.float32, device=ids.device),
               torch.empty(N, dtype=torch.float32, device=ids.device))
    draft, choice, logq, score = out
    lilicorr_viterbi_walk(_dev(S, "S", (torch.float32,)) if B > 1 else None,
                          _dev(S0, "S0", (torch.float32,)), _dev(logp, "logp", (torch.float32,)),
                          _dev(ids, "ids", (torch.int32,)), N, B, K, float(logp_weight),
                          _dev(draft, "draft", (torch.int32,)),
                          _dev(choice, "choice", (torch.int32,)),
                          _dev(logq, "logq", (torch.float32,)),
                          _dev(score, "score", (torch.float32,)), _stream())
    return draft, choice, logq, score


def score_walk_workspace(N: int, B: int, K: int, device="cuda") -> torch.Tensor:
    """A zero-filled workspace for score_walk (the library keeps it zeroed between calls)."""
    need = lilicorr_score_walk_workspace_bytes(N, B, K)
    if need == 0:
        raise LilicorrError(f"score_walk does not support N={N}, B={B}, K={K}")
    return torch.zeros(need, dtype=torch.uint8, device=device)


def score_walk(ids: torch.Tensor, logp: torch.Tensor, E: torch.Tensor, packed: torch.Tensor,
               anchor_out=None, sigma: float = SIGMA, logp_weight: float = 0.0, *,
               scores: bool = False, out=None, workspace=None):
    """Steps 2-4 in one pass -> (draft, choice, logq[, S, S0 when scores=True])."""
    N, B, K = ids.shape
    V, d = E.shape
    dev = ids.device
    if out is None:
        out = (torch.empty(N, B, dtype=torch.int32, device=dev),
               torch.empty(N, B, dtype=torch.int32, device=dev),
               torch.empty(N, B, dtype=torch.float32, device=dev))
    draft, choice, logq = out
    S = S0 = None
    if scores:
        S = torch.empty(N, max(B - 1, 0), K, K, dtype=torch.float32, device=dev)
        S0 = torch.empty(N, K, dtype=torch.float32, device=dev) if anchor_out is not None else None
    if workspace is None:
        workspace = score_walk_workspace(N, B, K, dev)
    lilicorr_score_walk(_dev(ids, "ids", (torch.int32,)), _dev(logp, "logp", (torch.float32,)),
                        _dev(E, "E", (torch.bfloat16, torch.float32)), _dtype_code(E), V, d,
                        _dev(packed, "packed"), _dev(anchor_out, "anchor_out", (torch.float32,)),
                        N, B, K, float(sigma), float(logp_weight),
                        _dev(S, "S", (torch.float32,)) if S is not None and B > 1 else None,
                        _dev(S0, "S0", (torch.float32,)), _dev(draft, "draft", (torch.int32,)),
                        _dev(choice, "choice", (torch.int32,)), _dev(logq, "logq", (torch.float32,)),
                        _dev(workspace, "workspace"), workspace.numel(), _stream())
    if scores:
        return draft, choice, logq, S, S0
    return draft, choice, logq


def score_walk_certified_workspace(N: int, B: int, K: int, device="cuda") -> torch.Tensor:
    """A zero-filled workspace for score_walk_certified (kept zeroed between calls)."""
    need = lilicorr_score_walk_certified_workspace_bytes(N, B, K)
    if need == 0:
        raise LilicorrError(f"score_walk_certified does not support N={N}, B={B}, K={K}")
    return torch.zeros(need, dtype=torch.uint8, device=device)


def score_walk_certified(ids: torch.Tensor, logp: torch.Tensor, E: torch.Tensor,
                         packed: torch.Tensor, anchor_out=None, sigma: float = SIGMA,
                         logp_weight: float = 0.0, margin: float = CERT_MARGIN, *,
                         scores: bool = False, out=None, workspace=None):
    """Steps 2-4 in one pass, near-tied decisions re-scored in fp64 -> (draft, choice, logq,
    rescored[, S, S0 when scores=True])."""
    N, B, K = ids.shape
    V, d = E.shape
    dev = ids.device
    if out is None:
        out = (torch.empty(N, B, dtype=torch.int32, device=dev),
               torch.empty(N, B, dtype=torch.int32, device=dev),
               torch.empty(N, B, dtype=torch.float32, device=dev),
               torch.empty(N, B, dtype=torch.int32, device=dev))
    draft, choice, logq, rescored = out
    S = S0 = None
    if scores:
        S = torch.empty(N, max(B - 1, 0), K, K, dtype=torch.float32, device=dev)
        S0 = torch.empty(N, K, dtype=torch.float32, device=dev) if anchor_out is not None else None
    if workspace is None:
        workspace = score_walk_certified_workspace(N, B, K, dev)
    lilicorr_score_walk_certified(
        _dev(ids, "ids", (torch.int32,)), _dev(logp, "logp", (torch.float32,)),
        _dev(E, "E", (torch.bfloat16, torch.float32)), _dtype_code(E), V, d,
        _dev(packed, "packed"), _dev(anchor_out, "anchor_out", (torch.float32,)), N, B, K,
        float(sigma), float(logp_weight), float(margin),
        _dev(S, "S", (torch.float32,)) if S is not None and B > 1 else None,
        _dev(S0, "S0", (torch.float32,)), _dev(draft, "draft", (torch.int32,)),
        _dev(choice, "choice", (torch.int32,)), _dev(logq, "logq", (torch.float32,)),
        _dev(rescored, "rescored", (torch.int32,)), _dev(workspace, "workspace"),
        workspace.numel(), _stream())
    if scores:
        return draft, choice, logq, rescored, S, S0
    return draft, choice, logq, rescored


def score_viterbi_workspace(N: int, B: int, K: int, device="cuda") -> torch.Tensor:
    """A zero-filled workspace for score_viterbi (the library keeps it zeroed between calls)."""
    need = lilicorr_score_viterbi_workspace_bytes(N, B, K)
    if need == 0:
        raise LilicorrError(f"score_viterbi does not support N={N}, B={B}, K={K}")
    return torch.zeros(need, dtype=torch.uint8, device=device)


def score_viterbi(ids: torch.Tensor, logp: torch.Tensor, E: torch.Tensor, packed: torch.Tensor,
                  anchor_out=None, sigma: float = SIGMA, logp_weight: float = 0.0, *,
                  scores: bool = False, out=None, workspace=None):
    """Steps 2-4 with the exact decode -> (draft, choice, logq, score[, S, S0 when scores=True])."""
    N, B, K = ids.shape
    V, d = E.shape
    dev = ids.device
    if out is None:
        out = (torch.empty(N, B, dtype=torch.int32, device=dev),
               torch.empty(N, B, dtype=torch.int32, device=dev),
               torch.empty(N, B, dtype=torch.float32, device=dev),
               torch.empty(N, dtype=torch.float32, device=dev))
    draft, choice, logq, score = out
    S = S0 = None
    if scores:
        S = torch.empty(N, max(B - 1, 0), K, K, dtype=torch.float32, device=dev)
        S0 = torch.empty(N, K, dtype=torch.float32, device=dev) if anchor_out is not None else None
    if workspace is None:
        workspace = score_viterbi_workspace(N, B, K, dev)
    lilicorr_score_viterbi(_dev(ids, "ids", (torch.int32,)), _dev(logp, "logp", (torch.float32,)),
                           _dev(E, "E", (torch.bfloat16, torch.float32)), _dtype_code(E), V, d,
                           _dev(packed, "packed"),
                           _dev(anchor_out, "anchor_out", (torch.float32,)), N, B, K,
                           float(sigma), float(logp_weight),
                           _dev(S, "S", (torch.float32,)) if S is not None and B > 1 else None,
                           _dev(S0, "S0", (torch.float32,)), _dev(draft, "draft", (torch.int32,)),
                           _dev(choice, "choice", (torch.int32,)),
                           _dev(logq, "logq", (torch.float32,)),
                           _dev(score, "score", (torch.float32,)), _dev(workspace, "workspace"),
                           workspace.numel(), _stream())
    if scores:
        return draft, choice, logq, score, S, S0
    return draft, choice, logq, score


def _decode_outputs(N, B, K, dev, anchor_out, extra, scores, out):
    """draft, choice, logq (+ the `extra` [N]-or-[N,B] output) and, with scores, S and S0."""
    if out is None:
        out = (torch.empty(N, B, dtype=torch.int32, device=dev),
               torch.empty(N, B, dtype=torch.int32, device=dev),
               torch.empty(N, B, dtype=torch.float32, device=dev))
        if extra == "score":
            out += (torch.empty(N, dtype=torch.float32, device=dev),)
        elif extra == "rescored":
            out += (torch.empty(N, B, dtype=torch.int32, device=dev),)
    S = S0 = None
    if scores:
        S = torch.empty(N, max(B - 1, 0), K, K, dtype=torch.float32, device=dev)
        S0 = torch.empty(N, K, dtype=torch.float32, device=dev) if anchor_out is not None else None
    return tuple(out), S, S0


def _vector_args(in_vec, out_vec, anchor_out, logp, ids):
    N, B, K, d = in_vec.shape
    if tuple(out_vec.shape) != (N, B, K, d) or tuple(ids.shape) != (N, B, K):
        raise LilicorrError("in_vec, out_vec must be [N, B, K, d] and ids [N, B, K]")
    return (N, B, K, d, _dev(in_vec, "in_vec", (torch.float32,)),
            _dev(out_vec, "out_vec", (torch.float32,)),
            _dev(anchor_out, "anchor_out", (torch.float32,)),
            _dev(logp, "logp", (torch.float32,)), _dev(ids, "ids", (torch.int32,)))


def pair_walk(in_vec: torch.Tensor, out_vec: torch.Tensor, logp: torch.Tensor, ids: torch.Tensor,
              anchor_out=None, sigma: float = SIGMA, logp_weight: float = 0.0, *,
              scores: bool = False, out=None, workspace=None):
    """Steps 3-4 in one pass over the vectors of step 2 -> (draft, choice, logq[, S, S0 when
    scores=True]); the workspace is score_walk's."""
    N, B, K, d, *ptrs = _vector_args(in_vec, out_vec, anchor_out, logp, ids)
    (draft, choice, logq), S, S0 = _decode_outputs(N, B, K, ids.device, anchor_out, None,
                                                   scores, out)
    if workspace is None:
        workspace = score_walk_workspace(N, B, K, ids.device)
    lilicorr_pair_walk(*ptrs, N, B, K, d, float(sigma), float(logp_weight),
                       _dev(S, "S", (torch.float32,)) if S is not None and B > 1 else None,
                       _dev(S0, "S0", (torch.float32,)), _dev(draft, "draft", (torch.int32,)),
                       _dev(choice, "choice", (torch.int32,)), _dev(logq, "logq", (torch.float32,)),
                       _dev(workspace, "workspace"), workspace.numel(), _stream())
    return (draft, choice, logq, S, S0) if scores else (draft, choice, logq)


def pair_walk_certified(in_vec: torch.Tensor, out_vec: torch.Tensor, logp: torch.Tensor,
                        ids: torch.Tensor, E: torch.Tensor, packed: torch.Tensor, anchor_out=None,
                        sigma: float = SIGMA, logp_weight: float = 0.0,
                        margin: float = CERT_MARGIN, *, scores: bool = False, out=None,
                        workspace=None):
    """Steps 3-4 in one pass, near-tied decisions re-scored in fp64 -> (draft, choice, logq,
    rescored[, S, S0 when scores=True]); the workspace is score_walk_certified's."""
    N, B, K, d, *ptrs = _vector_args(in_vec, out_vec, anchor_out, logp, ids)
    (draft, choice, logq, rescored), S, S0 = _decode_outputs(N, B, K, ids.device, anchor_out,
                                                             "rescored", scores, out)
    if workspace is None:
        workspace = score_walk_certified_workspace(N, B, K, ids.device)
    lilicorr_pair_walk_certified(
        *ptrs, _dev(E, "E", (torch.bfloat16, torch.float32)), _dtype_code(E), E.shape[0],
        _dev(packed, "packed"), N, B, K, d, float(sigma), float(logp_weight), float(margin),
        _dev(S, "S", (torch.float32,)) if S is not None and B > 1 else None,
        _dev(S0, "S0", (torch.float32,)), _dev(draft, "draft", (torch.int32,)),
        _dev(choice, "choice", (torch.int32,)), _dev(logq, "logq", (torch.float32,)),
        _dev(rescored, "rescored", (torch.int32,)), _dev(workspace, "workspace"),
        workspace.numel(), _stream())
    return (draft, choice, logq, rescored, S, S0) if scores else (draft, choice, logq, rescored)


def pair_viterbi(in_vec: torch.Tensor, out_vec: torch.Tensor, logp: torch.Tensor,
                 ids: torch.Tensor, anchor_out=None, sigma: float = SIGMA,
                 logp_weight: float = 0.0, *, scores: bool = False, out=None, workspace=None):
    """Steps 3-4 with the exact decode in one pass -> (draft, choice, logq, score[, S, S0 when
    scores=True]); the workspace is score_viterbi's."""
    N, B, K, d, *ptrs = _vector_args(in_vec, out_vec, anchor_out, logp, ids)
    (draft, choice, logq, score), S, S0 = _decode_outputs(N, B, K, ids.device, anchor_out,
                                                          "score", scores, out)
    if workspace is None:
        workspace = score_viterbi_workspace(N, B, K, ids.device)
    lilicorr_pair_viterbi(*ptrs, N, B, K, d, float(sigma), float(logp_weight),
                          _dev(S, "S", (torch.float32,)) if S is not None and B > 1 else None,
                          _dev(S0, "S0", (torch.float32,)), _dev(draft, "draft", (torch.int32,)),
                          _dev(choice, "choice", (torch.int32,)),
                          _dev(logq, "logq", (torch.float32,)),
                          _dev(score, "score", (torch.float32,)), _dev(workspace, "workspace"),
                          workspace.numel(), _stream())
    return (draft, choice, logq, score, S, S0) if scores else (draft, choice, logq, score)


class BlockGraph:
    """One draft block (top-K, then one fused pass) recorded as a HIP graph over fixed buffers.

    The outputs (ids, logp, draft, choice, logq, and score / rescored / S / S0 where they apply)
    are allocated here, and so are the in/out vector buffers where the fused pass does not apply
    (fp32 E or d above 256: the graph then holds the candidate vectors and the one-pass decode
    over them); launch() replays the block on the current stream over whatever `logits` holds
    then. The object keeps every buffer the graph points at alive until close().
    """

    def __init__(self, logits: torch.Tensor, K: int, E: torch.Tensor, packed: torch.Tensor,
                 anchor_out=None, sigma: float = SIGMA, logp_weight: float = 0.0,
                 decode: str = "greedy", margin: float = CERT_MARGIN, scores: bool = False):
        if decode not in DECODE:
            raise LilicorrError(f"unknown decode {decode!r}; one of {sorted(DECODE)}")
        N, B, V = logits.shape
        rows, d = E.shape
        dev = logits.device
        self.logits, self.E, self.packed, self.anchor_out = logits, E, packed, anchor_out
        self.ids = torch.empty(N, B, K, dtype=torch.int32, device=dev)
        self.logp = torch.empty(N, B, K, dtype=torch.float32, device=dev)
        self.topk_workspace = topk_workspace(N, B, V, K, dev)
        self.draft = torch.empty(N, B, dtype=torch.int32, device=dev)
        self.choice = torch.empty(N, B, dtype=torch.int32, device=dev)
        self.logq = torch.empty(N, B, dtype=torch.float32, device=dev)
        self.score = (torch.empty(N, dtype=torch.float32, device=dev) if decode == "exact"
                      else None)
        self.rescored = (torch.empty(N, B, dtype=torch.int32, device=dev)
                         if decode == "certified" else None)
        self.S = self.S0 = None
        if scores:
            self.S = torch.empty(N, max(B - 1, 0), K, K, dtype=torch.float32, device=dev)
            self.S0 = (torch.empty(N, K, dtype=torch.float32, device=dev)
                       if anchor_out is not None else None)
        ws_fn = {"greedy": score_walk_workspace, "certified": score_walk_certified_workspace,
                 "exact": score_viterbi_workspace}[decode]
        self.fused_workspace = ws_fn(N, B, K, dev)
        self.in_vec = self.out_vec = None
        if E.dtype != torch.bfloat16 or d > 256:
            self.in_vec = torch.empty(N, B, K, d, dtype=torch.float32, device=dev)
            self.out_vec = torch.empty_like(self.in_vec)
        a = BlockArgs()
        a.logits = _dev(logits, "logits", (torch.bfloat16, torch.float32))
        a.logits_dtype = _dtype_code(logits)
        a.N, a.B, a.V, a.K = N, B, V, K
        a.ids, a.logp = self.ids.data_ptr(), self.logp.data_ptr()
        a.topk_workspace = self.topk_workspace.data_ptr()
        a.topk_workspace_bytes = self.topk_workspace.numel()
        a.E = _dev(E, "E", (torch.bfloat16, torch.float32))
        a.e_dtype = _dtype_code(E)
        a.e_rows, a.d = rows, d
        a.packed_w = _dev(packed, "packed")
        a.anchor_out = _dev(anchor_out, "anchor_out", (torch.float32,))
        a.sigma, a.logp_weight = float(sigma), float(logp_weight)
        a.decode, a.margin = DECODE[decode], float(margin)
        a.S = self.S.data_ptr() if self.S is not None and B > 1 else None
        a.S0 = self.S0.data_ptr() if self.S0 is not None else None
        a.draft, a.choice, a.logq = (self.draft.data_ptr(), self.choice.data_ptr(),
                                     self.logq.data_ptr())
        a.score = self.score.data_ptr() if self.score is not None else None
        a.rescored = self.rescored.data_ptr() if self.rescored is not None else None
        a.fused_workspace = self.fused_workspace.data_ptr()
        a.fused_workspace_bytes = self.fused_workspace.numel()
        if self.in_vec is not None:
            a.in_vec, a.out_vec = self.in_vec.data_ptr(), self.out_vec.data_ptr()
        self.args = a
        self._graph = lilicorr_block_graph_create(a)

    def launch(self) -> None:
        if self._graph is None:
            raise LilicorrError("the graph was closed")
        lilicorr_block_graph_launch(self._graph, _stream())

    def close(self) -> None:
        """Releases the graph; the caller makes sure no replay is still running."""
        if self._graph is not None:
            lilicorr_block_graph_destroy(self._graph)
            self._graph = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def draft_block(logits: torch.Tensor, K: int, E: torch.Tensor, packed: torch.Tensor,
                anchor_out=None, sigma: float = SIGMA, logp_weight: float = 0.0):
    """The whole path on one stream: top-K -> vectors -> pair scores -> greedy walk."""
    ids, logp = topk(logits, K)
    in_vec, out_vec = candidate_vectors(ids, E, packed)
    S, S0 = pair_scores(in_vec, out_vec, anchor_out, sigma)
    draft, choice, logq = greedy_walk(S, S0, logp, ids, logp_weight)
    return {"ids": ids, "logp": logp, "in_vec": in_vec, "out_vec": out_vec, "S": S, "S0": S0,
            "draft": draft, "choice": choice, "logq": logq}


# ---- scoring-Transformer stand-in ---------------------------------------------------------------

def lilicorr_scorer_packed_bytes(H: int, heads: int, F: int, S: int) -> int:
    return load_library().lilicorr_scorer_packed_bytes(H, heads, F, S)


def lilicorr_scorer_pack(layer: ScorerLayer, H, heads, F, S, packed, stream) -> int:
    return _call("lilicorr_scorer_pack", ctypes.byref(layer), H, heads, F, S, packed, stream)


def lilicorr_scorer_workspace_bytes(N: int, S: int, K: int, H: int, F: int) -> int:
    return load_library().lilicorr_scorer_workspace_bytes(N, S, K, H, F)


def lilicorr_scorer_forward(X, N, S, K, H, heads, F, layers, packed, workspace, workspace_bytes,
                            stream) -> int:
    return _call("lilicorr_scorer_forward", X, N, S, K, H, heads, F, layers, packed, workspace,
                 workspace_bytes, stream)


def scorer_pack(layers: list, S: int) -> torch.Tensor:
    """Packs the layers (dicts of device tensors: w_qkv [H,3H], w_o [H,H], w_1 [H,F], w_2 [F,H]
    bf16; g_attn, g_ffn [H], dist_bias [heads, 2S-1], same_bias [heads] fp32) back to back."""
    H = layers[0]["w_qkv"].shape[0]
    F = layers[0]["w_1"].shape[1]
    heads = layers[0]["same_bias"].shape[0]
    nb = lilicorr_scorer_packed_bytes(H, heads, F, S)
    if nb == 0:
        raise LilicorrError(f"scorer does not support H={H}, heads={heads}, F={F}, S={S}")
    out = torch.empty(len(layers) * nb, dtype=torch.uint8, device=layers[0]["w_qkv"].device)
    shapes = {"w_qkv": (H, 3 * H), "w_o": (H, H), "w_1": (H, F), "w_2": (F, H), "g_attn": (H,),
              "g_ffn": (H,), "dist_bias": (heads, 2 * S - 1), "same_bias": (heads,)}
    for i, l in enumerate(layers):
        ptrs = {}
        for name, shape in shapes.items():
            t = l[name]
            if tuple(t.shape) != shape:
                raise LilicorrError(f"layer {i} {name} has shape {tuple(t.shape)}, expected {shape}")
            want = (torch.bfloat16,) if name.startswith("w_") else (torch.float32,)
            ptrs[name] = _dev(t, name, want)
        lilicorr_scorer_pack(ScorerLayer(**ptrs), H, heads, F, S, out.data_ptr() + i * nb, _stream())
    return out


def scorer_workspace(N: int, S: int, K: int, H: int, F: int, device="cuda") -> torch.Tensor:
    need = lilicorr_scorer_workspace_bytes(N, S, K, H, F)
    if need == 0:
        raise LilicorrError(f"scorer does not support N={N}, S={S}, K={K}, H={H}, F={F}")
    return torch.empty(need, dtype=torch.uint8, device=device)


def scorer_forward(X: torch.Tensor, packed: torch.Tensor, S: int, K: int, heads: int, F: int,
                   layers: int, *, workspace=None) -> torch.Tensor:
    """Runs the packed layers over X [N, S*K, H] fp32 in place; returns X."""
    N, L, H = X.shape
    if L != S * K:
        raise LilicorrError(f"X has {L} nodes per request, expected S*K = {S * K}")
    ws = workspace if workspace is not None else scorer_workspace(N, S, K, H, F, X.device)
    lilicorr_scorer_forward(_dev(X, "X", (torch.float32,)), N, S, K, H, heads, F, layers,
                            _dev(packed, "packed"), _dev(ws, "workspace"), ws.numel(), _stream())
    return X
