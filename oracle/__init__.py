"""CPU oracle of the LiLiCorr draft-correlation path (ctypes wrapper over lilicorr_oracle.c).

TEST INFRASTRUCTURE ONLY. Imported by tests/, by the smoke check and by the benchmark's
CPU-baseline leg; the product path never imports it. It shares no code with the HIP library.

All arrays are numpy, C-contiguous, on the host. bf16 tensors are passed as their uint16 bit
patterns. Each function mirrors one call of the library and returns fresh output arrays.
Parity status of every function is pinned by tests/test_oracle_*.py (see the design notes).
The scoring-Transformer stand-in's oracle is the numpy module `oracle.scorer`.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lilicorr_oracle.c")
_LIB = os.path.join(_HERE, "liblilicorr_oracle.so")

F32, BF16 = 0, 1

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, no fast-math, no fused multiply-add contraction,
    single-threaded)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-std=c11", "-fPIC", "-shared",
                               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        lib = ctypes.CDLL(_LIB)
        P, I64, I = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
        lib.oracle_topk.argtypes = [P, I, I64, I64, I64, I, P, P]
        lib.oracle_candidate_vectors.argtypes = [P, P, I, I64, I, P, P, I64, I64, I, P, P]
        lib.oracle_pair_scores.argtypes = [P, P, P, I64, I64, I, I, ctypes.c_float, P, P]
        lib.oracle_greedy_walk.argtypes = [P, P, P, P, I64, I64, I, ctypes.c_float, P, P, P]
        lib.oracle_viterbi_walk.argtypes = [P, P, P, P, I64, I64, I, ctypes.c_float, P, P, P, P]
        lib.oracle_candidate_features.argtypes = [P, I64, I, P]
        for f in (lib.oracle_topk, lib.oracle_candidate_vectors, lib.oracle_pair_scores,
                  lib.oracle_greedy_walk, lib.oracle_viterbi_walk, lib.oracle_candidate_features):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.uint16:
        return BF16
    raise TypeError(f"unsupported dtype {a.dtype} (float32 or uint16 bf16 bits)")


def _check(rc: int, what: str):
    if rc != 0:
        raise ValueError(f"oracle {what}: arguments break its preconditions")


def topk(logits: np.ndarray, K: int):
    """logits [N, B, V] float32 or bf16-bits uint16 -> ids [N, B, K] int32, logp [N, B, K] f32."""
    logits = np.ascontiguousarray(logits)
    N, B, V = logits.shape
    ids = np.zeros((N, B, K), np.int32)
    logp = np.zeros((N, B, K), np.float32)
    _check(_load().oracle_topk(_ptr(logits), _dtype_code(logits), N, B, V, K, _ptr(ids),
                               _ptr(logp)), "topk")
    return ids, logp


def candidate_vectors(ids: np.ndarray, E: np.ndarray, W_in: np.ndarray, W_out: np.ndarray):
    """ids [N, B, K] int32, E [V, d], W [d, d] f32 -> in_vec, out_vec [N, B, K, d] f32."""
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    E = np.ascontiguousarray(E)
    W_in = np.ascontiguousarray(W_in, dtype=np.float32)
    W_out = np.ascontiguousarray(W_out, dtype=np.float32)
    N, B, K = ids.shape
    V, d = E.shape
    in_vec = np.zeros((N, B, K, d), np.float32)
    out_vec = np.zeros((N, B, K, d), np.float32)
    _check(_load().oracle_candidate_vectors(_ptr(ids), _ptr(E), _dtype_code(E), V, d,
                                            _ptr(W_in), _ptr(W_out), N, B, K, _ptr(in_vec),
                                            _ptr(out_vec)), "candidate_vectors")
    return in_vec, out_vec


def pair_scores(in_vec: np.ndarray, out_vec: np.ndarray, anchor_out=None, sigma: float = 8.0):
    """in/out [N, B, K, d] f32 (+ anchor_out [N, d]) -> S [N, B-1, K, K], S0 [N, K] or None."""
    in_vec = np.ascontiguousarray(in_vec, dtype=np.float32)
    out_vec = np.ascontiguousarray(out_vec, dtype=np.float32)
    N, B, K, d = in_vec.shape
    S = np.zeros((N, max(B - 1, 0), K, K), np.float32)
    S0 = None
    if anchor_out is not None:
        anchor_out = np.ascontiguousarray(anchor_out, dtype=np.float32)
        S0 = np.zeros((N, K), np.float32)
    _check(_load().oracle_pair_scores(_ptr(in_vec), _ptr(out_vec), _ptr(anchor_out), N, B, K,
                                      d, float(sigma), _ptr(S), _ptr(S0)), "pair_scores")
    return S, S0


def greedy_walk(S: np.ndarray, S0, logp: np.ndarray, ids: np.ndarray, logp_weight: float = 0.0):
    """-> draft [N, B] int32, choice [N, B] int32, logq [N, B] f32."""
    logp = np.ascontiguousarray(logp, dtype=np.float32)
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    N, B, K = ids.shape
    S = np.ascontiguousarray(S, dtype=np.float32)
    if S0 is not None:
        S0 = np.ascontiguousarray(S0, dtype=np.float32)
    draft = np.zeros((N, B), np.int32)
    choice = np.zeros((N, B), np.int32)
    logq = np.zeros((N, B), np.float32)
    _check(_load().oracle_greedy_walk(_ptr(S), _ptr(S0), _ptr(logp), _ptr(ids), N, B, K,
                                      float(logp_weight), _ptr(draft), _ptr(choice), _ptr(logq)),
           "greedy_walk")
    return draft, choice, logq


def viterbi_walk(S: np.ndarray, S0, logp: np.ndarray, ids: np.ndarray, logp_weight: float = 0.0):
    """Exact max-path decode -> draft [N, B] int32, choice [N, B] int32, logq [N, B] f32,
    score [N] f32 (the path score g)."""
    logp = np.ascontiguousarray(logp, dtype=np.float32)
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    N, B, K = ids.shape
    S = np.ascontiguousarray(S, dtype=np.float32)
    if S0 is not None:
        S0 = np.ascontiguousarray(S0, dtype=np.float32)
    draft = np.zeros((N, B), np.int32)
    choice = np.zeros((N, B), np.int32)
    logq = np.zeros((N, B), np.float32)
    score = np.zeros((N,), np.float32)
    _check(_load().oracle_viterbi_walk(_ptr(S), _ptr(S0), _ptr(logp), _ptr(ids), N, B, K,
                                       float(logp_weight), _ptr(draft), _ptr(choice), _ptr(logq),
                                       _ptr(score)), "viterbi_walk")
    return draft, choice, logq, score


def candidate_features(logp: np.ndarray) -> np.ndarray:
    """logp [..., K] f32 (sorted top-K log-probabilities) -> feat [..., K, 5] f32."""
    logp = np.ascontiguousarray(logp, dtype=np.float32)
    K = logp.shape[-1]
    rows = int(np.prod(logp.shape[:-1]))
    feat = np.zeros(logp.shape + (5,), np.float32)
    _check(_load().oracle_candidate_features(_ptr(logp), rows, K, _ptr(feat)), "candidate_features")
    return feat
