"""CPU oracle of the scoring-Transformer stand-in (fp64, numpy).

TEST INFRASTRUCTURE ONLY. Imported by tests/, by the smoke check and by the benchmark's
CPU-baseline leg; the product path never imports it. It shares no code with the HIP library.

What is computed (implementation appendix, "Architecture"; hyper-parameter table): a stack of
bidirectional Transformer layers over one request's candidate lattice of S slots x K candidates
(L = S * K nodes, node j in slot j // K), hidden width H, `heads` attention heads of width
H / heads, feed-forward width F, RMSNorm and SiLU. Node order enters only through per-head
scalars summed into the pre-softmax scores: a table looked up by (query slot - key slot), and one
value for pairs of nodes in the same slot.

Readings of what the paper leaves open (each listed in the design notes):
  * pre-norm residual blocks: x += Wo . attn(rmsnorm(x; g_attn)); x += W2 . silu(W1 . rmsnorm(x;
    g_ffn)); no biases in the linear maps, no final norm (the head's next step is a linear map);
  * RMSNorm: x / sqrt(mean(x^2) + eps) * g with eps = 1e-6;
  * attention logits scaled by 1 / sqrt(H / heads); every node attends to every node of its own
    request, itself included;
  * precision of the stand-in: weights are bf16; every matrix-product input (the normalised
    activations, Q, K, V, the attention probabilities, the attention output, the SiLU output) is
    rounded to bf16 (round to nearest, ties to even); products are exact and sums are carried in
    fp64 here; the residual stream stays in full precision.
Functions take `exact=True` to skip every bf16 rounding (used by the pins against library
routines). Parity status: pinned by tests/test_oracle_scorer.py.
"""
from __future__ import annotations

import math

import numpy as np

EPS = 1e-6


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """uint16 bf16 bit patterns -> their exact values as float64."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bf16 value (8 significant bits; ties to even), directly
    from float64 (no intermediate fp32 rounding). Finite inputs in bf16's normal range."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                     # x = m * 2^e, 0.5 <= |m| < 1
    r = np.rint(np.ldexp(m, 8))            # 8 significant bits; np.rint rounds half to even
    return np.ldexp(r, e - 8)


def _q(x, exact):
    return x if exact else bf16_round(x)


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float = EPS) -> np.ndarray:
    """x / sqrt(mean over the last axis of x^2 + eps) * g."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(g, np.float64)


def silu(x: np.ndarray) -> np.ndarray:
    """x * sigmoid(x)."""
    x = np.asarray(x, dtype=np.float64)
    return x / (1.0 + np.exp(-x))


def lattice_bias(S: int, K: int, dist_bias: np.ndarray, same_bias: float) -> np.ndarray:
    """[L][L] additive attention bias of one head: dist_bias[(S - 1) + s_i - s_j], plus same_bias
    when s_i == s_j (s = node // K)."""
    s = np.arange(S * K) // K
    delta = s[:, None] - s[None, :]
    return np.asarray(dist_bias, np.float64)[(S - 1) + delta] + np.where(delta == 0, same_bias, 0.0)


def lattice_attention(q, k, v, S, K, dist_bias, same_bias, exact=False):
    """One head over one request: q, k, v [L][dh] (already rounded to bf16 unless exact).
    Returns softmax(q k^T / sqrt(dh) + bias) v, the probabilities rounded to bf16 before the
    product unless exact."""
    dh = q.shape[-1]
    z = (q @ k.T) / math.sqrt(dh) + lattice_bias(S, K, dist_bias, same_bias)
    z = z - z.max(axis=-1, keepdims=True)
    p = np.exp(z)
    p = p / p.sum(axis=-1, keepdims=True)
    return _q(p, exact) @ v


def scorer_layer(X: np.ndarray, layer: dict, S: int, K: int, heads: int, eps: float = EPS,
                 exact: bool = False) -> np.ndarray:
    """One pre-norm layer over X [N][L][H] (float64); returns the new residual stream.

    layer: w_qkv [H][3H], w_o [H][H], w_1 [H][F], w_2 [F][H] (float64 values of bf16 weights,
    applied as y = x @ W; Q, K, V are columns [0, H), [H, 2H), [2H, 3H), head h owning columns
    h*dh .. h*dh + dh - 1 of each), g_attn [H], g_ffn [H], dist_bias [heads][2S - 1],
    same_bias [heads]."""
    X = np.asarray(X, dtype=np.float64)
    N, L, H = X.shape
    assert L == S * K and H % heads == 0
    dh = H // heads
    # attention block
    xn = _q(rms_norm(X, layer["g_attn"], eps), exact)
    qkv = _q(xn @ layer["w_qkv"], exact)
    att = np.empty((N, L, H))
    for n in range(N):
        for h in range(heads):
            cols = slice(h * dh, (h + 1) * dh)
            q = qkv[n, :, 0 * H:1 * H][:, cols]
            k = qkv[n, :, 1 * H:2 * H][:, cols]
            v = qkv[n, :, 2 * H:3 * H][:, cols]
            att[n, :, cols] = lattice_attention(q, k, v, S, K, layer["dist_bias"][h],
                                                float(layer["same_bias"][h]), exact)
    X = X + _q(att, exact) @ layer["w_o"]
    # feed-forward block
    hn = _q(rms_norm(X, layer["g_ffn"], eps), exact)
    a = _q(silu(hn @ layer["w_1"]), exact)
    return X + a @ layer["w_2"]


def layer_from_arrays(w_qkv, w_o, w_1, w_2, g_attn, g_ffn, dist_bias, same_bias) -> dict:
    """A layer dict from host arrays: weights as uint16 bf16 bit patterns, the rest fp32."""
    f = lambda a: np.asarray(a, dtype=np.float64)
    return {"w_qkv": bf16_bits_to_f64(w_qkv), "w_o": bf16_bits_to_f64(w_o),
            "w_1": bf16_bits_to_f64(w_1), "w_2": bf16_bits_to_f64(w_2),
            "g_attn": f(g_attn), "g_ffn": f(g_ffn), "dist_bias": f(dist_bias),
            "same_bias": f(same_bias)}


def scorer_forward(X: np.ndarray, layers: list, S: int, K: int, heads: int, eps: float = EPS,
                   exact: bool = False) -> np.ndarray:
    """The layer stack over X [N][S*K][H]; returns float64 (the library's output is its fp32
    rounding)."""
    X = np.asarray(X, dtype=np.float64)
    for layer in layers:
        X = scorer_layer(X, layer, S, K, heads, eps, exact)
    return X
