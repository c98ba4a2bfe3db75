"""Seeded synthetic inputs for the LiLiCorr draft-correlation path.

This module only draws random numbers and lays them out; it holds none of the method's
arithmetic (no normalisation, selection, projection, scoring or decoding), so both the CPU
oracle and the HIP path can take their inputs from it without sharing any of the method.

The paper's own workloads (DFlash marginals over the Qwen3 vocabulary on SPEED and nine
public benchmarks, trained head weights) are not available; these tensors stand in for them
with the shapes of the paper's serving setting (block of 16 slots, Sec. 4.1 and the
hyper-parameter table of the implementation appendix) and with output-entropy tiers in the
spirit of the SPEED throughput split (Sec. 4.3).

Every tensor is drawn from its own ``torch.Generator`` whose seed is a fixed function of the
config seed, a tensor tag and, for logits, the request index, so one request's logits can be
regenerated on its own (used to sample full-size cases for the oracle).

Recipe per config (index: shapes; logits; vectors):

0: N=1, B=8, K=4, V=32000, d=64. fp32 logits N(0,1), +6 at one uniform id per slot.
   E [V,64] fp32 N(0,1); W_in, W_out [64,64] fp32 N(0,1/64).
1: N=1, B=16, K=8, V=151936, d=256. N(0,2^2) plus a Zipf(1.1)-ranked bump 4*r^-1.1 on 32
   distinct uniform ids (rank r=1..32), rounded to bf16 (RNE). E [V,256] bf16 N(0,0.02^2);
   W [256,256] fp32 N(0,1/256).
2: N=16, B=16, K=16, V=151936, d=256. As 1, with the noise std drawn per request from
   {0.5, 2, 4}.
3: N=64, B=16, K=16, V=151936, d=256. As 2 with the std chosen round-robin (request n takes
   [0.5, 2, 4][n % 3]), then 1% exact ties: in each slot ceil(0.01 V) = 1520 distinct uniform ids
   each take the bf16 value of an id drawn uniformly from that slot's 2K highest-ranked ids.
4: N=256, B=16, K=32, V=262144, d=512. bf16 N(0,3^2); +8 at one uniform id in each slot of a
   Bernoulli(1/2) subset of slots. E [V,512] bf16 N(0,0.02^2); W [512,512] fp32 N(0,1/512).

Scoring-Transformer stand-in (a cost-only stand-in of the head's encoder: random weights, no
trained values exist here). ScorerConfig: N requests, S slots, K candidates (L = S*K nodes),
width H, heads, feed-forward width F, layers. Node states X [N][L][H] fp32 N(0,1); per layer:
w_qkv [H][3H], w_o [H][H], w_1 [H][F] bf16 N(0, 1/H), w_2 [F][H] bf16 N(0, 1/F); RMSNorm gains
g_attn, g_ffn [H] fp32 1 + 0.1 N(0,1); attention biases dist_bias [heads][2S-1] and
same_bias [heads] fp32 0.5 N(0,1). The headline shape is N=64, S=15 (16-slot blocks, 15 drafted),
K=16, H=1024, 8 heads, F=2048, 2 layers (the paper's head widths and depth).

Measured softmax entropy over V=151936 without bumps: std 0.5 -> 11.8 nats (high-entropy
tier), std 2 -> 9.9 nats (mid), std 4 -> 5.0 nats (low).
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import torch

__all__ = ["Config", "CONFIGS", "config", "make_logits", "make_request_logits",
           "make_embedding", "make_weights", "make_inputs", "make_anchor", "ScorerConfig",
           "SCORER_HEADLINE", "make_scorer_inputs"]


@dataclass(frozen=True)
class Config:
    index: int
    name: str
    N: int
    B: int
    K: int
    V: int
    d: int
    logits_dtype: torch.dtype
    e_dtype: torch.dtype
    seed: int

    @property
    def rows(self) -> int:
        return self.N * self.B


CONFIGS = [
    Config(0, "tiny", 1, 8, 4, 32000, 64, torch.float32, torch.float32, 0),
    Config(1, "single", 1, 16, 8, 151936, 256, torch.bfloat16, torch.bfloat16, 1),
    Config(2, "tiers16", 16, 16, 16, 151936, 256, torch.bfloat16, torch.bfloat16, 2),
    Config(3, "headline64", 64, 16, 16, 151936, 256, torch.bfloat16, torch.bfloat16, 3),
    Config(4, "stress256", 256, 16, 32, 262144, 512, torch.bfloat16, torch.bfloat16, 4),
]

_TIER_STD = (0.5, 2.0, 4.0)

# tensor tags (part of each generator's seed)
_TAG_LOGITS, _TAG_E, _TAG_WIN, _TAG_WOUT, _TAG_TIER, _TAG_ANCHOR = 1, 2, 3, 4, 5, 6


def config(i: int) -> Config:
    return CONFIGS[i]


def _gen(seed: int, tag: int, sub: int = 0) -> torch.Generator:
    return torch.Generator().manual_seed(((seed * 1_000_003 + tag) * 1_000_033 + sub) & ((1 << 62) - 1))


def _request_std(cfg: Config, n: int) -> float:
    if cfg.index in (1,):
        return 2.0
    if cfg.index == 2:
        g = _gen(cfg.seed, _TAG_TIER)
        picks = torch.randint(0, 3, (cfg.N,), generator=g)
        return _TIER_STD[int(picks[n])]
    if cfg.index == 3:
        return _TIER_STD[n % 3]
    if cfg.index == 4:
        return 3.0
    return 1.0


def make_request_logits(cfg: Config, n: int) -> torch.Tensor:
    """Logits of request n, shape [B, V], dtype cfg.logits_dtype (CPU)."""
    B, V, K = cfg.B, cfg.V, cfg.K
    g = _gen(cfg.seed, _TAG_LOGITS, n)
    std = _request_std(cfg, n)
    x = torch.randn(B, V, generator=g, dtype=torch.float32)
    x.mul_(std)
    if cfg.index == 0:
        peak = torch.randint(0, V, (B,), generator=g)
        x[torch.arange(B), peak] += 6.0
        return x.contiguous()
    if cfg.index in (1, 2, 3):
        ranks = torch.arange(1, 33, dtype=torch.float64)
        bump = (4.0 * ranks.pow(-1.1)).to(torch.float32)
        for b in range(B):
            ids = torch.randperm(V, generator=g)[:32]
            x[b, ids] += bump
    if cfg.index == 4:
        planted = torch.rand(B, generator=g) < 0.5
        peak = torch.randint(0, V, (B,), generator=g)
        for b in range(B):
            if bool(planted[b]):
                x[b, peak[b]] += 8.0
    y = x.to(torch.bfloat16)  # round to nearest even
    if cfg.index == 3:
        n_tie = math.ceil(0.01 * V)
        for b in range(B):
            row = y[b]
            top = torch.topk(row.float(), 2 * K, sorted=True).indices
            dst = torch.randperm(V, generator=g)[:n_tie]
            src = top[torch.randint(0, 2 * K, (n_tie,), generator=g)]
            row[dst] = row[src].clone()
    return y.contiguous()


def make_logits(cfg: Config) -> torch.Tensor:
    """All logits, shape [N, B, V] (CPU)."""
    out = torch.empty(cfg.N, cfg.B, cfg.V, dtype=cfg.logits_dtype)
    for n in range(cfg.N):
        out[n] = make_request_logits(cfg, n)
    return out


def make_embedding(cfg: Config) -> torch.Tensor:
    """Candidate embedding table E, shape [V, d] (CPU)."""
    g = _gen(cfg.seed, _TAG_E)
    std = 1.0 if cfg.index == 0 else 0.02
    e = torch.randn(cfg.V, cfg.d, generator=g, dtype=torch.float32).mul_(std)
    return e.to(cfg.e_dtype).contiguous()


def make_weights(cfg: Config) -> tuple[torch.Tensor, torch.Tensor]:
    """W_in, W_out, each [d, d] fp32 N(0, 1/d) (CPU); applied as y = e @ W."""
    d = cfg.d
    w_in = torch.randn(d, d, generator=_gen(cfg.seed, _TAG_WIN), dtype=torch.float32) / math.sqrt(d)
    w_out = torch.randn(d, d, generator=_gen(cfg.seed, _TAG_WOUT), dtype=torch.float32) / math.sqrt(d)
    return w_in.contiguous(), w_out.contiguous()


def make_anchor(cfg: Config) -> torch.Tensor:
    """Optional anchor out vectors [N, d] fp32 N(0,1) (not unit norm; the scores normalise)."""
    g = _gen(cfg.seed, _TAG_ANCHOR)
    return torch.randn(cfg.N, cfg.d, generator=g, dtype=torch.float32).contiguous()


def make_inputs(cfg: Config) -> dict:
    w_in, w_out = make_weights(cfg)
    return {"logits": make_logits(cfg), "E": make_embedding(cfg), "W_in": w_in, "W_out": w_out}


@dataclass(frozen=True)
class ScorerConfig:
    N: int
    S: int
    K: int
    H: int = 1024
    heads: int = 8
    F: int = 2048
    layers: int = 2
    seed: int = 7

    @property
    def L(self) -> int:
        return self.S * self.K


SCORER_HEADLINE = ScorerConfig(N=64, S=15, K=16)

_TAG_SX, _TAG_SW = 11, 12


def make_scorer_inputs(sc: ScorerConfig) -> dict:
    """{"X": [N][L][H] fp32, "layers": [dict of CPU tensors per layer]} (see the module notes)."""
    H, F, S, heads = sc.H, sc.F, sc.S, sc.heads
    X = torch.randn(sc.N, sc.L, H, generator=_gen(sc.seed, _TAG_SX), dtype=torch.float32)
    layers = []
    for i in range(sc.layers):
        g = _gen(sc.seed, _TAG_SW, i)
        w = lambda r, c, fan: (torch.randn(r, c, generator=g) / math.sqrt(fan)).to(torch.bfloat16)
        layers.append({
            "w_qkv": w(H, 3 * H, H).contiguous(), "w_o": w(H, H, H).contiguous(),
            "w_1": w(H, F, H).contiguous(), "w_2": w(F, H, F).contiguous(),
            "g_attn": (1 + 0.1 * torch.randn(H, generator=g)).contiguous(),
            "g_ffn": (1 + 0.1 * torch.randn(H, generator=g)).contiguous(),
            "dist_bias": (0.5 * torch.randn(heads, 2 * S - 1, generator=g)).contiguous(),
            "same_bias": (0.5 * torch.randn(heads, generator=g)).contiguous(),
        })
    return {"X": X.contiguous(), "layers": layers}
