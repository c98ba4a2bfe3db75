#!/usr/bin/env python3
"""Benchmark of the LiLiCorr draft-correlation hot path on one MI355X.

One step = the whole path over one batch of synthetic input, on one stream:
    lilicorr_topk -> lilicorr_score_walk (candidate vectors, pair scores and greedy walk in one
    pass, the in/out vectors kept on chip)
for the headline workload (N = 64 requests, B = 16 slots, K = 16 candidates, V = 151936,
d = 256, bf16 logits). The metric is scored draft blocks per second (N blocks per step). Logits
rotate over four resident copies (1.2 GB, above the 256 MB Infinity Cache) so every step streams
its logits from HBM; the embedding table and packed weights stay resident, as served weights do.
The same steps through the four separate calls (topk -> candidate_vectors -> pair_scores ->
greedy_walk, in/out vectors through HBM) are timed too and reported beside it.

The timed loop calls the C ABI directly (arguments marshalled once), two calls per block; the
same block recorded once as a HIP graph per logits buffer and replayed with one
lilicorr_block_graph_launch per block is timed beside it.

Printed: one JSON line with the step throughput, a roofline entry for the dominant kernel (the
logits pass, its mean duration over back-to-back launches between two HIP events on the launch
stream), the logits-pass bandwidth at the stress workload (N = 256, K = 32, V = 262144), and the
CPU oracle timed on a bounded sample of the same workload on this host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "scored draft blocks/sec at N=64,B=16,K=16,V=151936; logits-pass HBM GB/s"
PEAK_HBM_GBS = 8000.0
ROTATE = 4
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "topk_lse_headline64_traffic.json")
TOPK_SRC = os.path.join(ROOT, "paper_2608_20530_amd", "csrc", "topk.hip")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-stress", action="store_true", help="skip the stress logits-pass line")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-scorer", action="store_true",
                    help="skip the scoring-Transformer stand-in line")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-workload line (both metrics at every workload)")
    ap.add_argument("--no-two-streams", action="store_true",
                    help="skip the two-stream timing (profiling runs of the one-stream kernels)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 1 GiB device copy (counter calibration under rocprofv3)")
    ap.add_argument("--workload-step", choices=["tiny", "single", "tiers16", "headline64",
                                                "stress256"],
                    help="only the per-workload step at one workload (for profiling runs): "
                         "prints its line and exits")
    ap.add_argument("--logits-only", choices=["headline", "stress"],
                    help="only the logits pass at one workload (for profiling runs): prints its "
                         "line and exits")
    return ap.parse_args()


def topk_kernel_hash() -> str:
    return hashlib.sha256(open(TOPK_SRC, "rb").read()).hexdigest()[:16]


def traffic_per_launch():
    """HBM bytes per logits-pass launch from the committed counter summary, or None when the
    kernel source changed since the counters were taken."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    if rec.get("topk_source_sha256_16") != topk_kernel_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


def time_logits_pass(L, torch, cfg, logits_list, iters, batches=5):
    """Logits-pass duration (s) at one workload: after three untimed batches, `batches` batches of
    `iters` back-to-back launches over the rotating buffers, each between two HIP events on the
    launch stream; returns the mean, smallest and largest per-launch mean of the batches."""
    K = cfg.K
    N, B, V = logits_list[0].shape
    ids = torch.empty(N, B, K, dtype=torch.int32, device="cuda")
    logp = torch.empty(N, B, K, dtype=torch.float32, device="cuda")
    ws = L.topk_workspace(N, B, V, K)
    lib = L.load_library()
    stream = torch.cuda.current_stream().cuda_stream
    args = [(lg.data_ptr(), L.BF16 if lg.dtype == torch.bfloat16 else L.F32, N, B, V, K,
             ids.data_ptr(), logp.data_ptr(), ws.data_ptr(), ws.numel(), stream)
            for lg in logits_list]

    def batch():
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for i in range(iters):
            lib.lilicorr_topk(*args[i % len(args)])
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / 1e3 / iters

    for _ in range(3):
        batch()
    t = [batch() for _ in range(batches)]
    if L.topk_wait_status(ws) != 0:
        raise RuntimeError("a bounded wait of the logits pass gave up: outputs invalid")
    return statistics.mean(t), min(t), max(t)


def stream_reader(torch):
    """A launcher of the plain streaming read (16-byte streaming-policy buffer loads, the logits
    pass's own load path, one contiguous segment per workgroup) of one resident buffer, queued on
    the current stream."""
    import ctypes

    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2608_20530_amd", "libbench_read.so"))
    lib.bench_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                      ctypes.c_int, ctypes.c_void_p]
    lib.bench_stream_read.restype = ctypes.c_int
    grid = 1024
    sink = torch.empty(grid * 256, dtype=torch.int32, device="cuda")

    def read(b):
        rc = lib.bench_stream_read(b.data_ptr(), b.numel() * b.element_size(), sink.data_ptr(),
                                   grid, torch.cuda.current_stream().cuda_stream)
        if rc != 0:
            raise RuntimeError(f"bench_stream_read failed ({rc})")
    return read


def stream_read_rate(torch, bufs, iters=20, batches=3):
    """GB/s of the plain streaming read over the same resident buffers, rotated and timed like the
    logits pass (batches of `iters` back-to-back launches between two HIP events, after one
    untimed batch; the mean per-launch time): the read ceiling the logits pass is compared with."""
    read = stream_reader(torch)

    def batch():
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for i in range(iters):
            read(bufs[i % len(bufs)])
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / 1e3 / iters

    batch()
    sec = statistics.mean(batch() for _ in range(batches))
    nbytes = bufs[0].numel() * bufs[0].element_size()
    return nbytes / sec / 1e9


def median_launch_us(torch, fn, iters=50, warmup=5):
    """Median duration of one call of fn, from HIP events on the current stream."""
    for _ in range(warmup):
        fn()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(iters)]
    torch.cuda.synchronize()
    for a, b in ev:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    return statistics.median(a.elapsed_time(b) for a, b in ev) * 1e3


def per_config_rates(L, torch, c, inp, iters=100, warmup=10, batches=10):
    """Both metrics at one workload: blocks/s of the step (logits pass, then the fused pass or the
    separate calls, through the C ABI with arguments marshalled once) and the logits pass's GB/s,
    each over `iters` back-to-back calls in `batches` batches between two HIP events (the mean,
    and the median, p10 and p90 of the batch means), beside a plain streaming read of the same
    logits buffers timed the same way. The logits rotate over enough resident copies (at least
    1 GiB in all) that every call reads its logits from HBM, as in the headline loop."""
    lg = inp["logits"].cuda()
    nbytes = lg.numel() * lg.element_size()
    copies = max(1, min(1024, -(-(1 << 30) // nbytes)))
    lgs = [lg] + [lg.clone() for _ in range(copies - 1)]
    E = inp["E"].cuda()
    packed = L.pack_weights(inp["W_in"].cuda(), inp["W_out"].cuda())
    N, B, K, V = c.N, c.B, c.K, c.V
    ids = torch.empty(N, B, K, dtype=torch.int32, device="cuda")
    logp = torch.empty(N, B, K, dtype=torch.float32, device="cuda")
    ws = L.topk_workspace(N, B, V, K)
    draft = torch.empty(N, B, dtype=torch.int32, device="cuda")
    choice = torch.empty_like(draft)
    logq = torch.empty(N, B, dtype=torch.float32, device="cuda")
    # the fused pass holds both sides' fp32 projections in LDS (bf16 tables, d <= 256); other
    # workloads take the candidate vectors, then pair scores and walk in one pass. Every call goes
    # straight to the C ABI with its arguments marshalled once, as in the headline loop.
    lib = L.load_library()
    st = torch.cuda.current_stream().cuda_stream
    e_code = L.BF16 if E.dtype == torch.bfloat16 else L.F32
    l_code = L.BF16 if lg.dtype == torch.bfloat16 else L.F32
    fused = E.dtype == torch.bfloat16 and c.d <= 256
    ws_fused = L.score_walk_workspace(N, B, K)
    if fused:
        walk_args = (ids.data_ptr(), logp.data_ptr(), E.data_ptr(), e_code, V, c.d,
                     packed.data_ptr(), None, N, B, K, L.SIGMA, 0.0, None, None, draft.data_ptr(),
                     choice.data_ptr(), logq.data_ptr(), ws_fused.data_ptr(), ws_fused.numel(), st)

        def rest():
            if lib.lilicorr_score_walk(*walk_args) != 0:
                raise RuntimeError("lilicorr_score_walk failed")
    else:
        in_vec = torch.empty(N, B, K, c.d, dtype=torch.float32, device="cuda")
        out_vec = torch.empty_like(in_vec)
        cv_args = (ids.data_ptr(), E.data_ptr(), e_code, V, c.d, packed.data_ptr(), N, B, K,
                   in_vec.data_ptr(), out_vec.data_ptr(), st)
        pw_args = (in_vec.data_ptr(), out_vec.data_ptr(), None, logp.data_ptr(), ids.data_ptr(), N,
                   B, K, c.d, L.SIGMA, 0.0, None, None, draft.data_ptr(), choice.data_ptr(),
                   logq.data_ptr(), ws_fused.data_ptr(), ws_fused.numel(), st)

        def rest():
            if (lib.lilicorr_candidate_vectors(*cv_args) != 0 or
                    lib.lilicorr_pair_walk(*pw_args) != 0):
                raise RuntimeError("candidate_vectors -> pair_walk failed")

    tk_args = [(x.data_ptr(), l_code, N, B, V, K, ids.data_ptr(), logp.data_ptr(), ws.data_ptr(),
                ws.numel(), st) for x in lgs]

    def topk(i):
        if lib.lilicorr_topk(*tk_args[i % copies]) != 0:
            raise RuntimeError("lilicorr_topk failed")

    counter = [0]
    per = max(1, iters // batches)

    def batch(fn):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for _ in range(per):
            fn(counter[0])
            counter[0] += 1
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / 1e3 / per

    def spread(ts):
        q = sorted(ts)
        return {"median_us": statistics.median(q) * 1e6, "p10_us": q[len(q) // 10] * 1e6,
                "p90_us": q[min(len(q) - 1, (9 * len(q)) // 10)] * 1e6}

    for _ in range(warmup):
        topk(counter[0])
        rest()
        counter[0] += 1
    steps = [batch(lambda i: (topk(i), rest())) for _ in range(batches)]
    topks = [batch(topk) for _ in range(batches)]
    step, t_topk = statistics.mean(steps), statistics.mean(topks)
    if L.topk_wait_status(ws) != 0:
        raise RuntimeError("a bounded wait of the logits pass gave up: outputs invalid")
    read = stream_read_rate(torch, lgs, iters=max(10, min(100, copies * 4)))
    rules = None
    if not fused:
        # steps 3-4 over the vectors of the last step: each decode rule in one pass, and the two
        # separate calls it replaces
        S = torch.empty(N, max(B - 1, 1), K, K, dtype=torch.float32, device="cuda")
        score = torch.empty(N, dtype=torch.float32, device="cuda")
        resc = torch.empty(N, B, dtype=torch.int32, device="cuda")
        ws_x = L.score_viterbi_workspace(N, B, K)
        ws_c = L.score_walk_certified_workspace(N, B, K)
        rules = {
            "pair_walk_us": median_launch_us(torch, lambda: L.pair_walk(
                in_vec, out_vec, logp, ids, out=(draft, choice, logq), workspace=ws_fused)),
            "pair_viterbi_us": median_launch_us(torch, lambda: L.pair_viterbi(
                in_vec, out_vec, logp, ids, out=(draft, choice, logq, score), workspace=ws_x)),
            "separate_pair_scores_greedy_walk_us": median_launch_us(torch, lambda: (
                L.pair_scores(in_vec, out_vec, out=(S, None)),
                L.greedy_walk(S, None, logp, ids, out=(draft, choice, logq)))),
            "note": "median call durations (HIP events, host launch included)",
        }
        if E.dtype == torch.bfloat16:
            rules["pair_walk_certified_us"] = median_launch_us(torch, lambda: L.pair_walk_certified(
                in_vec, out_vec, logp, ids, E, packed, out=(draft, choice, logq, resc),
                workspace=ws_c))
            rules["certified_rescored"] = int((resc > 0).sum())
    return {"workload": f"{c.name}: N={N}, B={B}, K={K}, V={V}, d={c.d}, "
                        f"{'bf16' if lg.element_size() == 2 else 'fp32'} logits",
            "path": "lilicorr_topk -> " + ("lilicorr_score_walk" if fused else
                                            "lilicorr_candidate_vectors -> lilicorr_pair_walk"),
            "logits_copies": copies,
            "blocks_s": N / step, "step_us": step * 1e6, "step_batches": spread(steps),
            "logits_GB_s": nbytes / t_topk / 1e9, "logits_us": t_topk * 1e6,
            "logits_batches": spread(topks),
            "logits_frac_of_8TBs": nbytes / t_topk / 1e9 / PEAK_HBM_GBS,
            "stream_read_GB_s": read, "logits_frac_of_stream_read": nbytes / t_topk / 1e9 / read,
            "decode_rules": rules}


PEAK_BF16_TFLOPS = 2500.0


def scorer_rate(L, torch, workloads, iters=50, warmup=10):
    """The scoring-Transformer stand-in at the headline lattice (64 requests x 15 slots x 16
    candidates, width 1024, 8 heads, feed-forward 2048, two layers): mean forward time over
    back-to-back calls between two HIP events, and its matrix-core rate (algorithmic FLOPs: the
    four GEMMs and both attention products)."""
    sc = workloads.SCORER_HEADLINE
    inp = workloads.make_scorer_inputs(sc)
    layers = [{k: v.cuda() for k, v in l.items()} for l in inp["layers"]]
    packed = L.scorer_pack(layers, sc.S)
    X = inp["X"].cuda()
    ws = L.scorer_workspace(sc.N, sc.S, sc.K, sc.H, sc.F)
    fwd = lambda: L.scorer_forward(X, packed, sc.S, sc.K, sc.heads, sc.F, sc.layers, workspace=ws)
    for _ in range(warmup):
        fwd()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    for _ in range(iters):
        fwd()
    b.record()
    torch.cuda.synchronize()
    us = a.elapsed_time(b) * 1e3 / iters
    M = sc.N * sc.L
    flops = sc.layers * (2 * M * (4 * sc.H * sc.H + 2 * sc.H * sc.F)
                         + sc.N * (sc.H // 128) * 4 * sc.L * sc.L * 128)
    return {"workload": f"N={sc.N} requests, S={sc.S} slots x K={sc.K} candidates, H={sc.H}, "
                        f"{sc.heads} heads, F={sc.F}, {sc.layers} layers, bf16 matrix cores",
            "us_per_forward": us, "TFLOP_s": flops / us / 1e6, "GFLOP": flops / 1e9,
            "frac_of_bf16_peak": flops / us / 1e6 / PEAK_BF16_TFLOPS}


def calibration_copies(torch):
    """Three plain 1 GiB device copies: under rocprofv3 --pmc they calibrate what FETCH_SIZE and
    WRITE_SIZE read for a known number of bytes."""
    src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()


def cpu_baseline(cfg, inp, seconds):
    """The oracle chain, single-threaded, on whole requests of the workload until `seconds`."""
    import numpy as np

    import oracle

    lg = inp["logits"].view(__import__("torch").int16).numpy().view(np.uint16)
    E = inp["E"].view(__import__("torch").int16).numpy().view(np.uint16)
    W_in, W_out = inp["W_in"].numpy(), inp["W_out"].numpy()
    oracle.topk(lg[:1, :1, :64], 4)  # load/compile outside the timing
    done = 0
    t0 = time.perf_counter()
    while done < cfg.N:
        x = lg[done:done + 1]
        ids, logp = oracle.topk(x, cfg.K)
        iv, ov = oracle.candidate_vectors(ids, E, W_in, W_out)
        S, S0 = oracle.pair_scores(iv, ov, None, 8.0)
        oracle.greedy_walk(S, S0, logp, ids)
        done += 1
        if time.perf_counter() - t0 >= seconds:
            break
    dt = time.perf_counter() - t0
    return {"value": done / dt, "unit": "blocks/s", "cores": 1, "kind": "oracle",
            "sample": f"{done} of {cfg.N} requests of the headline workload (whole chain per "
                      f"request, fp64, single thread), {dt:.1f} s"}


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline_threads(cfg, inp, seconds):
    """The same oracle chain on every request of the workload, one request per task on a pool of
    threads (the oracle's C routines release the interpreter lock), so it runs on the host's
    cores; stops taking new requests after `seconds`."""
    import concurrent.futures

    import numpy as np

    import oracle

    lg = inp["logits"].view(__import__("torch").int16).numpy().view(np.uint16)
    E = inp["E"].view(__import__("torch").int16).numpy().view(np.uint16)
    W_in, W_out = inp["W_in"].numpy(), inp["W_out"].numpy()
    oracle.topk(lg[:1, :1, :64], 4)
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    t0 = time.perf_counter()

    def one(n):
        if time.perf_counter() - t0 >= seconds:
            return 0
        ids, logp = oracle.topk(lg[n:n + 1], cfg.K)
        iv, ov = oracle.candidate_vectors(ids, E, W_in, W_out)
        S, S0 = oracle.pair_scores(iv, ov, None, 8.0)
        oracle.greedy_walk(S, S0, logp, ids)
        return 1

    with concurrent.futures.ThreadPoolExecutor(threads) as ex:
        done = sum(ex.map(one, range(cfg.N)))
    dt = time.perf_counter() - t0
    return {"value": done / dt, "unit": "blocks/s", "cores": threads, "kind": "oracle",
            "sample": f"{done} of {cfg.N} requests of the headline workload (whole chain per "
                      f"request, fp64), one request per task on {threads} threads, {dt:.1f} s",
            "cpu_model": cpu_model(), "nproc": os.cpu_count()}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this path has no multi-GPU mode (asked for "
              f"--gpus {args.gpus}); the sharding design is in the design notes", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2608_20530_amd as L
    import workloads

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    L.load_library()

    if args.workload_step:
        c = next(c for c in workloads.CONFIGS if c.name == args.workload_step)
        line = {"per_workload": {c.name: per_config_rates(L, torch, c, workloads.make_inputs(c))}}
        if args.calibrate_copy:
            calibration_copies(torch)
        print(json.dumps(line), flush=True)
        return

    if args.logits_only:
        c = workloads.config(3 if args.logits_only == "headline" else 4)
        lg = workloads.make_logits(c).cuda()
        bufs = [lg] + [lg.clone() for _ in range(ROTATE - 1)] if c.index == 3 else [lg]
        t, lo, hi = time_logits_pass(L, torch, c, bufs, iters=100 if c.index == 3 else 20)
        nb = c.N * c.B * c.V * 2 + c.N * c.B * c.K * 8
        if args.calibrate_copy:
            calibration_copies(torch)
        print(json.dumps({"logits_pass": c.name, "us": t * 1e6, "us_batch_min": lo * 1e6,
                          "us_batch_max": hi * 1e6, "GB_s": nb / t / 1e9,
                          "frac_of_8TBs": nb / t / 1e9 / PEAK_HBM_GBS,
                          "algorithmic_bytes_per_launch": nb}), flush=True)
        return

    cfg = workloads.config(3)
    t_gen = time.perf_counter()
    inp = workloads.make_inputs(cfg)
    t_gen = time.perf_counter() - t_gen
    N, B, K, V, d = cfg.N, cfg.B, cfg.K, cfg.V, cfg.d
    logits0 = inp["logits"].cuda()
    logits_list = [logits0] + [logits0.clone() for _ in range(ROTATE - 1)]
    E = inp["E"].cuda()
    packed = L.pack_weights(inp["W_in"].cuda(), inp["W_out"].cuda())

    dev = "cuda"
    ids = torch.empty(N, B, K, dtype=torch.int32, device=dev)
    logp = torch.empty(N, B, K, dtype=torch.float32, device=dev)
    ws = L.topk_workspace(N, B, V, K)
    in_vec = torch.empty(N, B, K, d, dtype=torch.float32, device=dev)
    out_vec = torch.empty_like(in_vec)
    S = torch.empty(N, B - 1, K, K, dtype=torch.float32, device=dev)
    draft = torch.empty(N, B, dtype=torch.int32, device=dev)
    choice = torch.empty_like(draft)
    logq = torch.empty(N, B, dtype=torch.float32, device=dev)

    ws_fused = L.score_walk_workspace(N, B, K)
    lib = L.load_library()
    stream = torch.cuda.current_stream().cuda_stream

    # The timed step: lilicorr_topk then the fused greedy pass, two C-ABI calls per block with
    # their arguments marshalled once, so the host queues blocks well ahead of the GPU.
    topk_args = [(lg.data_ptr(), L.BF16, N, B, V, K, ids.data_ptr(), logp.data_ptr(),
                  ws.data_ptr(), ws.numel(), stream) for lg in logits_list]
    walk_args = (ids.data_ptr(), logp.data_ptr(), E.data_ptr(), L.BF16, E.shape[0], d,
                 packed.data_ptr(), None, N, B, K, L.SIGMA, 0.0, None, None, draft.data_ptr(),
                 choice.data_ptr(), logq.data_ptr(), ws_fused.data_ptr(), ws_fused.numel(),
                 stream)
    c_topk, c_walk = lib.lilicorr_topk, lib.lilicorr_score_walk

    def step(i):
        if c_topk(*topk_args[i % ROTATE]) != 0 or c_walk(*walk_args) != 0:
            raise RuntimeError("step failed")

    # The same block recorded once as a HIP graph per rotating logits buffer and replayed with
    # one lilicorr_block_graph_launch per block (the implementation appendix's serving recipe).
    graphs = [L.BlockGraph(lg, K, E, packed) for lg in logits_list]
    handles = [gr._graph for gr in graphs]
    graph_launch = lib.lilicorr_block_graph_launch

    def step_graph(i):
        if graph_launch(handles[i % ROTATE], stream) != 0:
            raise RuntimeError("lilicorr_block_graph_launch failed")

    def step_separate(i):
        L.topk(logits_list[i % ROTATE], K, out=(ids, logp), workspace=ws)
        L.candidate_vectors(ids, E, packed, out=(in_vec, out_vec))
        L.pair_scores(in_vec, out_vec, None, L.SIGMA, out=(S, None))
        L.greedy_walk(S, None, logp, ids, 0.0, out=(draft, choice, logq))

    def timed(fn, steps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            fn(i)
        torch.cuda.synchronize()
        return time.perf_counter() - t0

    def topk_batch(reps):
        """Mean duration of one logits-pass launch over `reps` back-to-back launches on the
        rotating buffers, between two HIP events on the launch stream (kernel plus the
        sub-microsecond dispatch gap of a full queue)."""
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for i in range(reps):
            c_topk(*topk_args[i % ROTATE])
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / 1e3 / reps

    # Bring the GPU to its working clock (the inputs were just generated on the host and the GPU
    # sat idle; the first few hundred passes run through a clock dip): 1000 logits passes (~50
    # ms), untimed. Then the logits pass alone, timed, for the roofline entry; then each way
    # through the block: W untimed steps, K timed steps.
    reps = 200
    topk_batch(1000)
    topk_s = topk_batch(reps)
    for i in range(args.warmup):
        step(i)
    elapsed = timed(step, args.steps)
    for i in range(args.warmup):
        step_graph(i)
    graph_elapsed = timed(step_graph, args.steps)
    for i in range(args.warmup):
        step_separate(i)
    sep_elapsed = timed(step_separate, args.steps)
    # Consecutive blocks of independent request batches alternate between two streams (default
    # priority), each with its own outputs and workspaces: one block's correlation pass can run
    # beside the next block's logits pass. Drafts are checked against the one-stream result.
    s2 = torch.cuda.Stream()
    ids2, logp2 = torch.empty_like(ids), torch.empty_like(logp)
    ws2 = L.topk_workspace(N, B, V, K)
    ws_fused2 = L.score_walk_workspace(N, B, K)
    draft2, choice2, logq2 = torch.empty_like(draft), torch.empty_like(choice), torch.empty_like(logq)
    topk_args2 = [(lg.data_ptr(), L.BF16, N, B, V, K, ids2.data_ptr(), logp2.data_ptr(),
                   ws2.data_ptr(), ws2.numel(), s2.cuda_stream) for lg in logits_list]
    walk_args2 = ((ids2.data_ptr(), logp2.data_ptr()) + walk_args[2:15] +
                  (draft2.data_ptr(), choice2.data_ptr(), logq2.data_ptr(), ws_fused2.data_ptr(),
                   ws_fused2.numel(), s2.cuda_stream))

    def step_two_streams(i):
        if i % 2 == 0:
            step(i)
        elif c_topk(*topk_args2[i % ROTATE]) != 0 or c_walk(*walk_args2) != 0:
            raise RuntimeError("step failed")

    two_elapsed = None
    if not args.no_two_streams:
        torch.cuda.synchronize()
        for i in range(args.warmup):
            step_two_streams(i)
        two_elapsed = timed(step_two_streams, args.steps)
        expect = []
        for b in range(2):
            step(b)
            torch.cuda.synchronize()
            expect.append(draft.clone())
        step_two_streams(0)
        step_two_streams(1)
        torch.cuda.synchronize()
        if not (torch.equal(draft, expect[0]) and torch.equal(draft2, expect[1])):
            raise RuntimeError("two-stream drafts differ from the one-stream drafts")
    two_note = "" if two_elapsed is None else f", two streams: {two_elapsed:.4f} s"
    print(f"[bench] timed {args.steps} steps in {elapsed:.4f} s (graph replay: "
          f"{graph_elapsed:.4f} s, separate calls: {sep_elapsed:.4f} s{two_note})",
          file=sys.stderr, flush=True)
    if L.topk_wait_status(ws) != 0 or L.topk_wait_status(ws2) != 0 or any(
            L.topk_wait_status(gr.topk_workspace) != 0 for gr in graphs):
        raise RuntimeError("a bounded wait of the logits pass gave up: outputs invalid")
    for gr in graphs:
        gr.close()

    ms_per_step = elapsed / args.steps * 1e3
    value = N * args.steps / elapsed
    logits_bytes = N * B * V * 2
    algo_bytes = logits_bytes + N * B * K * 8
    achieved = algo_bytes / topk_s / 1e9
    traffic = traffic_per_launch()

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "blocks/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "headline: N=64 requests, B=16 slots, K=16, V=151936, d=256, "
                               "bf16 logits (3 entropy tiers, 1% exact ties), bf16 embeddings, "
                               "fp32 weights; no anchor; sigma=8",
                   "path": "lilicorr_topk -> lilicorr_score_walk (C ABI, two calls per block)",
                   "N": N, "B": B, "K": K, "V": V, "d": d, "logits_dtype": "bf16",
                   "logits_rotation": ROTATE},
        "roofline": {"bound": "hbm", "kernel": "topk_lse_kernel", "achieved": achieved,
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS,
                     "traffic": traffic, "avg_launch_us": topk_s * 1e6,
                     "algorithmic_bytes_per_launch": algo_bytes,
                     "timing": f"{reps} back-to-back launches over the rotating buffers between "
                               "two HIP events on the launch stream"},
        "graph_replay": {"path": "the same block as one HIP graph per logits buffer, one "
                                 "lilicorr_block_graph_launch per block",
                         "ms_per_step": graph_elapsed / args.steps * 1e3,
                         "value": N * args.steps / graph_elapsed},
        "two_streams": None if two_elapsed is None else {
            "path": "the timed step's two C-ABI calls, consecutive blocks alternating between "
                    "two streams with their own buffers",
            "ms_per_step": two_elapsed / args.steps * 1e3,
            "value": N * args.steps / two_elapsed},
        "separate_calls": {"path": "topk -> candidate_vectors -> pair_scores -> greedy_walk",
                           "ms_per_step": sep_elapsed / args.steps * 1e3,
                           "value": N * args.steps / sep_elapsed},
    }

    # the two decode rules of the decode-rule appendix, each in the fused pass and stand-alone,
    # on the candidates of the last timed step
    ws_exact = L.score_viterbi_workspace(N, B, K)
    score = torch.empty(N, dtype=torch.float32, device=dev)
    L.pair_scores(*L.candidate_vectors(ids, E, packed, out=(in_vec, out_vec)), None, L.SIGMA,
                  out=(S, None))
    fused_greedy = median_launch_us(torch, lambda: L.score_walk(
        ids, logp, E, packed, out=(draft, choice, logq), workspace=ws_fused))
    fused_exact = median_launch_us(torch, lambda: L.score_viterbi(
        ids, logp, E, packed, out=(draft, choice, logq, score), workspace=ws_exact))
    ws_cert = L.score_walk_certified_workspace(N, B, K)
    resc = torch.empty(N, B, dtype=torch.int32, device=dev)
    fused_cert = median_launch_us(torch, lambda: L.score_walk_certified(
        ids, logp, E, packed, out=(draft, choice, logq, resc), workspace=ws_cert))
    out["decode_rules"] = {
        "fused_greedy_us": fused_greedy,
        "fused_certified_us": fused_cert,
        "certified_rescored": int((resc > 0).sum()),
        "certified_changed": int((resc == 2).sum()),
        "fused_exact_us": fused_exact,
        "greedy_walk_us": median_launch_us(torch, lambda: L.greedy_walk(
            S, None, logp, ids, 0.0, out=(draft, choice, logq))),
        "viterbi_walk_us": median_launch_us(torch, lambda: L.viterbi_walk(
            S, None, logp, ids, 0.0, out=(draft, choice, logq, score))),
        "step_us_greedy": topk_s * 1e6 + fused_greedy,
        "step_us_certified": topk_s * 1e6 + fused_cert,
        "step_us_exact": topk_s * 1e6 + fused_exact,
        "note": "median call durations (HIP events, host launch included); steps add the mean "
                "logits-pass launch",
    }

    if not args.no_stress:
        c4 = workloads.config(4)
        t = time.perf_counter()
        lg4 = workloads.make_logits(c4).cuda()
        print(f"[bench] stress logits generated in {time.perf_counter() - t:.1f} s", file=sys.stderr,
              flush=True)
        t3, lo3, hi3 = time_logits_pass(L, torch, cfg, logits_list, iters=100)
        feat = torch.empty(N, B, K, 5, dtype=torch.float32, device=dev)
        feat_us = median_launch_us(torch, lambda: L.topk(
            logits_list[0], K, out=(ids, logp, feat), workspace=ws, features=True))
        plain_us = median_launch_us(torch, lambda: L.topk(logits_list[0], K, out=(ids, logp),
                                                          workspace=ws))
        read3 = stream_read_rate(torch, logits_list, iters=100)
        logits_list = None
        torch.cuda.empty_cache()
        t4, lo4, hi4 = time_logits_pass(L, torch, c4, [lg4], iters=20)
        read4 = stream_read_rate(torch, [lg4])
        b4 = c4.N * c4.B * c4.V * 2 + c4.N * c4.B * c4.K * 8
        out["logits_pass"] = {
            "method": "per-launch mean over batches of back-to-back launches (100 at the "
                      "headline over 4 rotating buffers, 20 at the stress shape), 5 batches "
                      "after three untimed batches; HIP events on the launch stream",
            "headline": {"GB_s": algo_bytes / t3 / 1e9, "us": t3 * 1e6,
                         "us_batch_min": lo3 * 1e6, "us_batch_max": hi3 * 1e6,
                         "frac_of_8TBs": algo_bytes / t3 / 1e9 / PEAK_HBM_GBS,
                         "stream_read_GB_s": read3,
                         "frac_of_stream_read": algo_bytes / t3 / 1e9 / read3,
                         "with_features_us_median": feat_us, "same_buffer_us_median": plain_us},
            "stress": {"GB_s": b4 / t4 / 1e9, "us": t4 * 1e6,
                       "us_batch_min": lo4 * 1e6, "us_batch_max": hi4 * 1e6,
                       "frac_of_8TBs": b4 / t4 / 1e9 / PEAK_HBM_GBS,
                       "stream_read_GB_s": read4,
                       "frac_of_stream_read": b4 / t4 / 1e9 / read4,
                       "workload": "N=256, B=16, K=32, V=262144, bf16 logits"},
        }
        del lg4

    if not args.no_configs:
        # both metrics at every workload (the headline's figures here come from the cold-step
        # protocol of per_config_rates, not from the timed loop above)
        logits_list = None
        torch.cuda.empty_cache()
        per = {}
        for ci in range(len(workloads.CONFIGS)):
            c = workloads.config(ci)
            pinp = inp if ci == cfg.index else workloads.make_inputs(c)
            per[c.name] = per_config_rates(L, torch, c, pinp)
            del pinp
            torch.cuda.empty_cache()
            print(f"[bench] workload {c.name} done", file=sys.stderr, flush=True)
        out["per_workload"] = per

    if not args.no_scorer:
        out["scorer"] = scorer_rate(L, torch, workloads)

    if args.calibrate_copy:
        calibration_copies(torch)

    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(cfg, inp, args.cpu_seconds)
        out["cpu_baseline"]["cpu_model"] = cpu_model()
        out["cpu_baseline_all_cores"] = cpu_baseline_threads(cfg, inp, args.cpu_seconds)

    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
