"""Host-side checks of the C ABI (no GPU): the library loads, exports every symbol that
include/lilicorr.h declares, and rejects bad arguments before launching anything."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lilicorr.h")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(lilicorr_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    import paper_2608_20530_amd as L

    L.load_library()
    return L


def test_header_declares_the_path(L):
    names = _declared()
    for n in ["lilicorr_topk", "lilicorr_topk_features", "lilicorr_topk_workspace_bytes", "lilicorr_pack_weights",
              "lilicorr_packed_weight_bytes", "lilicorr_candidate_vectors", "lilicorr_pair_scores",
              "lilicorr_greedy_walk", "lilicorr_viterbi_walk", "lilicorr_score_walk",
              "lilicorr_score_viterbi", "lilicorr_score_viterbi_workspace_bytes", "lilicorr_score_walk_workspace_bytes",
              "lilicorr_score_walk_certified", "lilicorr_score_walk_certified_workspace_bytes",
              "lilicorr_block_graph_create", "lilicorr_block_graph_launch",
              "lilicorr_block_graph_destroy", "lilicorr_status_string",
              "lilicorr_topk_wait_status", "lilicorr_set_wait_limit", "lilicorr_pair_walk",
              "lilicorr_pair_walk_certified", "lilicorr_pair_viterbi"]:
        assert n in names


def test_every_declared_symbol_is_exported(L):
    lib = ctypes.CDLL(L.LIB_PATH)
    for n in _declared():
        assert hasattr(lib, n), n


def test_status_strings(L):
    assert L.lilicorr_status_string(0) == "ok"
    for code in (-1, -2, -3, -4, -5, -6):
        assert L.lilicorr_status_string(code) not in ("ok", "unknown status")
    assert L.lilicorr_status_string(-99) == "unknown status"


def test_size_queries(L):
    assert L.lilicorr_packed_weight_bytes(256) == 2 * 3 * 256 * 256 * 2 + 2 * 256 * 256 * 4
    # fragments padded to an even number of 32-deep k-blocks and whole groups of four
    # 16-column blocks: d = 48 -> 64 x 64 per term
    assert L.lilicorr_packed_weight_bytes(48) == 2 * 3 * 64 * 64 * 2 + 2 * 48 * 48 * 4
    assert L.lilicorr_packed_weight_bytes(80) == 2 * 3 * 128 * 128 * 2 + 2 * 80 * 80 * 4
    assert L.lilicorr_packed_weight_bytes(8) == 0
    assert L.lilicorr_packed_weight_bytes(2048) == 0
    # headline shapes run one workgroup per row: the workspace is the 256-byte status header
    H = 256
    assert L.lilicorr_topk_workspace_bytes(64, 16, 151936, 16) == H
    assert L.lilicorr_topk_workspace_bytes(256, 16, 262144, 32) == H
    # a single request is split over several workgroups per row
    assert L.lilicorr_topk_workspace_bytes(1, 16, 151936, 8) > H
    assert L.lilicorr_topk_workspace_bytes(1, 16, 151936, 65) == 0
    # the split rule, through the workspace size (header, then rows x segments x (16-byte
    # partial header + K keys)): few rows whose short segments (<= 8192 logits) all run at once
    # take ceil(V / 8192) of them
    part = lambda K: 16 + 8 * K
    assert L.lilicorr_topk_workspace_bytes(1, 16, 151936, 8) == H + 16 * 19 * part(8)
    assert L.lilicorr_topk_workspace_bytes(1, 8, 32000, 4) == H + 8 * 4 * part(4)
    assert L.lilicorr_topk_workspace_bytes(1, 1, 300000, 64) == H + 37 * part(64)
    # more rows x segments than run at once: streaming segments of >= 12288 logits
    assert L.lilicorr_topk_workspace_bytes(2, 16, 151936, 16) == H + 32 * 12 * part(16)
    assert L.lilicorr_topk_workspace_bytes(16, 16, 151936, 16) == H + 256 * 4 * part(16)
    # rows shorter than one short segment stay whole
    assert L.lilicorr_topk_workspace_bytes(1, 2, 5000, 8) == H


A = 4096  # a fake, 16-byte aligned "device" address: never dereferenced on these paths


def test_topk_argument_errors(L):
    lib = L.load_library()
    ok = (A, 1, 2, 3, 1000, 8, A, A, A, 256, None)
    def call(i, v):
        args = list(ok)
        args[i] = v
        return lib.lilicorr_topk(*args)
    assert call(0, None) == -1          # logits
    assert call(6, None) == -1          # ids
    assert call(7, None) == -1          # logp
    assert call(1, 7) == -1             # dtype
    assert call(2, 0) == -1             # N
    assert call(3, 0) == -1             # B
    assert call(4, 0) == -1             # V
    assert call(5, 0) == -1             # K
    assert call(5, 65) == -2            # K > 64
    assert call(5, 1001) == -2          # K > V
    assert call(0, A + 2) == -3         # alignment
    # every call needs the workspace's status header; split rows need room for partials too
    assert call(9, 255) == -4           # workspace_bytes below the 256-byte header
    assert call(8, A + 4) == -3         # workspace alignment (with enough bytes)
    args = list(ok)
    args[2], args[3], args[4] = 1, 1, 151936
    assert lib.lilicorr_topk(*args) == -4
    args[9] = 256
    assert lib.lilicorr_topk(*args) == -4


def test_wait_status_argument_errors(L):
    lib = L.load_library()
    assert lib.lilicorr_topk_wait_status(None, None) == -1
    assert lib.lilicorr_topk_wait_status(A + 4, None) == -3


def test_topk_features_argument_errors(L):
    lib = L.load_library()
    ok = [A, 1, 2, 3, 1000, 8, A, A, A, None, 0, None]
    def call(i, v):
        args = list(ok)
        args[i] = v
        return lib.lilicorr_topk_features(*args)
    assert call(8, None) == -1          # feat is required
    assert call(6, None) == -1          # ids
    assert call(5, 65) == -2            # K > 64
    assert call(8, A + 4) == -3         # feat alignment


def test_other_argument_errors(L):
    lib = L.load_library()
    assert lib.lilicorr_pack_weights(None, A, 64, A, None) == -1
    assert lib.lilicorr_pack_weights(A, A, 40, A, None) == -2
    assert lib.lilicorr_pack_weights(A, A + 4, 64, A, None) == -3
    cv = [A, A, 1, 1000, 64, A, 2, 3, 4, A, A, None]
    assert lib.lilicorr_candidate_vectors(*cv[:2], 5, *cv[3:]) == -1
    bad = list(cv); bad[4] = 2048
    assert lib.lilicorr_candidate_vectors(*bad) == -2
    bad = list(cv); bad[9] = A + 8
    assert lib.lilicorr_candidate_vectors(*bad) == -3
    ps = [A, A, None, 2, 3, 4, 64, 8.0, A, None, None]
    bad = list(ps); bad[8] = None
    assert lib.lilicorr_pair_scores(*bad) == -1   # S required when B > 1
    bad = list(ps); bad[2] = A
    assert lib.lilicorr_pair_scores(*bad) == -1   # S0 required with an anchor
    bad = list(ps); bad[7] = float("nan")
    assert lib.lilicorr_pair_scores(*bad) == -1
    bad = list(ps); bad[6] = 24
    assert lib.lilicorr_pair_scores(*bad) == -2
    gw = [A, None, A, A, 2, 3, 4, 0.0, A, None, None, None]
    bad = list(gw); bad[0] = None
    assert lib.lilicorr_greedy_walk(*bad) == -1   # S required when B > 1
    bad = list(gw); bad[6] = 65
    assert lib.lilicorr_greedy_walk(*bad) == -2
    bad = list(gw); bad[8] = A + 4
    assert lib.lilicorr_greedy_walk(*bad) == -3


def test_viterbi_argument_errors(L):
    lib = L.load_library()
    vw = [A, None, A, A, 2, 3, 4, 0.0, A, None, None, None, None]
    bad = list(vw); bad[0] = None
    assert lib.lilicorr_viterbi_walk(*bad) == -1      # S required when B > 1
    bad = list(vw); bad[8] = None
    assert lib.lilicorr_viterbi_walk(*bad) == -1      # draft
    bad = list(vw); bad[7] = float("nan")
    assert lib.lilicorr_viterbi_walk(*bad) == -1
    bad = list(vw); bad[6] = 65
    assert lib.lilicorr_viterbi_walk(*bad) == -2      # K > 64
    bad = list(vw); bad[5] = 8193
    assert lib.lilicorr_viterbi_walk(*bad) == -2      # B > 8192
    bad = list(vw); bad[5], bad[6] = 2000, 64
    assert lib.lilicorr_viterbi_walk(*bad) == -2      # B * K > 65536
    bad = list(vw); bad[11] = A + 4
    assert lib.lilicorr_viterbi_walk(*bad) == -3      # score alignment


def test_score_walk_sizes_and_argument_errors(L):
    lib = L.load_library()
    # 256-byte block of per-request counters, then N x (1 + (B-1) K) 8-byte table rows
    assert L.lilicorr_score_walk_workspace_bytes(64, 16, 16) == 256 + 64 * 241 * 8
    assert L.lilicorr_score_walk_workspace_bytes(2, 3, 4) == 256 + 2 * 9 * 8
    assert L.lilicorr_score_walk_workspace_bytes(65, 1, 1) == 512 + 65 * 8
    assert L.lilicorr_score_walk_workspace_bytes(1, 2, 65) == 0
    assert L.lilicorr_score_walk_workspace_bytes(1, 20000, 1) == 0
    ws = L.lilicorr_score_walk_workspace_bytes(2, 3, 4)
    ok = [A, A, A, 1, 1000, 64, A, None, 2, 3, 4, 8.0, 0.0, None, None, A, None, None, A, ws, None]
    def call(**kw):
        names = ["ids", "logp", "E", "e_dtype", "V", "d", "packed", "anchor", "N", "B", "K",
                 "sigma", "lw", "S", "S0", "draft", "choice", "logq", "ws", "ws_bytes", "stream"]
        args = list(ok)
        for k, v in kw.items():
            args[names.index(k)] = v
        return lib.lilicorr_score_walk(*args)
    assert call(ids=None) == -1
    assert call(draft=None) == -1
    assert call(ws=None) == -1
    assert call(e_dtype=7) == -1
    assert call(sigma=float("nan")) == -1
    assert call(lw=float("inf")) == -1
    assert call(e_dtype=0) == -2        # fp32 embeddings: use the separate calls
    assert call(d=512) == -2            # above the fused path's d
    assert call(d=40) == -2
    assert call(K=65) == -2
    assert call(B=20000, K=1) == -2     # the request's table would not fit in LDS
    assert call(draft=A + 4) == -3
    assert call(anchor=A + 8) == -3
    assert call(ws_bytes=ws - 1) == -4


def test_score_walk_certified_sizes_and_argument_errors(L):
    lib = L.load_library()
    # counters, the table rows, then one 8-byte contender mask per table row
    assert L.lilicorr_score_walk_certified_workspace_bytes(64, 16, 16) == 256 + 64 * 241 * 16
    assert L.lilicorr_score_walk_certified_workspace_bytes(2, 3, 4) == 256 + 2 * 9 * 16
    assert L.lilicorr_score_walk_certified_workspace_bytes(1, 2, 65) == 0
    ws = L.lilicorr_score_walk_certified_workspace_bytes(2, 3, 4)
    names = ["ids", "logp", "E", "e_dtype", "V", "d", "packed", "anchor", "N", "B", "K", "sigma",
             "lw", "margin", "S", "S0", "draft", "choice", "logq", "rescored", "ws", "ws_bytes",
             "stream"]
    ok = [A, A, A, 1, 1000, 64, A, None, 2, 3, 4, 8.0, 0.0, 2.0 ** -14, None, None, A, None, None,
          None, A, ws, None]
    def call(**kw):
        args = list(ok)
        for k, v in kw.items():
            args[names.index(k)] = v
        return lib.lilicorr_score_walk_certified(*args)
    assert call(ids=None) == -1
    assert call(ws=None) == -1
    assert call(margin=-1.0) == -1
    assert call(margin=float("nan")) == -1
    assert call(margin=float("inf")) == -1
    assert call(e_dtype=0) == -2
    assert call(d=512) == -2
    assert call(rescored=A + 4) == -3
    assert call(ws_bytes=ws - 1) == -4
    # the plain pass's workspace is too small for the contender masks
    assert call(ws_bytes=L.lilicorr_score_walk_workspace_bytes(2, 3, 4)) == -4


def test_block_args_layout_matches_the_header(L, tmp_path):
    """The binding's BlockArgs has the C struct's size and field offsets (compiled with gcc)."""
    import ctypes
    import subprocess

    fields = [f for f, _ in L.BlockArgs._fields_]
    src = tmp_path / "layout.c"
    src.write_text("#include <stdio.h>\n#include <stddef.h>\n#include \"lilicorr.h\"\n"
                   "int main(void) {\n"
                   "  printf(\"%zu\\n\", sizeof(lilicorr_block_args));\n" +
                   "".join(f"  printf(\"%zu\\n\", offsetof(lilicorr_block_args, {f}));\n"
                           for f in fields) + "  return 0;\n}\n")
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-std=c11", "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include",
                           "-I", os.path.join(ROOT, "include"), "-o", str(exe), str(src)])
    got = [int(x) for x in subprocess.check_output([str(exe)]).split()]
    assert got[0] == ctypes.sizeof(L.BlockArgs)
    assert got[1:] == [getattr(L.BlockArgs, f).offset for f in fields]


def test_block_graph_argument_errors(L):
    import ctypes
    lib = L.load_library()
    handle = ctypes.c_void_p(123)
    assert lib.lilicorr_block_graph_create(None, ctypes.byref(handle)) == -1
    a = L.BlockArgs()
    assert lib.lilicorr_block_graph_create(ctypes.byref(a), None) == -1
    a.decode = 7
    assert lib.lilicorr_block_graph_create(ctypes.byref(a), ctypes.byref(handle)) == -1
    assert handle.value is None                 # set to NULL on every error
    assert lib.lilicorr_block_graph_launch(None, None) == -1
    lib.lilicorr_block_graph_destroy(None)      # ignored


def test_score_viterbi_sizes_and_argument_errors(L):
    lib = L.load_library()
    # counters, then N x ((B-1) K K + K) fp32 scores exchanged between workgroups
    assert L.lilicorr_score_viterbi_workspace_bytes(64, 16, 16) == 256 + 64 * (15 * 256 + 16) * 4
    assert L.lilicorr_score_viterbi_workspace_bytes(1, 8193, 1) == 0
    assert L.lilicorr_score_viterbi_workspace_bytes(1, 2000, 64) == 0
    ws = L.lilicorr_score_viterbi_workspace_bytes(2, 3, 4)
    ok = [A, A, A, 1, 1000, 64, A, None, 2, 3, 4, 8.0, 0.0, None, None, A, None, None, None, A, ws,
          None]
    def call(i, v):
        args = list(ok)
        args[i] = v
        return lib.lilicorr_score_viterbi(*args)
    assert call(0, None) == -1        # ids
    assert call(19, None) == -1       # workspace
    assert call(3, 0) == -2           # fp32 embeddings
    assert call(5, 512) == -2         # d above the fused pass
    assert call(18, A + 4) == -3      # score alignment
    assert call(20, ws - 1) == -4


def test_pair_walk_argument_errors(L):
    """The one-pass decode over precomputed vectors: any width the vector call supports (d <= 1024;
    certified d <= 512 with bf16 rows), the fused calls' workspaces."""
    lib = L.load_library()
    ws = L.lilicorr_score_walk_workspace_bytes(2, 3, 4)
    names = ["in", "out", "anchor", "logp", "ids", "N", "B", "K", "d", "sigma", "lw", "S", "S0",
             "draft", "choice", "logq", "ws", "ws_bytes", "stream"]
    ok = [A, A, None, A, A, 2, 3, 4, 512, 8.0, 0.0, None, None, A, None, None, A, ws, None]

    def call(**kw):
        args = list(ok)
        for k, v in kw.items():
            args[names.index(k)] = v
        return lib.lilicorr_pair_walk(*args)
    assert call(**{"in": None}) == -1
    assert call(out=None) == -1
    assert call(ids=None) == -1
    assert call(draft=None) == -1
    assert call(ws=None) == -1
    assert call(N=0) == -1
    assert call(sigma=float("nan")) == -1
    assert call(d=40) == -2
    assert call(d=1040) == -2
    assert call(K=65) == -2
    assert call(B=20000, K=1) == -2
    assert call(N=65536) == -2
    assert call(out=A + 4) == -3
    assert call(logq=A + 8) == -3
    assert call(ws_bytes=ws - 1) == -4

    wsc = L.lilicorr_score_walk_certified_workspace_bytes(2, 3, 4)
    cnames = ["in", "out", "anchor", "logp", "ids", "E", "e_dtype", "V", "packed", "N", "B", "K",
              "d", "sigma", "lw", "margin", "S", "S0", "draft", "choice", "logq", "rescored", "ws",
              "ws_bytes", "stream"]
    cok = [A, A, None, A, A, A, 1, 1000, A, 2, 3, 4, 512, 8.0, 0.0, 2.0 ** -14, None, None, A,
           None, None, None, A, wsc, None]

    def ccall(**kw):
        args = list(cok)
        for k, v in kw.items():
            args[cnames.index(k)] = v
        return lib.lilicorr_pair_walk_certified(*args)
    assert ccall(E=None) == -1
    assert ccall(packed=None) == -1
    assert ccall(V=0) == -1
    assert ccall(e_dtype=7) == -1
    assert ccall(margin=-1.0) == -1
    assert ccall(e_dtype=0) == -2       # the re-scoring reads bf16 rows
    assert ccall(d=528) == -2           # one vector per 512 threads at most
    assert ccall(packed=A + 4) == -3
    assert ccall(rescored=A + 4) == -3
    assert ccall(ws_bytes=ws) == -4     # the plain pass's workspace lacks the contender masks

    wse = L.lilicorr_score_viterbi_workspace_bytes(2, 3, 4)
    enames = ["in", "out", "anchor", "logp", "ids", "N", "B", "K", "d", "sigma", "lw", "S", "S0",
              "draft", "choice", "logq", "score", "ws", "ws_bytes", "stream"]
    eok = [A, A, None, A, A, 2, 3, 4, 1024, 8.0, 0.0, None, None, A, None, None, None, A, wse, None]

    def ecall(**kw):
        args = list(eok)
        for k, v in kw.items():
            args[enames.index(k)] = v
        return lib.lilicorr_pair_viterbi(*args)
    assert ecall(logp=None) == -1
    assert ecall(B=8193, K=1) == -2
    assert ecall(B=2000, K=64) == -2
    assert ecall(score=A + 4) == -3
    assert ecall(ws_bytes=wse - 1) == -4


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    import paper_2608_20530_amd as L

    monkeypatch.setattr(L, "_lib", None)
    monkeypatch.setattr(L, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(L.LilicorrError):
        L.load_library()


def test_scorer_size_queries_and_rejections(L):
    H, F, heads, S = 1024, 2048, 8, 15
    packed = L.lilicorr_scorer_packed_bytes(H, heads, F, S)
    # transposed weights (3H^2 + H^2 + 2 H F bf16) + gains + biases, each section 256-byte aligned
    assert packed >= 2 * (4 * H * H + 2 * H * F) + 8 * H + 4 * heads * 2 * S
    assert packed % 256 == 0
    assert L.lilicorr_scorer_packed_bytes(320, 2, F, S) == 0      # H not a multiple of 256
    assert L.lilicorr_scorer_packed_bytes(H, 4, F, S) == 0        # heads * 128 != H
    assert L.lilicorr_scorer_packed_bytes(H, heads, 200, S) == 0  # F not a multiple of 128
    assert L.lilicorr_scorer_packed_bytes(H, heads, F, 0) == 0
    ws = L.lilicorr_scorer_workspace_bytes(64, 15, 16, H, F)
    M = 64 * 240
    assert ws >= 2 * (M * H + M * 2 * H + 64 * H * 240 + M * H + M * F)
    assert L.lilicorr_scorer_workspace_bytes(1, 17, 16, H, F) == 0   # L = 272 > 256
    assert L.lilicorr_scorer_workspace_bytes(0, 15, 16, H, F) == 0
    # null pointers are rejected before anything is launched
    assert L.load_library().lilicorr_scorer_forward(None, 1, 15, 16, H, heads, F, 2, None, None, 0,
                                                    None) == -1
    assert L.load_library().lilicorr_scorer_pack(ctypes.byref(L.ScorerLayer()), H, heads, F, S,
                                                 None, None) == -1
