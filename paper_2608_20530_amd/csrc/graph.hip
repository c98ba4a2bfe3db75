// One draft block as one captured HIP graph: the logits pass followed by the fused matching and
// decode pass (or, where that pass does not apply, the candidate vectors followed by the one-pass
// decode over them), recorded once through the library's own entry points and replayed with a
// single launch. The paper serves candidate extraction, matching and selection as one graph replay per
// block (implementation appendix, serving); this is that replay on HIP graphs. Host code only.
#include <hip/hip_runtime.h>
#include <new>

#include "lilicorr.h"

struct lilicorr_graph {
  hipGraph_t graph;
  hipGraphExec_t exec;
};

namespace {

lilicorr_status record_block(const lilicorr_block_args* a, hipStream_t s) {
  lilicorr_status st = lilicorr_topk(a->logits, a->logits_dtype, a->N, a->B, a->V, a->K, a->ids,
                                     a->logp, a->topk_workspace, a->topk_workspace_bytes, s);
  if (st != LILICORR_OK) return st;
  // the fused pass takes bf16 tables up to d = 256 (its own checks reject the rest)
  if (a->e_dtype != LILICORR_BF16 || a->d > 256) {
    if (!a->in_vec || !a->out_vec) return LILICORR_ERR_INVALID_ARG;
    st = lilicorr_candidate_vectors(a->ids, a->E, a->e_dtype, a->e_rows, a->d, a->packed_w, a->N,
                                    a->B, a->K, a->in_vec, a->out_vec, s);
    if (st != LILICORR_OK) return st;
    switch (a->decode) {
      case LILICORR_DECODE_GREEDY:
        return lilicorr_pair_walk(a->in_vec, a->out_vec, a->anchor_out, a->logp, a->ids, a->N,
                                  a->B, a->K, a->d, a->sigma, a->logp_weight, a->S, a->S0,
                                  a->draft, a->choice, a->logq, a->fused_workspace,
                                  a->fused_workspace_bytes, s);
      case LILICORR_DECODE_CERTIFIED:
        return lilicorr_pair_walk_certified(
            a->in_vec, a->out_vec, a->anchor_out, a->logp, a->ids, a->E, a->e_dtype, a->e_rows,
            a->packed_w, a->N, a->B, a->K, a->d, a->sigma, a->logp_weight, a->margin, a->S,
            a->S0, a->draft, a->choice, a->logq, a->rescored, a->fused_workspace,
            a->fused_workspace_bytes, s);
      case LILICORR_DECODE_EXACT:
        return lilicorr_pair_viterbi(a->in_vec, a->out_vec, a->anchor_out, a->logp, a->ids, a->N,
                                     a->B, a->K, a->d, a->sigma, a->logp_weight, a->S, a->S0,
                                     a->draft, a->choice, a->logq, a->score, a->fused_workspace,
                                     a->fused_workspace_bytes, s);
    }
    return LILICORR_ERR_INVALID_ARG;
  }
  switch (a->decode) {
    case LILICORR_DECODE_GREEDY:
      return lilicorr_score_walk(a->ids, a->logp, a->E, a->e_dtype, a->e_rows, a->d, a->packed_w,
                                 a->anchor_out, a->N, a->B, a->K, a->sigma, a->logp_weight, a->S,
                                 a->S0, a->draft, a->choice, a->logq, a->fused_workspace,
                                 a->fused_workspace_bytes, s);
    case LILICORR_DECODE_CERTIFIED:
      return lilicorr_score_walk_certified(
          a->ids, a->logp, a->E, a->e_dtype, a->e_rows, a->d, a->packed_w, a->anchor_out, a->N,
          a->B, a->K, a->sigma, a->logp_weight, a->margin, a->S, a->S0, a->draft, a->choice,
          a->logq, a->rescored, a->fused_workspace, a->fused_workspace_bytes, s);
    case LILICORR_DECODE_EXACT:
      return lilicorr_score_viterbi(a->ids, a->logp, a->E, a->e_dtype, a->e_rows, a->d,
                                    a->packed_w, a->anchor_out, a->N, a->B, a->K, a->sigma,
                                    a->logp_weight, a->S, a->S0, a->draft, a->choice, a->logq,
                                    a->score, a->fused_workspace, a->fused_workspace_bytes, s);
  }
  return LILICORR_ERR_INVALID_ARG;
}

}  // namespace

extern "C" lilicorr_status lilicorr_block_graph_create(const lilicorr_block_args* args,
                                                       lilicorr_graph** out) {
  if (!args || !out) return LILICORR_ERR_INVALID_ARG;
  *out = nullptr;
  if (args->decode != LILICORR_DECODE_GREEDY && args->decode != LILICORR_DECODE_CERTIFIED &&
      args->decode != LILICORR_DECODE_EXACT)
    return LILICORR_ERR_INVALID_ARG;
  // capture on a stream of our own (default priority): the null stream cannot be captured, and
  // recording executes nothing
  hipStream_t s;
  if (hipStreamCreateWithFlags(&s, hipStreamNonBlocking) != hipSuccess) return LILICORR_ERR_HIP;
  lilicorr_status st = LILICORR_OK;
  hipGraph_t graph = nullptr;
  if (hipStreamBeginCapture(s, hipStreamCaptureModeRelaxed) != hipSuccess) {
    st = LILICORR_ERR_HIP;
  } else {
    st = record_block(args, s);
    const hipError_t end = hipStreamEndCapture(s, &graph);
    if (st == LILICORR_OK && (end != hipSuccess || graph == nullptr)) st = LILICORR_ERR_HIP;
  }
  hipGraphExec_t exec = nullptr;
  if (st == LILICORR_OK && hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0) != hipSuccess)
    st = LILICORR_ERR_HIP;
  lilicorr_graph* g = nullptr;
  if (st == LILICORR_OK) {
    g = new (std::nothrow) lilicorr_graph{graph, exec};
    if (!g) st = LILICORR_ERR_HIP;
  }
  if (st != LILICORR_OK) {
    if (exec) (void)hipGraphExecDestroy(exec);
    if (graph) (void)hipGraphDestroy(graph);
  }
  (void)hipStreamDestroy(s);
  (void)hipGetLastError();  // a failed capture leaves its error behind; the status reports it
  *out = g;
  return st;
}

extern "C" lilicorr_status lilicorr_block_graph_launch(lilicorr_graph* graph, hipStream_t stream) {
  if (!graph) return LILICORR_ERR_INVALID_ARG;
  return hipGraphLaunch(graph->exec, stream) == hipSuccess ? LILICORR_OK : LILICORR_ERR_HIP;
}

extern "C" void lilicorr_block_graph_destroy(lilicorr_graph* graph) {
  if (!graph) return;
  (void)hipGraphExecDestroy(graph->exec);
  (void)hipGraphDestroy(graph->graph);
  delete graph;
}
