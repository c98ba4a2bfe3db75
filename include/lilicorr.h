/*
 * lilicorr.h — C ABI of the LiLiCorr draft-correlation hot path on MI355X (gfx950).
 *
 * LiLiCorr (Lightweight Likelihood Correlation of Parallel Drafts) turns the per-slot vocabulary
 * logits of a parallel block drafter into one coherent draft: it keeps the top-K candidates of
 * every slot (Sec. 3.2), gives each candidate a unit-norm "in" and "out" vector (Sec. 3.2 and the
 * implementation appendix), scores every adjacent pair with sigma * cos(out, in) (Eq. pair) and
 * commits the block left to right with a greedy argmax walk (Sec. 3.5), whose local softmax is
 * Eq. (localar).
 *
 * Conventions shared by every call
 *  - Tensors are caller-owned, device-resident (HBM), contiguous, row-major with the innermost
 *    dimension last, and 16-byte aligned. bf16 tensors hold raw bfloat16 bit patterns.
 *  - N requests, B slots per request (every slot carries logits and candidates; the optional
 *    anchor of the paper, its slot 0, enters only through anchor_out / S0), K candidates per
 *    slot, V vocabulary size, d width of the in/out vectors.
 *  - Every call is asynchronous on `stream` (0 = the null stream) and allocates no memory;
 *    the library keeps no state between calls, so concurrent calls on different streams are safe
 *    when their outputs do not overlap. (The graph objects of lilicorr_block_graph_create are
 *    the one exception: the caller creates and destroys them.)
 *  - Arguments are validated on the host before anything is launched: a negative status means
 *    nothing was launched and no output was written. LILICORR_ERR_HIP reports a failed launch.
 *  - Preconditions the library does not check (reading device data would cost a sync): logits
 *    finite or -inf with at least one finite value per slot; ids inside [0, V). Breaking them
 *    gives unspecified (but memory-safe) results.
 *  - Limits: 1 <= K <= min(V, 64); B >= 1; N >= 1; d a multiple of 16 with 16 <= d <= 1024;
 *    N*B*V < 2^62; V < 2^31.
 */
#ifndef LILICORR_H_
#define LILICORR_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    LILICORR_F32 = 0,  /* IEEE binary32 */
    LILICORR_BF16 = 1, /* bfloat16 bit patterns (uint16) */
} lilicorr_dtype;

typedef enum {
    LILICORR_OK = 0,
    LILICORR_ERR_INVALID_ARG = -1, /* null pointer, size out of range, bad dtype */
    LILICORR_ERR_UNSUPPORTED = -2, /* a limit above is exceeded */
    LILICORR_ERR_ALIGNMENT = -3,   /* a pointer is not 16-byte aligned */
    LILICORR_ERR_WORKSPACE = -4,   /* workspace missing or smaller than required */
    LILICORR_ERR_HIP = -5,         /* a kernel launch failed */
    LILICORR_ERR_TIMEOUT = -6,     /* a bounded wait inside a kernel gave up (see
                                      lilicorr_topk_wait_status): outputs are invalid */
} lilicorr_status;

/*
 * Step 1 — vocabulary-wide log-normalisation fused with top-K candidate selection.
 * Sec. 3.2 keeps the drafter's K most probable tokens of every slot as candidates; the paper's
 * serving path extracts them in the same kernel that normalises the logits over the vocabulary
 * (implementation appendix, "Serving").
 *
 *   logits    [N][B][V] in `dtype` (LILICORR_F32 or LILICORR_BF16), read once.
 *   ids       [N][B][K] int32 out: token ids ordered by logit descending, ties to the lower id
 *             (-0 and +0 compare equal).
 *   logp      [N][B][K] fp32 out: logits[id] - log(sum_v exp(logits[v])). The same inputs give
 *             the same ids and logp bit for bit on every call.
 *   workspace device scratch of at least lilicorr_topk_workspace_bytes(N, B, V, K) bytes (at
 *             least 256), owned by the caller and zero-filled once before its first use. Its
 *             first 256 bytes hold the wait status word (below), which the calls only ever set;
 *             the rest is clobbered by every call. Calls sharing a workspace must not overlap.
 *
 * The kernel's waits (a producer wave for ring space, the consumer wave for work) are bounded.
 * A wait that gives up (never expected: the bound is ~4M polls) does not stop the kernel: the
 * call completes, its outputs are invalid, and a bit is set in the workspace's status word.
 */
size_t lilicorr_topk_workspace_bytes(int64_t N, int64_t B, int64_t V, int K);
lilicorr_status lilicorr_topk(const void *logits, lilicorr_dtype dtype, int64_t N, int64_t B,
                              int64_t V, int K, int32_t *ids, float *logp, void *workspace,
                              size_t workspace_bytes, hipStream_t stream);

/*
 * Wait status of the top-K calls that used `workspace` since its status word was last cleared:
 * waits for `stream` to finish what it holds, reads the word, clears it, and returns
 * LILICORR_ERR_TIMEOUT if some wait gave up (the outputs of at least one of those calls are
 * invalid), LILICORR_OK otherwise. Synchronous; not for use inside graph capture.
 * LILICORR_ERR_INVALID_ARG for a NULL workspace, LILICORR_ERR_HIP if a HIP call fails.
 */
lilicorr_status lilicorr_topk_wait_status(const void *workspace, hipStream_t stream);

/*
 * Spin limit of the bounded waits in kernels launched after this call, process-wide (a testing
 * and diagnosis hook: a small limit makes waits give up so that their reporting can be checked
 * while every kernel still runs to its end). spins < 0 restores the default (2^22).
 */
void lilicorr_set_wait_limit(int64_t spins);

/*
 * Step 1 with the candidates' confidence features: the same call as lilicorr_topk (same
 * arguments, workspace and errors), plus, from the same pass over the logits,
 *   feat   [N][B][K][5] fp32 out, the five scalars the head reads for each candidate
 *          (implementation appendix, node construction), for the candidate at rank k of its slot:
 *          { logp_k, exp(logp_k), logp_0 - logp_k, k / (K-1) (0 when K = 1), 1 if k == 0 else 0 }.
 *          Required (not NULL), 16-byte aligned.
 */
lilicorr_status lilicorr_topk_features(const void *logits, lilicorr_dtype dtype, int64_t N,
                                       int64_t B, int64_t V, int K, int32_t *ids, float *logp,
                                       float *feat, void *workspace, size_t workspace_bytes,
                                       hipStream_t stream);

/*
 * Step 2 — candidate in/out vectors. Each candidate carries an out vector and an in vector in
 * R^d, each normalised to unit L2 norm (Sec. 3.2; the two linear heads of the implementation
 * appendix). The trained head is out of reach here; its final linear heads are stood in for by
 * u_in = E[id] W_in and u_out = E[id] W_out (row-vector convention, W[i][j] maps input i to
 * output j), then v = u / ||u|| (a zero u gives a zero v).
 *
 * lilicorr_pack_weights converts W_in, W_out ([d][d] fp32, device) once into the library's
 * matrix-core layout: each fp32 weight is split exactly into three bf16 terms whose sum is the
 * fp32 value, so bf16 products accumulate in fp32 to fp32-grade results.
 *   packed    device buffer of lilicorr_packed_weight_bytes(d) bytes, owned by the caller.
 *
 * lilicorr_candidate_vectors
 *   ids       [N][B][K] int32 (as produced by step 1); an id outside [0, V) gives zero vectors.
 *   E         [V][d] embedding table in `e_dtype` (bf16 uses matrix cores; fp32 uses vector FMA).
 *   packed_w  buffer filled by lilicorr_pack_weights for the same d.
 *   in_vec, out_vec  [N][B][K][d] fp32 out.
 */
size_t lilicorr_packed_weight_bytes(int d);
lilicorr_status lilicorr_pack_weights(const float *W_in, const float *W_out, int d, void *packed,
                                      hipStream_t stream);
lilicorr_status lilicorr_candidate_vectors(const int32_t *ids, const void *E,
                                           lilicorr_dtype e_dtype, int64_t V, int d,
                                           const void *packed_w, int64_t N, int64_t B, int K,
                                           float *in_vec, float *out_vec, hipStream_t stream);

/*
 * Step 3 — batched pair matching scores, Eq. (pair): phi(s, k, k') = sigma * cos(out_{s,k},
 * in_{s+1,k'}); one K x K matrix per adjacent slot pair, batched over the block (Sec. 3.5).
 *
 *   in_vec, out_vec  [N][B][K][d] fp32 (need not be normalised: the cosine normalises).
 *   anchor_out       [N][d] fp32 or NULL: the anchor's out vector (K_0 = 1 in Eq. pair).
 *   sigma            fixed cosine scale (8.0 in the paper's hyper-parameter table).
 *   S                [N][B-1][K][K] fp32 out: S[n][t][k][k'] = sigma*cos(out[n][t][k], in[n][t+1][k']).
 *                    May be NULL when B == 1.
 *   S0               [N][K] fp32 out, required iff anchor_out != NULL:
 *                    S0[n][k'] = sigma*cos(anchor_out[n], in[n][0][k']).
 * A cosine with a zero vector is 0.
 */
lilicorr_status lilicorr_pair_scores(const float *in_vec, const float *out_vec,
                                     const float *anchor_out, int64_t N, int64_t B, int K, int d,
                                     float sigma, float *S, float *S0, hipStream_t stream);

/*
 * Step 4 — greedy left-to-right walk (Sec. 3.5) and the local log-likelihood of Eq. (localar).
 * For every request n, slot t = 0..B-1:
 *   z_t[k] = P_t[k] + logp_weight * logp[n][t][k]   (one fp32 rounding; logp_weight = 0 is the
 *            paper's rule), with P_0 = S0[n] (all zeros when S0 is NULL) and
 *            P_t = S[n][t-1][c_{t-1}] for t >= 1,
 *   c_t    = the lowest k attaining max_k z_t[k],
 *   draft[n][t] = ids[n][t][c_t], choice[n][t] = c_t, logq[n][t] = z_t[c_t] - log sum_k exp z_t[k].
 *
 *   S       [N][B-1][K][K] fp32 (may be NULL when B == 1); S0 [N][K] fp32 or NULL.
 *   logp    [N][B][K] fp32 (read only when logp_weight != 0, but must be valid).
 *   ids     [N][B][K] int32.
 *   draft   [N][B] int32 out; choice [N][B] int32 out or NULL; logq [N][B] fp32 out or NULL.
 */
lilicorr_status lilicorr_greedy_walk(const float *S, const float *S0, const float *logp,
                                     const int32_t *ids, int64_t N, int64_t B, int K,
                                     float logp_weight, int32_t *draft, int32_t *choice,
                                     float *logq, hipStream_t stream);

/*
 * Exact max-path decode (the decode-rule appendix): the path c = (c_0 .. c_{B-1}) maximising
 * Eq. (pathscore), g(c) = P_0[c_0] + sum_{t>=1} S[n][t-1][c_{t-1}][c_t]
 * (+ logp_weight * sum_t logp[n][t][c_t]), with P_0 = S0[n] or all zero when S0 is NULL, found
 * by dynamic programming in O(B K^2). Ties go to the lowest index (predecessor and final
 * candidate), which returns, among all maximising paths, the smallest read from the last slot
 * backwards. Path sums and comparisons are double: every fp32 term is widened exactly and each
 * partial sum is rounded once, in the order of g above (the lambda term after its slot's matching
 * term), so the maximiser is exact unless two path sums differ by less than that rounding.
 *   S, S0, logp, ids, logp_weight   as for lilicorr_greedy_walk.
 *   draft, choice  [N][B] int32 out (choice may be NULL): the path's tokens and indices.
 *   logq           [N][B] fp32 out or NULL: Eq. (localar) along the path,
 *                  z_t[c_t] - log sum_k exp z_t[k] with z_t[k] = P_t(c_{t-1}, k) (+ lambda logp).
 *   score          [N] fp32 out or NULL: g of the returned path, rounded once to fp32.
 * Limits: K <= 64, B <= 8192, B * K <= 65536 (LILICORR_ERR_UNSUPPORTED otherwise).
 */
lilicorr_status lilicorr_viterbi_walk(const float *S, const float *S0, const float *logp,
                                      const int32_t *ids, int64_t N, int64_t B, int K,
                                      float logp_weight, int32_t *draft, int32_t *choice,
                                      float *logq, float *score, hipStream_t stream);

/*
 * Steps 2-4 in one pass (Sec. 3.5: all pair matrices in one batched pass, then the greedy walk;
 * the implementation appendix serves matching and selection as a single replay): the draft,
 * choice and logq that lilicorr_candidate_vectors -> lilicorr_pair_scores -> lilicorr_greedy_walk
 * give on the same inputs, without writing the in/out vectors to memory.
 *   ids, logp      [N][B][K] from step 1.
 *   E, e_dtype, V, d, packed_w   as for lilicorr_candidate_vectors (bf16 E only, d <= 256).
 *   anchor_out     [N][d] fp32 or NULL, as for lilicorr_pair_scores.
 *   sigma          cosine scale of Eq. (pair); logp_weight as for lilicorr_greedy_walk.
 *   S, S0          optional outputs, NULL to skip: the pair scores as lilicorr_pair_scores defines
 *                  them (S0 only with anchor_out).
 *   draft, choice, logq   as for lilicorr_greedy_walk (choice and logq may be NULL).
 *   workspace      lilicorr_score_walk_workspace_bytes(N, B, K) bytes of device memory, owned by
 *                  the caller, zero-filled once before its first use; every call leaves it ready
 *                  for the next (its counters back at zero). Calls sharing a workspace must not
 *                  overlap in time.
 * Limits: K <= 64, 1 + (B-1) K <= 16384, bf16 E, d a multiple of 16 and at most 256
 * (LILICORR_ERR_UNSUPPORTED otherwise; LILICORR_ERR_WORKSPACE if the workspace is too small).
 * lilicorr_score_walk_workspace_bytes returns 0 outside these limits.
 */
size_t lilicorr_score_walk_workspace_bytes(int64_t N, int64_t B, int K);
lilicorr_status lilicorr_score_walk(const int32_t *ids, const float *logp, const void *E,
                                    lilicorr_dtype e_dtype, int64_t V, int d,
                                    const void *packed_w, const float *anchor_out, int64_t N,
                                    int64_t B, int K, float sigma, float logp_weight, float *S,
                                    float *S0, int32_t *draft, int32_t *choice, float *logq,
                                    void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * lilicorr_score_walk without a workspace, for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid allocation). Same
 * arguments, results, limits and errors as lilicorr_score_walk, minus the workspace: its
 * counters and walk table live in an 8 MiB array the library holds on each GPU it runs on, from
 * the first call on that GPU until the process ends. The call allocates nothing (no hipMalloc,
 * no library allocation); it zeroes its counters with a small kernel on `stream` before the pass
 * (no memset node, so it can be recorded into a graph). All calls on one GPU share that array:
 * calls that overlap in time on one GPU (another stream, another thread) race and give wrong
 * results. LILICORR_ERR_WORKSPACE when the call would need more than the array holds, i.e. when
 * lilicorr_score_walk_workspace_bytes(N, B, K) > 8 MiB (about 4,300 requests of 16 slots x 16
 * candidates); LILICORR_ERR_HIP if the array's device address cannot be obtained.
 */
lilicorr_status lilicorr_score_walk_noalloc(const int32_t *ids, const float *logp, const void *E,
                                            lilicorr_dtype e_dtype, int64_t V, int d,
                                            const void *packed_w, const float *anchor_out,
                                            int64_t N, int64_t B, int K, float sigma,
                                            float logp_weight, float *S, float *S0,
                                            int32_t *draft, int32_t *choice, float *logq,
                                            hipStream_t stream);

/*
 * lilicorr_score_walk with certified decisions. The greedy rule (Sec. 3.5) commits the candidate
 * with the largest matching score of Eq. (pair); the pass computes those scores in fp32, whose
 * error can reorder two nearly equal scores. Here every walk decision whose fp32 winner is
 * within `margin` of another candidate is decided again from the definitions in double
 * precision: each contender's u = e W (double, rows summed in order), v = u / ||u|| rounded to
 * fp32, S = fp32(sigma * <o, i> / (||o|| ||i||)) with the sums over the fp32 vectors in index
 * order, z = S (+ logp_weight * logp, one fp32 rounding), then the lowest index among the
 * largest z. Every step is a correctly rounded IEEE double operation in a fixed order, so the
 * decision equals that of a plain double-precision evaluation of the same formulas whenever the
 * fp32 scores are within margin / 2 of those values.
 *   margin       fp32 score gap at or below which a decision is re-scored; finite and >= 0.
 *   S, S0        as for lilicorr_score_walk; entries of re-scored contenders hold the
 *                re-scored values.
 *   logq         as for lilicorr_score_walk; for a re-scored decision the pass's value moved by
 *                the re-scored difference between the new and the fp32 winner.
 *   rescored     [N][B] int32 out or NULL: 0 decision not re-scored, 1 re-scored and unchanged,
 *                2 re-scored and changed from the fp32 winner. 16-byte aligned.
 *   workspace    lilicorr_score_walk_certified_workspace_bytes(N, B, K) bytes, zero-filled once,
 *                as for lilicorr_score_walk.
 * Other arguments, limits and errors as for lilicorr_score_walk; the fp32 weights come from the
 * packed buffer's copy. LILICORR_ERR_INVALID_ARG for a negative or non-finite margin.
 */
size_t lilicorr_score_walk_certified_workspace_bytes(int64_t N, int64_t B, int K);
lilicorr_status lilicorr_score_walk_certified(const int32_t *ids, const float *logp, const void *E,
                                              lilicorr_dtype e_dtype, int64_t V, int d,
                                              const void *packed_w, const float *anchor_out,
                                              int64_t N, int64_t B, int K, float sigma,
                                              float logp_weight, float margin, float *S,
                                              float *S0, int32_t *draft, int32_t *choice,
                                              float *logq, int32_t *rescored, void *workspace,
                                              size_t workspace_bytes, hipStream_t stream);

/*
 * The same single pass with the exact max-path decode in place of the greedy walk (the decode-rule
 * appendix serves each rule as one fused kernel): the draft, choice, logq and score that
 * lilicorr_candidate_vectors -> lilicorr_pair_scores -> lilicorr_viterbi_walk give on the same
 * inputs. Arguments as for lilicorr_score_walk, plus score ([N] fp32 or NULL, as for
 * lilicorr_viterbi_walk); workspace of lilicorr_score_viterbi_workspace_bytes(N, B, K) bytes,
 * zero-filled once, with the same rules. Limits: K <= 64, B <= 8192, B * K <= 65536, bf16 E,
 * d a multiple of 16 and at most 256.
 */
size_t lilicorr_score_viterbi_workspace_bytes(int64_t N, int64_t B, int K);
lilicorr_status lilicorr_score_viterbi(const int32_t *ids, const float *logp, const void *E,
                                       lilicorr_dtype e_dtype, int64_t V, int d,
                                       const void *packed_w, const float *anchor_out, int64_t N,
                                       int64_t B, int K, float sigma, float logp_weight, float *S,
                                       float *S0, int32_t *draft, int32_t *choice, float *logq,
                                       float *score, void *workspace, size_t workspace_bytes,
                                       hipStream_t stream);

/*
 * Steps 3-4 in one pass over the vectors of step 2, for any width lilicorr_candidate_vectors
 * produces (Sec. 3.5: all pair matrices of the block in one batched pass, then the walk; the
 * fused calls above hold both sides' vectors on chip, which bounds them to d <= 256). The draft,
 * choice and logq are those lilicorr_pair_scores -> lilicorr_greedy_walk give on the same inputs,
 * and S / S0 (when requested) are the same values, without S going to memory and back.
 *   in_vec, out_vec  [N][B][K][d] fp32 from lilicorr_candidate_vectors; anchor_out [N][d] or NULL.
 *   logp, ids        [N][B][K] from step 1.
 *   sigma, logp_weight, S, S0, draft, choice, logq   as for lilicorr_score_walk.
 *   workspace        lilicorr_score_walk_workspace_bytes(N, B, K) bytes, zero-filled once, with
 *                    the rules of lilicorr_score_walk (calls sharing one must not overlap).
 * Limits: K <= 64, 1 + (B-1) K <= 16384, N <= 65535, d a multiple of 16 and at most 1024
 * (LILICORR_ERR_UNSUPPORTED otherwise; LILICORR_ERR_WORKSPACE if the workspace is too small).
 */
lilicorr_status lilicorr_pair_walk(const float *in_vec, const float *out_vec,
                                   const float *anchor_out, const float *logp, const int32_t *ids,
                                   int64_t N, int64_t B, int K, int d, float sigma,
                                   float logp_weight, float *S, float *S0, int32_t *draft,
                                   int32_t *choice, float *logq, void *workspace,
                                   size_t workspace_bytes, hipStream_t stream);

/*
 * lilicorr_pair_walk with certified decisions, as lilicorr_score_walk_certified defines them:
 * a decision whose fp32 winner is within `margin` of another candidate is decided again from the
 * embedding rows and the fp32 weights in double precision.
 *   E, e_dtype, V, packed_w   the embedding table and packed weights the vectors were made from
 *                             (bf16 E only; the fp32 weights come from the packed buffer's copy).
 *   margin, rescored          as for lilicorr_score_walk_certified.
 *   workspace                 lilicorr_score_walk_certified_workspace_bytes(N, B, K) bytes.
 * Other arguments and limits as for lilicorr_pair_walk, with d at most 512.
 */
lilicorr_status lilicorr_pair_walk_certified(const float *in_vec, const float *out_vec,
                                             const float *anchor_out, const float *logp,
                                             const int32_t *ids, const void *E,
                                             lilicorr_dtype e_dtype, int64_t V,
                                             const void *packed_w, int64_t N, int64_t B, int K,
                                             int d, float sigma, float logp_weight, float margin,
                                             float *S, float *S0, int32_t *draft, int32_t *choice,
                                             float *logq, int32_t *rescored, void *workspace,
                                             size_t workspace_bytes, hipStream_t stream);

/*
 * The same pass with the exact max-path decode (decode-rule appendix): the draft, choice, logq and
 * score that lilicorr_pair_scores -> lilicorr_viterbi_walk give on the same inputs. Arguments as
 * for lilicorr_pair_walk plus score ([N] fp32 or NULL); workspace of
 * lilicorr_score_viterbi_workspace_bytes(N, B, K) bytes. Limits: K <= 64, B <= 8192,
 * B * K <= 65536, N <= 65535, d a multiple of 16 and at most 1024.
 */
lilicorr_status lilicorr_pair_viterbi(const float *in_vec, const float *out_vec,
                                      const float *anchor_out, const float *logp,
                                      const int32_t *ids, int64_t N, int64_t B, int K, int d,
                                      float sigma, float logp_weight, float *S, float *S0,
                                      int32_t *draft, int32_t *choice, float *logq, float *score,
                                      void *workspace, size_t workspace_bytes,
                                      hipStream_t stream);

/*
 * One draft block as one HIP graph (implementation appendix, serving: candidate extraction,
 * matching and selection replayed as one graph per block). lilicorr_block_graph_create records
 * lilicorr_topk followed by one fused pass (greedy, certified greedy or exact decode) with the
 * arguments below, on a stream of its own, without running anything. Where the fused pass does
 * not apply (fp32 E, or d above 256) it records lilicorr_candidate_vectors into in_vec / out_vec
 * followed by the one-pass decode over them (lilicorr_pair_walk, lilicorr_pair_walk_certified or
 * lilicorr_pair_viterbi, with the same fused_workspace) instead; every replay then runs the
 * block on whatever the buffers hold at that time. The graph keeps the pointers: the buffers
 * must stay allocated, at the same addresses, until the graph is destroyed, and replays that
 * share buffers must not overlap in time. Unlike the calls above, create allocates the graph's
 * host-side objects (no device buffers); launch and destroy allocate nothing.
 * Errors: any status the recorded calls would return for these arguments (nothing is recorded
 * then and *graph is NULL), LILICORR_ERR_INVALID_ARG for a NULL args or graph pointer or an
 * unknown decode, LILICORR_ERR_HIP if capture or instantiation fails.
 */
typedef enum {
    LILICORR_DECODE_GREEDY = 0,    /* lilicorr_score_walk */
    LILICORR_DECODE_CERTIFIED = 1, /* lilicorr_score_walk_certified */
    LILICORR_DECODE_EXACT = 2,     /* lilicorr_score_viterbi */
} lilicorr_decode;

typedef struct {
    /* step 1, as for lilicorr_topk */
    const void *logits;
    lilicorr_dtype logits_dtype;
    int64_t N, B, V;
    int K;
    int32_t *ids;
    float *logp;
    void *topk_workspace;
    size_t topk_workspace_bytes;
    /* steps 2-4, as for the fused pass `decode` names (e_rows is that call's V: rows of E) */
    const void *E;
    lilicorr_dtype e_dtype;
    int64_t e_rows;
    int d;
    const void *packed_w;
    const float *anchor_out;
    float sigma, logp_weight;
    lilicorr_decode decode;
    float margin;       /* certified only */
    float *S, *S0;      /* optional */
    int32_t *draft, *choice;
    float *logq;
    float *score;       /* exact only, optional */
    int32_t *rescored;  /* certified only, optional */
    void *fused_workspace;
    size_t fused_workspace_bytes;
    /* [N][B][K][d] fp32 each: required where the fused pass does not apply, else unused */
    float *in_vec, *out_vec;
} lilicorr_block_args;

typedef struct lilicorr_graph lilicorr_graph;

lilicorr_status lilicorr_block_graph_create(const lilicorr_block_args *args,
                                            lilicorr_graph **graph);
/* Replays the block on `stream` (asynchronous, as every call above). */
lilicorr_status lilicorr_block_graph_launch(lilicorr_graph *graph, hipStream_t stream);
/* Releases the graph (NULL is ignored); the caller makes sure no replay is still running. */
void lilicorr_block_graph_destroy(lilicorr_graph *graph);

/*
 * Scoring-Transformer stand-in — the encoder of the paper's speculative head (implementation
 * appendix, "Architecture"; widths and depth from the hyper-parameter table): a stack of
 * bidirectional Transformer layers over each request's candidate lattice of S slots x K
 * candidates (L = S * K nodes, node j in slot j / K), width H, H / 128 heads of width 128,
 * feed-forward width F, RMSNorm and SiLU. Node order enters only through per-head scalars
 * summed into the pre-softmax scores: a table looked up by (query slot - key slot), and one value
 * for pairs of nodes in the same slot. Each layer is pre-norm:
 *     x += Wo . attn(rmsnorm(x; g_attn));   x += W2 . silu(W1 . rmsnorm(x; g_ffn))
 * with rmsnorm(x; g) = x / sqrt(mean(x^2) + 1e-6) * g, attention logits scaled by 1/sqrt(128),
 * every node attending to every node of its request. A cost-only stand-in: the weights are the
 * caller's (random here); there is no trained head. Precision: bf16 weights; every matrix-core
 * input (normalised activations, Q, K, V, attention probabilities, attention output, SiLU output)
 * is rounded to bf16 (nearest, ties to even); fp32 accumulation; fp32 residual stream.
 *
 * One layer's parameters, all device pointers (weights as raw bf16 bit patterns, applied as
 * y = x W):
 *   w_qkv     [H][3H]  columns [0,H) = Q, [H,2H) = K, [2H,3H) = V; head h owns columns
 *                      h*128 .. h*128+127 of each part
 *   w_o       [H][H];  w_1 [H][F];  w_2 [F][H]
 *   g_attn, g_ffn  [H] fp32 RMSNorm gains
 *   dist_bias [heads][2S-1] fp32: entry (S-1) + (s_query - s_key)
 *   same_bias [heads] fp32
 */
typedef struct {
    const uint16_t *w_qkv, *w_o, *w_1, *w_2;
    const float *g_attn, *g_ffn, *dist_bias, *same_bias;
} lilicorr_scorer_layer;

/* Bytes of one packed layer (weights transposed for the matrix cores, gains, biases) for these
 * sizes; 0 if the sizes are unsupported. */
size_t lilicorr_scorer_packed_bytes(int H, int heads, int F, int64_t S);

/* Packs one layer into `packed` (device, 16-byte aligned, lilicorr_scorer_packed_bytes bytes,
 * caller-owned). `layer` is a host struct of device pointers, read on the stream; the packed
 * layer serves every forward call with the same H, heads, F and S.
 * Limits: H a multiple of 256 with 256 <= H <= 4096 and heads = H / 128; F a multiple of 128
 * with 128 <= F <= 16384; 1 <= S <= 256. */
lilicorr_status lilicorr_scorer_pack(const lilicorr_scorer_layer *layer, int H, int heads, int F,
                                     int64_t S, void *packed, hipStream_t stream);

/* Device scratch bytes lilicorr_scorer_forward needs; 0 if the sizes are unsupported. */
size_t lilicorr_scorer_workspace_bytes(int64_t N, int64_t S, int K, int H, int F);

/* Runs `layers` packed layers over X [N][S*K][H] fp32 in place (device, 16-byte aligned).
 * `packed` holds the layers back to back (layers * lilicorr_scorer_packed_bytes bytes, packed
 * with the same H, heads, F and S). workspace: lilicorr_scorer_workspace_bytes bytes of device
 * scratch, caller-owned, no initial contents needed, clobbered.
 * Limits: those of lilicorr_scorer_pack, and 1 <= K, L = S*K <= 256, N >= 1,
 * N*L*max(3H, F)*4 < 2^31. */
lilicorr_status lilicorr_scorer_forward(float *X, int64_t N, int64_t S, int K, int H, int heads,
                                        int F, int layers, const void *packed, void *workspace,
                                        size_t workspace_bytes, hipStream_t stream);

/* Static, human-readable name of a status code. */
const char *lilicorr_status_string(lilicorr_status s);

#ifdef __cplusplus
}
#endif

#endif /* LILICORR_H_ */
