/*
 * mita.h - C ABI of the MI355X (gfx950) MiTA forward library.
 *
 * Mixture-of-Top-k Attention (arXiv 2602.01219, Sec. 3.2 and Algorithm 1 in
 * Appendix B), forward pass, s routed experts per query:
 *
 *   q_lm  = AdaptiveAvgPool(Q)                 landmark queries  (Sec. 3.2; Tab. A1)
 *   S     = K^T q_lm / sqrt(d)                 landmark-key scores (Eq. top-k; Alg. 1)
 *   I_i   = Top_k(S[i, :])                     expert key sets     (Eq. top-k)
 *   K^(i), V^(i) = K[:, I_i], V[:, I_i]        expert tiles        (Eq. gather)
 *   v_lm_i = Atten(q_lm_i, K, V)               landmark values     (Eq. landmark-value)
 *   e_j(q) = rank-j landmark under q . q_lm_i  routing             (Sec. 3.2, routing logits)
 *   o     = V* softmax(K*^T q / sqrt(d)),  K* = [q_lm, K^(e_1(q)), ..., K^(e_s(q))],
 *           V* likewise                        output              (Eq. mita; Eq. shared-expert)
 * Landmark queries may instead be picked by random selection (Tab. A1) or be
 * supplied by the caller (mita_landmarks_select, mita_forward_lm).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Device pointers. Every tensor argument is a device pointer (HIP device
 *    memory) owned by the caller; the library never allocates device memory
 *    and keeps no state between calls (apart from a thread-local error
 *    string). Pointers must be 16-byte aligned.
 *  - Layout. Tensors are contiguous row-major. q, k, v, o are [B, H, N, d]
 *    (the paper's d x N per head, tokens as rows). Token t sits at position
 *    (t / grid_w, t % grid_w) of the patch grid. Landmark i sits at
 *    (i / lm_w, i % lm_w) of the landmark grid.
 *  - Element type. cfg->dtype selects the storage type of q, k, v, o, q_lm,
 *    v_lm, k_x, v_x: MITA_F32 (float) or MITA_BF16 (bfloat16 bits). All
 *    accumulation, scores, logits and softmax are fp32 in both cases.
 *  - Streams. `stream` is a hipStream_t (NULL = the legacy default stream).
 *    Calls only enqueue work on it and return; they never synchronise the
 *    host (except mita_timer_read).
 *  - Errors. Arguments are validated on the host before anything is
 *    enqueued; on error nothing is launched and a status != MITA_OK is
 *    returned, with details from mita_last_error(). No exception crosses the
 *    ABI. NaN inputs are a caller error: results are then unspecified (but
 *    every kernel still stays in bounds and terminates); the top-k order
 *    ranks a NaN score as -inf.
 *  - Workspace. Entry points that take (ws, ws_bytes) need at least
 *    mita_workspace_size(cfg, which) bytes of device memory there, 256-byte
 *    aligned; its contents on entry do not matter. Calls sharing one
 *    workspace on different streams race.
 */
#ifndef MITA_H
#define MITA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define MITA_OK 0
#define MITA_ERR_INVALID_ARG 1   /* bad sizes/grids, k or M out of [1, N], null or misaligned pointer, o aliasing an input, both branches off */
#define MITA_ERR_UNSUPPORTED 2   /* d not in {64, 128}; s outside [1, MITA_MAX_S]; unknown dtype; N beyond the supported maximum */
#define MITA_ERR_WORKSPACE 3     /* ws_bytes smaller than mita_workspace_size() */
#define MITA_ERR_HIP 4           /* a HIP runtime or launch failure; see mita_last_error() */

/* Storage types. */
#define MITA_F32 0
#define MITA_BF16 1

/* Flags (cfg->flags). */
#define MITA_FLAG_STAGED_GATHER 0x1u  /* mita_forward: materialise the expert tiles (Eq. gather) and
                                         attend over them, instead of reading the selected K/V rows
                                         in place inside the attention kernel. Same results. */
#define MITA_FLAG_FULL_SCORES 0x2u    /* mita_forward: store the whole score matrix S and select the
                                         top-k sets from it (the mita_scores + mita_topk path), instead
                                         of selecting inside the score pass. Same results. */

/* Largest sequence length the library accepts. */
#define MITA_MAX_N 65536
/* Largest number of routed experts per query. */
#define MITA_MAX_S 4

typedef void *mita_stream_t; /* a hipStream_t */

/*
 * Problem description (Algorithm 1 "Require": Q, K, V in R^{d x N}, the number of
 * landmark queries m, the expert width k; s routed experts per query, Eq. mita).
 */
typedef struct {
  int32_t B, H, N, d;      /* batch, heads, tokens, head dim; d in {64, 128} */
  int32_t grid_h, grid_w;  /* token grid, grid_h * grid_w == N; grid_h == 1 gives 1-D pooling */
  int32_t M, lm_h, lm_w;   /* landmarks (the paper's m), lm_h * lm_w == M, lm_h <= grid_h, lm_w <= grid_w */
  int32_t k;               /* expert width, 1 <= k <= N */
  int32_t s;               /* routed experts per query, 1 <= s <= MITA_MAX_S and s <= M (Eq. mita; the paper
                              runs s = 1). With s > 1 the keys of the s experts are concatenated as
                              Eq. mita writes them: a key two of a query's experts select counts twice.
                              Ignored when use_routed == 0. */
  int32_t use_shared;      /* shared expert (Eq. shared-expert): landmarks as keys, landmark values as values */
  int32_t use_routed;      /* routed top-k expert (Eq. mita-expert); at least one of the two must be set */
  int32_t dtype;           /* MITA_F32 or MITA_BF16 */
  float scale;             /* softmax/score scale; 0 means 1/sqrt(d) */
  uint32_t flags;          /* MITA_FLAG_* */
} mita_cfg_t;

/* Workspace kinds for mita_workspace_size. */
#define MITA_WS_FORWARD 0
#define MITA_WS_SCORES 1
#define MITA_WS_TOPK 2
#define MITA_WS_ROUTE 3
#define MITA_WS_ATTEND 4
#define MITA_WS_BACKWARD 5
#define MITA_WS_TOME 6

/* Host-only validation of cfg (no device needed). Returns a status code. */
int mita_check(const mita_cfg_t *cfg);

/* Bytes of workspace entry point `which` needs for cfg (0 if cfg is invalid). */
size_t mita_workspace_size(const mita_cfg_t *cfg, int which);

/* Static description of a status code; never NULL. */
const char *mita_status_string(int status);

/* Detail of the last failure on the calling thread ("" if none). */
const char *mita_last_error(void);

/*
 * The whole forward (Algorithm 1; output Eq. mita).
 *   q, k, v : [B, H, N, d] inputs;  o : [B, H, N, d] output (must not overlap q, k, v).
 *   ws      : >= mita_workspace_size(cfg, MITA_WS_FORWARD) bytes.
 * With s > 1 the attention runs expert by expert and the s partial results of
 * each query are merged by their log-sum-exp (the expert-wise evaluation of
 * Eq. mita that Sec. 3.2 allows); the shared expert goes with the rank-1 one.
 * The top-k sets are those mita_topk computes from mita_scores' S (bit for
 * bit), but S is normally not stored: a pivot estimated from a sample of
 * each score row bounds the row's top-k from below, the score pass lists
 * only the scores above it, and the exact selection runs on that list. A row
 * whose list turns out too short or too long is recomputed in full and
 * selected exactly (see mita_forward_fallbacks). Without MITA_FLAG_FULL_SCORES
 * this applies when mita_select_plan reports it: always for N <= 1024, else
 * when a pivot rank and a list cap (at most 8192) exist for which each way a
 * row's list can miss has probability <= 1e-9 per row on inputs whose scores
 * are exchangeable over token positions (k up to about N / 8).
 */
int mita_forward(const mita_cfg_t *cfg, const void *q, const void *k, const void *v, void *o,
                 void *ws, size_t ws_bytes, mita_stream_t stream);

/*
 * mita_forward for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same forward and results, with its workspace in a static device array of
 * MITA_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on
 * until the process ends. It calls no hipMalloc, hipFree or other
 * allocating routine. The calling thread's current device must be the one
 * the stream and tensors belong to.
 *   q, k, v, o : as mita_forward.
 * Returns MITA_ERR_WORKSPACE (launching nothing) when the forward needs more
 * workspace than the scratch holds (mita_workspace_size(cfg, MITA_WS_FORWARD)
 * > MITA_NOALLOC_SCRATCH_BYTES). Every call on one GPU uses that GPU's one
 * array: calls that overlap on one GPU (other streams or threads) race.
 */
#define MITA_NOALLOC_SCRATCH_BYTES (64u << 20)
int mita_forward_noalloc(const mita_cfg_t *cfg, const void *q, const void *k, const void *v, void *o,
                         mita_stream_t stream);

/*
 * Diagnostic: the number of landmark rows whose top-k selection in the last
 * mita_forward on workspace ws fell back to recomputing the full score row
 * (0 when that forward stored the whole score matrix). Waits for `stream`.
 *   count : host pointer, output.
 */
int mita_forward_fallbacks(const mita_cfg_t *cfg, const void *ws, size_t ws_bytes, int64_t *count,
                           mita_stream_t stream);

/*
 * Diagnostic, host only: how mita_forward selects the top-k sets for cfg.
 * *fused = 1 if the selection runs inside the score pass (then *ns keys of
 * each landmark row are sampled, the pivot is the *rank-th largest sampled
 * score and the exact selection takes lists of up to *cap candidates), 0 if
 * the whole score matrix is stored and selected from. Any output may be NULL.
 */
int mita_select_plan(const mita_cfg_t *cfg, int32_t *fused, int32_t *ns, int32_t *rank, int32_t *cap);

/*
 * Landmark queries (Sec. 3.2: average pooling over uniformly spaced windows;
 * Algorithm 1 AdaptiveAvgPool; Tab. A1 makes 2-D pooling the default).
 * Window of landmark (a, b): rows [floor(a*gh/lh), ceil((a+1)*gh/lh)), columns
 * [floor(b*gw/lw), ceil((b+1)*gw/lw)).
 *   q    : [B, H, N, d];  q_lm : [B, H, M, d] output (fp32 mean, rounded once to dtype).
 */
int mita_landmarks(const mita_cfg_t *cfg, const void *q, void *q_lm, mita_stream_t stream);

/*
 * Landmark queries by random selection (Tab. A1, landmark extraction): the
 * caller draws the tokens, landmark i of slice (b, h) is the query of token
 * sel[b, h, i].
 *   q   : [B, H, N, d];  sel : [B, H, M] int32, entries in [0, N) (distinct, as
 *         the selection draws them; repeats are not rejected);
 *   q_lm : [B, H, M, d] output (copied rows). An entry outside [0, N) gives a
 *         row of NaN (nothing is read for it).
 */
int mita_landmarks_select(const mita_cfg_t *cfg, const void *q, const int32_t *sel, void *q_lm,
                          mita_stream_t stream);

/*
 * Landmark queries by token merging (Tab. A1 lists ToMe among the landmark
 * extractions): bipartite soft matching applied in rounds until M tokens
 * remain. A round over the current sequence of n merged tokens (each the mean
 * of its tokens' queries, in sequence order) splits it into A (even
 * positions) and B (odd positions); each A token's match is its B token of
 * largest cosine similarity (lower B position on ties); the r = min(n - M,
 * |A|) edges of largest similarity (lower A position on ties) merge each of
 * those A tokens into its match; the survivors keep their order. Landmark i
 * is the mean of the queries of the tokens merged into the i-th final token.
 *   q : [B, H, N, d];  q_lm : [B, H, M, d] output;
 *   assign : [B, H, N] int32 output, the landmark of every token, or NULL;
 *   ws : >= mita_workspace_size(cfg, MITA_WS_TOME) bytes.
 * Member sums are exact in 64-bit fixed point (units of 2^-32), so the
 * result does not depend on the order of the merge additions; the
 * similarities are fp32. Queries whose window sums reach 2^31 in magnitude
 * overflow that format (results then unspecified; every access stays in
 * bounds). Feed q_lm to mita_forward_lm for the forward with these landmarks.
 */
int mita_landmarks_tome(const mita_cfg_t *cfg, const void *q, void *q_lm, int32_t *assign, void *ws,
                        size_t ws_bytes, mita_stream_t stream);

/*
 * mita_forward with caller-supplied landmark queries (random selection, or any
 * other extraction): every step of Algorithm 1 after AdaptiveAvgPool, with
 * q_lm in its place. lm_h, lm_w, grid_h and grid_w are validated as for
 * mita_forward but not otherwise used.
 *   q_lm : [B, H, M, d] input;  q, k, v, o, ws : as mita_forward
 *          (ws >= mita_workspace_size(cfg, MITA_WS_FORWARD) bytes).
 */
int mita_forward_lm(const mita_cfg_t *cfg, const void *q, const void *k, const void *v, const void *q_lm,
                    void *o, void *ws, size_t ws_bytes, mita_stream_t stream);

/*
 * Landmark-key scores and landmark values, computed together (Sec. 3.2 notes
 * Eq. top-k and Eq. landmark-value share K^T q_lm).
 *   q_lm   : [B, H, M, d] landmark queries;  k, v : [B, H, N, d].
 *   scores : [B, H, M, N] fp32 output, S[i, n] = fl(q_lm_i . k_n) * scale, or NULL.
 *   v_lm   : [B, H, M, d] output, v_lm_i = sum_n softmax_n(S[i, :]) v_n (Eq. landmark-value), or NULL.
 *   ws     : >= mita_workspace_size(cfg, MITA_WS_SCORES) bytes.
 */
int mita_scores(const mita_cfg_t *cfg, const void *q_lm, const void *k, const void *v,
                float *scores, void *v_lm, void *ws, size_t ws_bytes, mita_stream_t stream);

/*
 * Top-k selection per landmark (Eq. top-k), exact: I_i holds the k token
 * indices that come first when tokens are ordered by larger S[i, n], equal
 * scores by lower n (-0 equals +0). Written in ascending index order.
 *   scores : [B, H, M, N] fp32;  idx : [B, H, M, k] int32 output.  Requires N <= MITA_MAX_N.
 *   ws     : may be NULL (mita_workspace_size(cfg, MITA_WS_TOPK) is 0).
 */
int mita_topk(const mita_cfg_t *cfg, const float *scores, int32_t *idx, void *ws, size_t ws_bytes,
              mita_stream_t stream);

/*
 * Expert tiles (Eq. gather): k_x[b,h,i,j,:] = k[b,h,idx[b,h,i,j],:], likewise v_x.
 *   idx : [B, H, M, k] int32, every entry in [0, N);  k_x, v_x : [B, H, M, k, d] outputs.
 */
int mita_gather(const mita_cfg_t *cfg, const void *k, const void *v, const int32_t *idx,
                void *k_x, void *v_x, mita_stream_t stream);

/*
 * Routing (Sec. 3.2: logits Q^T q_lm, rank-j expert e_j(q); Algorithm 1 ArgMax,
 * ArgSort, BinCount, CumSum). With s = 1, expert[n] is the lowest i attaining
 * the maximum of fl(q_n . q_lm_i) * scale and queries are grouped by expert,
 * stably:
 *   q : [B, H, N, d];  q_lm : [B, H, M, d].
 *   expert  : [B, H, N] int32 output;
 *   perm    : [B, H, N] int32 output, tokens of expert 0, then expert 1, ..., ascending inside a group;
 *   offsets : [B, H, M+1] int32 output, offsets[0] = 0, offsets[M] = N, group i = perm[offsets[i] : offsets[i+1]].
 * With s > 1, expert[n, j] is the landmark of rank j when landmarks are
 * ordered by larger fl(q_n . q_lm_i) * scale, equal values by lower i; the
 * (query, rank) pairs p = n * s + j are grouped into 2 M groups: pair p goes
 * to group expert[n, j] if j = 0 and to group M + expert[n, j] otherwise,
 * stably in p:
 *   expert  : [B, H, N, s] int32 output;
 *   perm    : [B, H, N * s] int32 output, pair ids grouped as above;
 *   offsets : [B, H, 2M+1] int32 output, offsets[2M] = N * s.
 *   ws      : >= mita_workspace_size(cfg, MITA_WS_ROUTE) bytes.
 */
int mita_route(const mita_cfg_t *cfg, const void *q, const void *q_lm, int32_t *expert,
               int32_t *perm, int32_t *offsets, void *ws, size_t ws_bytes, mita_stream_t stream);

/*
 * Attention of every query over the shared expert and its s routed experts,
 * as one softmax over the concatenated keys (Eq. mita; Algorithm 1's
 * shared-expert attention, varlen expert attention and online-softmax combine).
 *   q : [B, H, N, d];  q_lm, v_lm : [B, H, M, d] (read if use_shared);
 *   k_x, v_x : [B, H, M, k, d] expert tiles (read if use_routed);
 *   perm, offsets : routing as produced by mita_route for the same s (read if use_routed);
 *   o : [B, H, N, d] output in token order.
 *   ws : >= mita_workspace_size(cfg, MITA_WS_ATTEND) bytes (with s > 1 it holds the
 *        fp32 partial result and log-sum-exp of every (query, expert) pair).
 */
int mita_attend(const mita_cfg_t *cfg, const void *q, const void *q_lm, const void *v_lm,
                const void *k_x, const void *v_x, const int32_t *perm, const int32_t *offsets,
                void *o, void *ws, size_t ws_bytes, mita_stream_t stream);

/*
 * Backward pass: the gradients of mita_forward's output o with respect to q,
 * k and v for an upstream gradient dO, by the chain rule through Eq. mita (the
 * softmax over the shared and routed keys), Eq. landmark-value (the softmax
 * over all keys that forms the landmark values) and the pooling of the
 * landmark queries (Sec. 3.2). The top-k sets (Eq. top-k) and the routing are
 * held fixed: they change only where two scores or logits cross, so no
 * gradient flows through a selection or an argmax. The call recomputes them
 * (and the landmarks and landmark values) from q, k, v exactly as
 * mita_forward does.
 *   q, k, v : [B, H, N, d] the forward's inputs;  o : [B, H, N, d] its output;
 *   dO : [B, H, N, d] upstream gradient;  dq, dk, dv : [B, H, N, d] outputs in
 *        the io type (must not overlap the inputs or each other).
 *   ws : >= mita_workspace_size(cfg, MITA_WS_BACKWARD) bytes.
 * Requires s = 1 when use_routed is set (MITA_ERR_UNSUPPORTED otherwise). The
 * key-side gradients are summed with fp32 atomic adds, whose order varies:
 * dk, dv and dq are reproducible only to rounding, not bit for bit.
 */
int mita_backward(const mita_cfg_t *cfg, const void *q, const void *k, const void *v, const void *o,
                  const void *dO, void *dq, void *dk, void *dv, void *ws, size_t ws_bytes, mita_stream_t stream);

/*
 * Per-launch timing of mita_forward with HIP events (profiling aid).
 * A timer holds event slots for up to max_calls forward calls. Each
 * mita_forward_timed call records one event on the stream before its first
 * kernel and one behind each kernel it launches (at most MITA_MAX_LAUNCHES),
 * so the interval of a launch is that kernel's time on the stream. Every
 * launch belongs to one of MITA_NUM_STAGES stages (0 landmarks, 1 scores,
 * 2 top-k, 3 gather, 4 routing, 5 attention); a kernel that does the work of
 * two stages (the forward's selection finish runs inside the routing
 * launches) counts under the later one, and a stage that launches nothing
 * takes no time.
 */
#define MITA_NUM_STAGES 6
#define MITA_MAX_LAUNCHES 32
typedef struct mita_timer mita_timer_t;
int mita_timer_create(mita_timer_t **timer, int max_calls);
int mita_timer_destroy(mita_timer_t *timer);
int mita_timer_reset(mita_timer_t *timer);
/* Waits for the recorded events; fills ms[call * MITA_NUM_STAGES + stage] with
 * the summed launch times of each stage; *n_calls = calls recorded. */
int mita_timer_read(mita_timer_t *timer, float *ms, int ms_len, int *n_calls);
/* Waits for the recorded events; for recorded call `call`, fills the first
 * *n_launches entries of kernels (static kernel names, owned by the library),
 * stages and ms (each array holds at least cap entries). */
int mita_timer_launches(mita_timer_t *timer, int call, int cap, const char **kernels, int32_t *stages, float *ms,
                        int32_t *n_launches);
int mita_forward_timed(const mita_cfg_t *cfg, const void *q, const void *k, const void *v, void *o,
                       void *ws, size_t ws_bytes, mita_stream_t stream, mita_timer_t *timer);
/* mita_backward with the per-launch timing of mita_forward_timed. */
int mita_backward_timed(const mita_cfg_t *cfg, const void *q, const void *k, const void *v, const void *o,
                        const void *dO, void *dq, void *dk, void *dv, void *ws, size_t ws_bytes,
                        mita_stream_t stream, mita_timer_t *timer);
/* mita_forward_lm with the per-launch timing of mita_forward_timed. */
int mita_forward_lm_timed(const mita_cfg_t *cfg, const void *q, const void *k, const void *v, const void *q_lm,
                          void *o, void *ws, size_t ws_bytes, mita_stream_t stream, mita_timer_t *timer);

#ifdef __cplusplus
}
#endif
#endif /* MITA_H */
