/*
 * dartree.h - C ABI of libdartree: DARTree fixed-width draft-tree construction
 * on one AMD Instinct MI355X (gfx950).
 *
 * The library implements the construction of Algorithm 1 ("DARTree
 * Construction", Sec. 3.2) and the deferred pruning of Sec. 3.3 (eq. (5),
 * Lemma 1) of "DARTree: Speculative Diffusion Decoding with Autoregressive
 * Draft Trees" (arXiv 2608.13524):
 *
 *   for d = 1..L, for every node u_<d of S_{d-1} in one batch:
 *     t   = A r(u_<d)                              correction head, state part
 *     a   = bf16(tanh(t + H_d))                    correction feature
 *     z   = L_d^base + U a                         corrected logits, all V tokens
 *     log q~_d = log_softmax(z / tau)              tau = T if T > 0 else 1
 *     C(u_<d) = top-k ids of z, (z desc, id asc)   per-node candidate set
 *     s(u_1:d) = (s(u_<d) + log q~_d(u_d)) + beta  eq. (5), one depth at a time
 *     S_d = top-W children by (s desc, parent slot asc, token asc)
 *     r(u_1:d) = bf16(tanh(t + e U[u_d])), e = fp32(sqrt(h))   state update
 *   T = top-B of S = S_1 u ... u S_L by (s desc, depth asc, slot asc)
 *
 * The paper fixes only the signature of the correction head g(H_d, r(u_<d))
 * and that r(u_1:d) is computed from r(u_<d) and u_d; the Elman residual head
 * above (A [h][h], U [V][h] with U's rows doubling as token embeddings) is
 * this library's choice.  With beta <= 0 the top-B set is prefix-closed and
 * equals best-first heap selection (Lemma 1); beta > 0 is rejected.
 *
 * Conventions for every entry point:
 *  - Device pointers are HIP device memory owned by the caller; the library
 *    never allocates or frees device memory and keeps no pointer after return.
 *  - All work is enqueued on `stream` (a hipStream_t; 0 = the null stream);
 *    no call synchronises the host with the device (except the debug checks
 *    enabled by DARTREE_DEBUG=1, see "Depth order").  Outputs are valid once
 *    the stream's work completes.
 *  - Every argument is validated on the host before anything is enqueued;
 *    on any error nothing is enqueued and no output is written.
 *  - One workspace must not be used by two calls that may run concurrently.
 *  - Input values are assumed finite; non-finite inputs give undefined trees
 *    (never out-of-bounds accesses).
 *  - Layouts are dense row-major with the rightmost index fastest.  "act"
 *    tensors are bfloat16 (raw 16-bit patterns) in DARTREE_BF16 mode and
 *    float32 in DARTREE_FP32 mode.  Every pointer must be 16-byte aligned.
 */
#ifndef DARTREE_H
#define DARTREE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DARTREE_ABI_VERSION 8

/* Limits of this implementation (calls beyond them return
 * DARTREE_ERR_UNSUPPORTED). */
#define DARTREE_MAX_VOCAB (1 << 20)      /* V */
#define DARTREE_MAX_DEPTH 64             /* L */
#define DARTREE_MAX_WIDTH 2048           /* W */
#define DARTREE_MAX_BRANCH 32            /* k over the full vocabulary */
#define DARTREE_MAX_CANDIDATES 256       /* K of a shared candidate set (k <= K) */
#define DARTREE_MAX_SORT 4096            /* n_{d-1}*k candidates, |S| nodes, B */
#define DARTREE_MAX_HEAP_BUDGET 1024     /* B of the sequential heap (pops per round) */

typedef enum dartree_status {
  DARTREE_OK = 0,
  DARTREE_ERR_INVALID_ARG = 1, /* a size, value or pointer violates the contract */
  DARTREE_ERR_UNSUPPORTED = 2, /* valid per the paper but beyond this library's limits */
  DARTREE_ERR_WORKSPACE = 3,   /* workspace missing, misaligned or smaller than required */
  DARTREE_ERR_HIP = 4,         /* a kernel launch failed (hipGetLastError) */
  DARTREE_ERR_ORDER = 5,       /* Algorithm 1's depths out of order on a workspace: the call would read
                                  levels no earlier call produced (see "Depth order" below) */
  DARTREE_ERR_NONFINITE = 6    /* debug mode only: a normaliser of the depth just run is not finite */
} dartree_status;

typedef enum dartree_precision {
  DARTREE_FP32 = 0, /* every tensor fp32, no intermediate rounding */
  DARTREE_BF16 = 1  /* head weights, hidden and states bf16; logits fp32; bf16 MFMA with fp32 accumulation */
} dartree_precision;

typedef enum dartree_head {
  DARTREE_HEAD_RNN = 0,    /* recurrent correction: r(u_1:d) = act(tanh(t(u_<d) + e U[u_d])), the
                              state summarises the whole prefix (Sec. 2.2, the Domino head) */
  DARTREE_HEAD_MARKOV = 1  /* Markov correction (Sec. 2.2, the DSpark-Markov head of Table 3):
                              r(u_1:d) = act(e U[u_d]), the last token's embedding only, so the
                              children's distribution depends on the path through its last token;
                              prefix_state is then the last verified token's embedding */
} dartree_head;

/* Scalar arguments of Algorithm 1 (host struct). */
typedef struct dartree_params {
  int32_t batch;       /* b >= 1 independent requests, each built as its own tree */
  int32_t vocab;       /* V >= 1 */
  int32_t hidden;      /* h >= 1; a multiple of 64 in DARTREE_BF16 mode */
  int32_t depth;       /* L = gamma, the draft block length, 1..DARTREE_MAX_DEPTH */
  int32_t width;       /* W, layer width (nodes kept per depth), >= 1 */
  int32_t branch;      /* k, candidate children scored per node, 1 <= k <= V */
  int32_t budget;      /* B, verification budget (nodes of the emitted tree), >= 1 */
  int32_t precision;   /* dartree_precision */
  float temperature;   /* T >= 0, finite; tau = T if T > 0 else 1 */
  float depth_bonus;   /* beta <= 0, finite (Lemma 1 needs beta <= 0) */
  int32_t candidates;  /* K >= 0.  0: every node is scored over the whole vocabulary
                          and keeps its own top-k (the "Full" variant of Appendix D;
                          k <= DARTREE_MAX_BRANCH).  K > 0: Alg. 1 as printed - each
                          request and depth uses the shared candidate set
                          C_d = TopK(L_d^base, K) by (value desc, id asc); the head
                          scores only C_d and log q~ is normalised over C_d; each
                          node keeps its top-k of C_d, 1 <= k <= K <= V (k = K keeps
                          all of C_d, the paper's default K = 64) */
  int32_t head;        /* dartree_head: how a child's state is formed (t, a, z are the same) */
} dartree_params;

/* Device inputs of one round (the inputs Algorithm 1 takes). */
typedef struct dartree_inputs {
  const float* drafter_logits; /* L^base: fp32 [b][L][V] */
  const void* drafter_hidden;  /* H: act [b][L][h] */
  const void* prefix_state;    /* r_0: act [b][h], the root state of each request */
  const void* head_A;          /* A: act [h][h], state transition (t_i = sum_j A[i][j] r_j) */
  const void* head_U;          /* U: act [V][h], output projection and token embedding */
} dartree_inputs;

/* Device outputs: the flattened verification tree of each request (Sec. 2.3).
 * Nodes are in canonical breadth-first order: depth ascending, then the
 * parent's output index ascending, then token ascending.  Slots at and after
 * num_nodes[i] hold token -1, parent -1, depth 0, score -inf, mask 0. */
typedef struct dartree_tree {
  int32_t* tokens;    /* [b][B] token id of the node */
  int32_t* parents;   /* [b][B] output index of the parent; -1 for depth-1 nodes (children of the root) */
  int32_t* depths;    /* [b][B] 1..L */
  float* scores;      /* [b][B] s_beta of the node, eq. (5) */
  uint64_t* mask;     /* [b][B][ceil(B/64)] tree-attention mask: bit (j % 64) of word
                         j / 64 in row i is set iff node j is node i or an ancestor of it;
                         the verified context is visible to every node and is not stored */
  int32_t* num_nodes; /* [b] min(B, |S|) */
} dartree_tree;

/* Device destination of dartree_export_supertree.  n_d = min(W, n_{d-1} k),
 * n_0 = 1.  Level arrays use a fixed stride W per request; per-parent arrays
 * use a fixed stride b*W rows per depth, where depth d's rows are
 * q * n_{d-1} + j for parent slot j of request q.  Any member may be NULL
 * (not copied). */
typedef struct dartree_supertree {
  int32_t* tokens;    /* [L][b][W] token of slot i of S_d (i < n_d) */
  int32_t* parents;   /* [L][b][W] parent's slot in S_{d-1} (0, the root, at d = 1) */
  float* scores;      /* [L][b][W] s_beta */
  float* lse;         /* [L][b*W] log sum_v exp(z_v / tau) of each parent row */
  float* cand_logp;   /* [L][b*W][k] log q~ of the row's top-k candidates, best first */
  int32_t* cand_ids;  /* [L][b*W][k] their token ids */
  int32_t* csets;     /* [b][L][K] shared candidate sets C_d, best first (candidates > 0 only) */
} dartree_supertree;

/* ABI version (DARTREE_ABI_VERSION of the built library). */
int32_t dartree_abi_version(void);

/* Static English description of a status code; never NULL. */
const char* dartree_status_string(dartree_status status);

/* Host-only check of `p` against the contract above (no HIP call). */
dartree_status dartree_validate(const dartree_params* p);

/* Bytes of device workspace needed by the calls below for `p` (host only).
 * The workspace holds every level of the supertree, per-parent candidates
 * and the per-depth scratch (states, features, logits [b*W][V] fp32). */
dartree_status dartree_workspace_size(const dartree_params* p, size_t* bytes);

/* Depth order.  Algorithm 1's loop runs d = 1..L and depth d reads the level
 * and states depth d - 1 left in the workspace.  The library records, per
 * workspace (by address, up to 256 workspaces, least recently used dropped),
 * the parameters and the last depth enqueued by dartree_expand_depth or
 * dartree_build_tree on the host.  dartree_expand_depth(d > 1) on a
 * workspace whose record is not (the same parameters, d - 1), and
 * dartree_prune on one whose record is not depth L, return DARTREE_ERR_ORDER
 * with nothing enqueued; d = 1 always starts a new round.  Memory that held
 * a round of the same parameters at the same address keeps that round's
 * record until depth 1 runs on it again.  Replays of a
 * captured graph do not update the record.  Each depth's selection kernel
 * also writes {parameters, d} into the workspace; with the environment
 * variable DARTREE_DEBUG=1 (read once per process) dartree_expand_depth and
 * dartree_prune synchronise the stream and check that device record too,
 * and dartree_expand_depth checks, after its kernels ran, that the depth's
 * normalisers are finite (DARTREE_ERR_NONFINITE).  Debug checks are skipped
 * while the stream is being captured. */

/* One iteration of Algorithm 1's depth loop (d = 1..L): score every child of
 * every node of S_{d-1} over the full vocabulary, keep the top-W as S_d and
 * compute their states.  Reads S_{d-1} from `ws` (d = 1 reads
 * in->prefix_state), so depths must be enqueued in order 1..L on one stream
 * with the same workspace (DARTREE_ERR_ORDER otherwise, see above).
 * ws: device, 256-byte aligned, >= workspace_size. */
dartree_status dartree_expand_depth(const dartree_params* p, const dartree_inputs* in,
                                    int32_t d, void* ws, size_t ws_bytes, hipStream_t stream);

/* Deferred best-first pruning (Sec. 3.3, Algorithm 1 after the loop): top-B of
 * the supertree held in `ws` after dartree_expand_depth(1..L), emitted as the
 * flattened tree with parent indices and the ancestor-or-self mask.
 * DARTREE_ERR_ORDER if the workspace's record is not depth L. */
dartree_status dartree_prune(const dartree_params* p, const void* ws, size_t ws_bytes,
                             const dartree_tree* out, hipStream_t stream);

/* Algorithm 1 end to end: expand_depth(1..L) then prune. */
dartree_status dartree_build_tree(const dartree_params* p, const dartree_inputs* in,
                                  void* ws, size_t ws_bytes, const dartree_tree* out,
                                  hipStream_t stream);

/* Kernels of one round, in launch order, as indexed by dartree_build_tree_timed. */
#define DARTREE_KERNEL_HEAD 0   /* t = A r, a = bf16(tanh(t + H_d)) */
#define DARTREE_KERNEL_LOGITS 1 /* z = L_d^base + U a (over C_d with shared candidate sets) */
#define DARTREE_KERNEL_LSE 2    /* log-softmax normaliser and per-row top-k (row segments);
                                   with shared candidate sets: the sets of every depth,
                                   at d = 1 only (nothing at d > 1) */
#define DARTREE_KERNEL_SELECT 3 /* segment merge (or the softmax over C_d), segmented top-W
                                   and the state update of the kept children (no state
                                   update at d = L) */
#define DARTREE_KERNELS_PER_DEPTH 4

/* dartree_build_tree that also records `events` (created by the caller, for
 * instance with hipEventCreate) on `stream` around each launch: for depth d
 * and kernel kind c, events[2 i] before and events[2 i + 1] after, with
 * i = (d - 1) * DARTREE_KERNELS_PER_DEPTH + c; the prune is i = L *
 * DARTREE_KERNELS_PER_DEPTH.  `events` holds 2 (4 L + 1) entries; NULL
 * entries are not recorded.  For measuring kernel durations inside a round. */
dartree_status dartree_build_tree_timed(const dartree_params* p, const dartree_inputs* in, void* ws,
                                        size_t ws_bytes, const dartree_tree* out, hipEvent_t* events,
                                        hipStream_t stream);

/* Copy the supertree levels and per-parent candidates out of `ws` into the
 * caller's device buffers (layouts in dartree_supertree), for inspection.
 * Levels past the last depth enqueued hold stale values; DARTREE_ERR_ORDER
 * if no depth has been enqueued on `ws` with these parameters. */
dartree_status dartree_export_supertree(const dartree_params* p, const void* ws, size_t ws_bytes,
                                        const dartree_supertree* dst, hipStream_t stream);

/* Copy the states r(u) of the nodes of S_d (act [b][n_d][h], row q*n_d + i
 * for slot i of request q) out of `ws` into `dst` (device).  Valid for
 * 1 <= d < L once dartree_expand_depth(d) has run and until
 * dartree_expand_depth(d + 2) is enqueued (states are double-buffered; the
 * last depth computes none); DARTREE_ERR_ORDER outside that window. */
dartree_status dartree_export_states(const dartree_params* p, const void* ws, size_t ws_bytes, int32_t d,
                                     void* dst, hipStream_t stream);

/* Copy the features a = act(tanh(A r + H_d)) of depth d's parent rows (act
 * [b][n_{d-1}][h], row q*n_{d-1} + j for parent slot j of request q) out of
 * `ws` into `dst` (device), for inspection.  Valid once
 * dartree_expand_depth(d) has run and until the next depth is enqueued
 * (DARTREE_ERR_ORDER otherwise). */
dartree_status dartree_export_features(const dartree_params* p, const void* ws, size_t ws_bytes, int32_t d,
                                       void* dst, hipStream_t stream);

/* ---- single steps on caller buffers --------------------------------------
 * The kernels of one depth, exposed for callers that assemble their own loop
 * (and for testing each step on injected inputs). */

/* Bytes of device scratch dartree_project needs for this shape (host only;
 * 0 for shapes that never split a tile along K).  bf16 with >= 512 rows and
 * >= 16384 columns: 64 MB for partial tiles, plus rows * hidden * 2 bytes for
 * a copy of x in MFMA-fragment order when rows is a multiple of 512. */
dartree_status dartree_project_workspace_size(int32_t precision, int32_t rows, int32_t vocab, int32_t hidden,
                                              size_t* bytes);

/* Corrected logits (Algorithm 1, every prefix of a depth corrected in one batch):
 * z[m][v] = bias[m / rows_per_group][v] + sum_i x[m][i] U[v][i]
 * for m < rows, v < vocab.  x: act [rows][hidden]; U: act [vocab][hidden];
 * bias: fp32 rows of length vocab, row g at bias + g * bias_stride (elements);
 * z: fp32 [rows][vocab].  precision as in dartree_params.
 * ws/ws_bytes: device scratch of dartree_project_workspace_size bytes
 * (256-byte aligned; may be NULL when that size is 0, else
 * DARTREE_ERR_WORKSPACE).  With bf16 and >= 512 rows the output tiles of a
 * last partial wave over the compute units are split along K and their
 * partial sums added in a fixed order, so the result is deterministic for a
 * given device (the split depends on its number of compute units). */
dartree_status dartree_project(int32_t precision, int32_t rows, int32_t vocab, int32_t hidden,
                               int32_t rows_per_group, const void* x, const void* U,
                               const float* bias, int64_t bias_stride, float* z,
                               void* ws, size_t ws_bytes, hipStream_t stream);

/* Row-wise log-softmax normaliser and top-k of z / tau (tau = T if T > 0 else 1):
 * lse[m] = log sum_v exp(z[m][v] / tau); cand_ids[m][0..k) are the k best ids
 * by (z desc, id asc) and cand_logp[m][i] = (z[m][id] - max_v z[m][v]) / tau
 * - log sum_v exp((z[m][v] - max) / tau).  z: fp32 [rows][vocab];
 * ws/ws_bytes: device scratch of dartree_lse_topk_workspace_size bytes
 * (may be NULL when that size is 0). */
dartree_status dartree_lse_topk_workspace_size(int32_t rows, int32_t vocab, int32_t k, size_t* bytes);
dartree_status dartree_lse_topk(const float* z, int32_t rows, int32_t vocab, int32_t k,
                                float temperature, float* lse, float* cand_logp,
                                int32_t* cand_ids, void* ws, size_t ws_bytes, hipStream_t stream);

/* dartree_lse_topk for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same kernels and results, with the row-segment records kept in a
 * static device array of the library, DARTREE_LSE_TOPK_STATIC_SCRATCH_BYTES
 * per GPU, held until the process ends.  That size covers every call
 * dartree_lse_topk_workspace_size accepts (a larger need would return
 * DARTREE_ERR_UNSUPPORTED).  The call allocates nothing and takes no
 * workspace; its first call on a device looks up the array's address there
 * (DARTREE_ERR_HIP if that fails).  Every call on one GPU shares the array:
 * calls that may overlap on one GPU (several streams, several host threads)
 * race and give undefined results; calls ordered on one stream do not. */
#define DARTREE_LSE_TOPK_STATIC_SCRATCH_BYTES (576 * 1024)
dartree_status dartree_lse_topk_noalloc(const float* z, int32_t rows, int32_t vocab, int32_t k,
                                        float temperature, float* lse, float* cand_logp, int32_t* cand_ids,
                                        hipStream_t stream);

/* Shared candidate sets (Alg. 1, C_d = TopK(L_d^base, K)) of `rows` rows of
 * fp32 logits [rows][vocab]: ids [rows][K] in (value desc, id asc) order,
 * 1 <= K <= min(vocab, DARTREE_MAX_CANDIDATES).  The workspace (size from
 * dartree_candidate_sets_workspace_size) holds per-row group maxima. */
dartree_status dartree_candidate_sets_workspace_size(int32_t rows, int32_t vocab, int32_t K, size_t* bytes);
dartree_status dartree_candidate_sets(const float* logits, int32_t rows, int32_t vocab, int32_t K, int32_t* ids,
                                      void* ws, size_t ws_bytes, hipStream_t stream);

/* Segmented top-W (Algorithm 1, the W best children of each request kept):
 * for each request q < batch, candidates (j, i) for parent j < n_parent and
 * rank i < k score s = (parent_score[q][j] + cand_logp[q*n_parent + j][i]) + beta
 * (parent_score may be NULL: every parent scores 0, the root); the first n_keep
 * by (s desc, j asc, token asc) are written in that order to out_tokens,
 * out_parents (j) and out_scores, each [batch][n_keep].
 * n_parent * k <= DARTREE_MAX_SORT and n_keep <= n_parent * k. */
dartree_status dartree_select_topw(int32_t batch, int32_t n_parent, int32_t k, int32_t n_keep,
                                   float depth_bonus, const float* parent_score,
                                   const float* cand_logp, const int32_t* cand_ids,
                                   int32_t* out_tokens, int32_t* out_parents, float* out_scores,
                                   hipStream_t stream);

/* Deferred top-B prune of a supertree given in the dartree_supertree level
 * layout (tokens, parents, scores: [L][b][W], level sizes from p).  Same
 * output as dartree_prune. */
dartree_status dartree_prune_levels(const dartree_params* p, const int32_t* tokens,
                                    const int32_t* parents, const float* scores,
                                    const dartree_tree* out, hipStream_t stream);

/* ---- the node-at-a-time baseline ------------------------------------------
 * Sequential correction with a best-first heap (Sec. 3.1; "Seq. Correction
 * w. Heap" of Table 2), the exact construction DARTree's depth-wise schedule
 * replaces.  Per request: the head is run on the root and its k best children
 * (by z desc, id asc) are candidates; then B times: pop the best candidate
 * prefix by (s desc, depth asc, parent's pop index asc, child rank asc), add
 * it to the tree and, if its depth is below L, run the head on it under its
 * own token history (r = bf16(tanh(t_parent + e U[token])), then t, a, z,
 * log q~ as in Algorithm 1's loop body, over the full vocabulary or over C_d
 * when candidates > 0) and make its k best children candidates.  The head
 * therefore runs once per pop, on one prefix per request at a time.  Scores,
 * precision, temperature and the shared sets follow dartree_params as above;
 * `width` is not used.  The popped prefixes (min(B, size of the k-capped
 * prefix tree) of them, prefix-closed) are emitted as dartree_tree.
 * B <= DARTREE_MAX_HEAP_BUDGET. */

/* Device destination of dartree_export_heap.  Slot i of request q is its i-th
 * popped prefix (slot 0: the root); step i ran the head on slot i.  Any
 * member may be NULL (not copied). */
typedef struct dartree_heap_trace {
  int32_t* tokens;     /* [b][B+1] token of slot i (-1 for the root) */
  int32_t* parents;    /* [b][B+1] slot of its parent (-1 for the root) */
  int32_t* depths;     /* [b][B+1] depth (0 for the root) */
  float* scores;       /* [b][B+1] s_beta (0 for the root) */
  int32_t* num_popped; /* [b] prefixes popped */
  float* lse;          /* [B][b] log sum_v exp(z_v / tau) of slot i's row (slots the head ran on) */
  float* cand_logp;    /* [B][b][k] log q~ of slot i's k best children, best first */
  int32_t* cand_ids;   /* [B][b][k] their token ids */
  void* states;        /* act [B+1][b][h] r of slot i (slots 1.. the head ran on) */
  int32_t* csets;      /* [b][L][K] shared candidate sets (candidates > 0 only) */
  void* features;      /* act [B][b][h] the feature row a of slot i (steps the head ran) */
} dartree_heap_trace;

/* Bytes of device workspace for dartree_build_tree_heap (host only). */
dartree_status dartree_heap_workspace_size(const dartree_params* p, size_t* bytes);

/* One round of the sequential heap for every request, enqueued on `stream`
 * as 4 launches per pop (3 with shared candidate sets, plus the sets once)
 * and one emission; no host synchronisation, so the round can be captured in
 * a graph.  ws: device, 256-byte aligned, >= dartree_heap_workspace_size. */
dartree_status dartree_build_tree_heap(const dartree_params* p, const dartree_inputs* in, void* ws,
                                       size_t ws_bytes, const dartree_tree* out, hipStream_t stream);

/* Copy the pops, the per-step children and states of the last
 * dartree_build_tree_heap on `ws` into the caller's buffers (for inspection). */
dartree_status dartree_export_heap(const dartree_params* p, const void* ws, size_t ws_bytes,
                                   const dartree_heap_trace* dst, hipStream_t stream);

/* ---- the consumer of the emitted tree ----------------------------------------
 * What the target model does with the tree (Sec. 2.1, Sec. 2.3, Sec. 4.1). */

/* Acceptance walk.  For request q (tree arrays as written by the builds
 * above: tokens, parents [b][B], num_nodes [b]), target [b][B+1] holds the
 * target's token after the verified context (index 0) and after the path of
 * node i (index i + 1): its greedy prediction at T = 0, its sample at T = 1
 * (exact target-sample matching).  From the root, move to the child whose
 * token equals the target's token at the current position; stop at the first
 * position without one.  Writes the output indices of the accepted nodes in
 * path order to accepted [b][max_len] (-1 after the last), their count to
 * num_accepted [b] (at most max_len), and the target's token at the last
 * accepted position to bonus [b]: the round advances num_accepted + 1 tokens.
 * 1 <= budget <= DARTREE_MAX_SORT; max_len >= 1 (a path has at most L nodes). */
dartree_status dartree_accept_walk(int32_t batch, int32_t budget, int32_t max_len, const int32_t* tokens,
                                   const int32_t* parents, const int32_t* num_nodes, const int32_t* target,
                                   int32_t* accepted, int32_t* num_accepted, int32_t* bonus, hipStream_t stream);

/* Shape of one tree-attention layer (grouped-query attention). */
typedef struct dartree_attn_params {
  int32_t batch;     /* b requests */
  int32_t budget;    /* B tree slots per request (the rows of the emitted tree) */
  int32_t max_ctx;   /* context positions held per request, 0 .. 261888 (1023 segments of 256) */
  int32_t heads_q;   /* query heads, a multiple of heads_kv */
  int32_t heads_kv;  /* key/value heads; query head h reads key/value head h / (heads_q / heads_kv) */
  int32_t head_dim;  /* 128 */
  float scale;       /* softmax scale (> 0), e.g. 1 / sqrt(head_dim) */
} dartree_attn_params;

/* Bytes of device workspace for dartree_tree_attention (host only).  With
 * fewer than 512 (request, key/value head, 64-query-row tile) blocks the
 * context is split into segments of 256 positions whose partial results are
 * merged (the workspace holds them); with 512 or more every block covers all
 * keys and the size is 0. */
dartree_status dartree_tree_attention_workspace_size(const dartree_attn_params* p, size_t* bytes);

/* One attention layer over the flattened trees (Sec. 2.3): the query of
 * node i attends to the first ctx_len[q] context positions (ctx_len NULL: all
 * max_ctx) and to the tree nodes j whose bit is set in mask row i (its
 * ancestors and itself, as emitted):
 *   out[q][i][h] = sum_j softmax_j(scale q[q][i][h] . k_j) v_j,
 * and a row that sees nothing is 0.  q: bf16 [b][B][heads_q][128];
 * k_ctx, v_ctx: bf16 [b][max_ctx][heads_kv][128] (may be NULL if max_ctx = 0);
 * k_tree, v_tree: bf16 [b][B][heads_kv][128], node i's own key and value;
 * mask: u64 [b][B][ceil(B/64)]; out: fp32 [b][B][heads_q][128].  bf16
 * products with fp32 accumulation; the softmax weights are rounded to bf16
 * for the weighted sum of values.  ws: device, 256-byte aligned, >=
 * dartree_tree_attention_workspace_size (per-segment partial results; may be
 * NULL when that size is 0). */
dartree_status dartree_tree_attention(const dartree_attn_params* p, const void* q, const void* k_ctx,
                                      const void* v_ctx, const void* k_tree, const void* v_tree,
                                      const uint64_t* mask, const int32_t* ctx_len, float* out, void* ws,
                                      size_t ws_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* DARTREE_H */
