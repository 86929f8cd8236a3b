// Internal declarations shared by the libdartree kernels and the C ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dartree.h"

namespace dartree {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// bfloat16 <-> fp32 on raw 16-bit patterns (finite values; nearest-even).
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}

// Order-preserving map of an fp32 score to a key that sorts ascending for
// descending scores (-0 and +0 are the same score).
__device__ __forceinline__ uint32_t score_desc_key(float s) {
  uint32_t u = __float_as_uint(s + 0.0f);
  uint32_t asc = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ~asc;
}
__device__ __forceinline__ float score_from_desc_key(uint32_t k) {
  uint32_t asc = ~k;
  uint32_t u = (asc & 0x80000000u) ? (asc & 0x7FFFFFFFu) : ~asc;
  return __uint_as_float(u);
}

// ---------------------------------------------------------------------------
// Launchers (host side).  They assume validated arguments.
// ---------------------------------------------------------------------------

// out[m][n] = epilogue(bias, sum_k x[m][k] * w[n][k]); row m belongs to group
// g = m / rows_per_group, whose bias row starts at bias + row(g) * bias_stride
// with row(g) = group_index[g] (device memory) if group_index is set, else g.
enum ProjEpilogue {
  EPI_LOGITS = 0,  // out (fp32) = acc + bias_f32
  EPI_HEAD = 1     // out (fp32) = acc ; act_out = act(tanh(acc + bias_act))
};

struct ProjArgs {
  int precision;
  int epilogue;
  int64_t M, N, K;
  int64_t rows_per_group;
  const void* x;         // act [M][K]
  const void* w;         // act [N][K]
  const float* bias_f32; // EPI_LOGITS
  const void* bias_act;  // EPI_HEAD
  int64_t bias_stride;   // elements between consecutive group bias rows
  const int32_t* group_index;  // optional device [M / rows_per_group]: bias row of each group
  float* out;            // fp32 [M][N]
  void* act_out;         // EPI_HEAD: act [M][N]
  float* split;          // optional device scratch of proj_split_bytes(...) bytes: partial sums of
                         // tiles split along K (without it no tile is split)
};
hipError_t launch_project(const ProjArgs& a, hipStream_t s);
// Scratch the product of this shape can use to split tiles along K (0 if none).
size_t proj_split_bytes(int precision, int epilogue, int64_t M, int64_t N, int64_t K);

// Row-wise online log-sum-exp and top-k (K3).  Rows are split into
// lse_topk_segments(rows, vocab) segments; with more than one, each segment
// leaves a record in scratch (lse_topk_scratch_bytes) and, if `merge`, a
// second kernel merges them into lse / cand_logp / cand_ids.  Without
// `merge` the records are left for launch_select_level.
int lse_topk_segments(int64_t rows, int64_t vocab);
size_t lse_topk_scratch_bytes(int64_t rows, int64_t vocab, int k);
hipError_t launch_lse_topk(const float* z, int64_t rows, int64_t vocab, int k, float tau,
                           float* lse, float* cand_logp, int32_t* cand_ids, void* scratch,
                           bool merge, hipStream_t s);

// One depth's selection (K4) with the K3 segment merge and the K5 state
// update.  Rows of request q are q * n_parent .. q * n_parent + n_parent - 1.
struct LevelArgs {
  int batch, n_parent, k, n_keep;
  float beta, tau;
  int parent_stride, out_stride;  // level entries of request q start at q * stride
  const float* parent_score;      // NULL: all zero (depth 1)
  int nseg;                       // > 1: merge the records in `part` and store lse / cand_*
  const float* part;
  float* lse;
  float* cand_logp;               // [rows][k]; read when nseg == 1
  int32_t* cand_ids;
  int32_t* out_tok;
  int32_t* out_par;
  float* out_score;
  int rows_ranked;                // each row's candidates are in rank order (only the first
                                  // min(k, n_keep) of a row can be kept)
  int shared_k;                   // K > 0: candidates from logits over the shared set C_d
  const float* zsh;               // [rows][K] corrected logits over C_d (shared_k > 0)
  const int32_t* cset;            // request q's C_d at cset + q * cset_stride
  int64_t cset_stride;
  int state;                      // 0: no state update
  int precision, hidden, vocab;
  int markov;                     // state = act(e U[token]) (Markov head), else act(tanh(t + e U[token]))
  const float* t;                 // [rows][hidden]
  const void* U;                  // act [V][hidden]
  float e;
  void* r_out;                    // act [batch * n_keep][hidden]
  uint32_t* stamp;                // optional: block 0 writes {key_lo, key_hi, depth} (the order check)
  uint32_t stamp_key_lo, stamp_key_hi;
  int stamp_depth;
};
hipError_t launch_select_level(const LevelArgs& a, hipStream_t s);
// Waves of one select_level block for branching factor k: a block merges the
// segment records of its request's parent rows one row per wave.
int select_level_waves(int k);

// Shared candidate sets C = TopK(logits row, K) of `rows` fp32 rows, ids in
// (value desc, id asc) order; scratch holds the per-chunk winners.
size_t candidate_sets_scratch_bytes(int64_t rows, int64_t vocab, int K);
bool candidate_sets_supported(int64_t vocab, int K);
hipError_t launch_candidate_sets(const float* logits, int64_t rows, int64_t vocab, int K, int32_t* ids,
                                 void* scratch, hipStream_t s);

// Corrected logits over the shared set: z[q*np + j][c] = lb[g*lb_stride + C[c]]
// + U[C[c]] . a[q*np + j], with C = cset + g * cset_stride and g =
// group_index[q] (device memory) if group_index is set, else q.
// Set ids are clamped into [0, vocab).
hipError_t launch_shared_logits(int precision, int batch, int np, int K, int hidden, int vocab, const void* a,
                                const void* U, const float* lb, int64_t lb_stride, const int32_t* cset,
                                int64_t cset_stride, const int32_t* group_index, float* z, hipStream_t s);

// Deferred top-B prune and tree emission (K6).
struct LevelShape {
  int32_t depth;
  int32_t width;
  int32_t n[DARTREE_MAX_DEPTH];     // n_d, d = 1..L at index d-1
  int32_t off[DARTREE_MAX_DEPTH + 1];  // prefix sums of n
};
hipError_t launch_prune_emit(int batch, const LevelShape& shape, int budget,
                             const int32_t* lvl_tok, const int32_t* lvl_par,
                             const float* lvl_score, const dartree_tree& out, hipStream_t s);

// Sequential correction with a best-first heap (the node-at-a-time
// construction of Sec. 3.1): one step per pop, after the head, logits and
// softmax pass of the node popped at the previous step (rows: one per
// request).  Slot i of request q is the i-th popped prefix (slot 0 = the
// root); per-slot arrays are [batch][budget + 1], per-step arrays
// [budget][batch][...] (step i expands slot i).
struct HeapArgs {
  int batch, budget, depth, k, vocab;
  int markov;                   // state = act(e U[token]) (Markov head)
  int shared_k;                 // K > 0: the step's row holds logits over C_d in zsh
  float beta, tau, e;
  int precision, hidden;
  int step;
  int nseg;                     // > 1: merge the row records in `part`
  const float* part;
  const float* zsh;             // [batch][K]
  const int32_t* cset;          // [batch][depth][K]
  int32_t* slot_tok;
  int32_t* slot_par;
  int32_t* slot_depth;
  float* slot_score;
  int32_t* slot_next;           // rank of the slot's next child not yet popped
  int32_t* slot_nch;            // number of children the slot was given
  uint64_t* cand_key;           // heap key of the slot's next child (~0: none)
  float* ch_lse;                // [budget][batch]
  float* ch_lp;                 // [budget][batch][k], children in rank order
  int32_t* ch_tok;
  int32_t* n_pop;               // [batch] prefixes popped so far
  int32_t* group_index;         // [batch] H / L^base / C_d row of the next expansion
  const float* t_store;         // [budget][batch][hidden]: t of slot i
  const void* U;
  void* r_store;                // act [budget + 1][batch][hidden]: r of slot i
};
hipError_t launch_heap_step(const HeapArgs& a, hipStream_t s);

// The consumer of the emitted tree: the acceptance walk, and one tree-attention
// layer (head_dim 128) in key segments merged by a second kernel.  Partial
// results per segment s, request q, key/value head h and query row r (r =
// node * group + query head within the group) live at index
// ((s * batch + q) * heads_kv + h) * rows_pad + r of part_o ([..][128]) and
// part_ml ([..][2]: running max in log2 units, sum).
hipError_t launch_accept_walk(int batch, int budget, int max_len, const int32_t* tokens, const int32_t* parents,
                              const int32_t* num_nodes, const int32_t* target, int32_t* accepted,
                              int32_t* n_accepted, int32_t* bonus, hipStream_t s);
struct AttnArgs {
  int batch, budget, max_ctx, heads_q, heads_kv, group;
  int nseg_ctx, seg_len, rows_pad;
  float scale_log2;             // softmax scale * log2(e)
  const uint16_t* q;            // bf16 [batch][budget][heads_q][128]
  const uint16_t* k_ctx;        // bf16 [batch][max_ctx][heads_kv][128]
  const uint16_t* v_ctx;
  const uint16_t* k_tree;       // bf16 [batch][budget][heads_kv][128]
  const uint16_t* v_tree;
  const uint64_t* mask;         // [batch][budget][ceil(budget / 64)]
  const int32_t* ctx_len;       // [batch] or NULL (max_ctx)
  float* part_o;
  float* part_ml;
  float* out;                   // fp32 [batch][budget][heads_q][128]
};
int attention_segment_len();
int attention_max_segments();   // limit of context segments + 1
// true when one block per (request, key/value head, 64-row tile) covers all
// keys (enough blocks for the chip): no partial results, no merge
bool attention_fused(int batch, int budget, int heads_q, int heads_kv);
hipError_t launch_tree_attention(const AttnArgs& a, hipStream_t s);
hipError_t launch_heap_emit(const HeapArgs& a, const dartree_tree& out, hipStream_t s);

}  // namespace dartree
