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
// m / rows_per_group, whose bias row starts at bias + group * bias_stride.
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
  float* out;            // fp32 [M][N]
  void* act_out;         // EPI_HEAD: act [M][N]
};
hipError_t launch_project(const ProjArgs& a, hipStream_t s);

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
  int precision, hidden;
  const float* t;                 // [rows][hidden]
  const void* U;                  // act [V][hidden]
  float e;
  void* r_out;                    // act [batch * n_keep][hidden]
};
hipError_t launch_select_level(const LevelArgs& a, hipStream_t s);

// Shared candidate sets C = TopK(logits row, K) of `rows` fp32 rows, ids in
// (value desc, id asc) order; scratch holds the per-chunk winners.
size_t candidate_sets_scratch_bytes(int64_t rows, int64_t vocab, int K);
bool candidate_sets_supported(int64_t vocab, int K);
hipError_t launch_candidate_sets(const float* logits, int64_t rows, int64_t vocab, int K, int32_t* ids,
                                 void* scratch, hipStream_t s);

// Corrected logits over the shared set: z[q*np + j][c] = lb[q*lb_stride + C[c]]
// + U[C[c]] . a[q*np + j], with C = cset + q * cset_stride.
hipError_t launch_shared_logits(int precision, int batch, int np, int K, int hidden, const void* a, const void* U,
                                const float* lb, int64_t lb_stride, const int32_t* cset, int64_t cset_stride,
                                float* z, hipStream_t s);

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

}  // namespace dartree
