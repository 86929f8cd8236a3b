// Selection and tree kernels of one round:
//  * select_topw  (Algorithm 1, "score each child ... retain the global top-W"):
//    per request, the n_parent * k candidates get s = (s_parent + log q~) + beta
//    (eq. (5) one depth at a time) and the best n_keep by
//    (s desc, parent slot asc, token asc) become S_d, in that order.
//  * state_update (Algorithm 1, "update their states"): r = act(tanh(t_parent
//    + e U[token])) for every kept child.
//  * prune_emit   (Sec. 3.3, deferred best-first pruning): top-B of the whole
//    supertree by (s desc, depth asc, slot asc) - prefix-closed by Lemma 1 -
//    flattened in canonical breadth-first order (depth, parent's output index,
//    token) with parent indices and the ancestor-or-self mask.
// Every selection packs its order into one 64-bit key (score mapped to an
// ascending key in the high word, the tie-break fields in the low word) and
// sorts the keys with a bitonic network in LDS, one block per request, so the
// result does not depend on thread timing.
#include <float.h>

#include "internal.hpp"

namespace dartree {
namespace {

constexpr int kSortMax = DARTREE_MAX_SORT;

__device__ void bitonic_sort(uint64_t* keys, int npad) {
  for (int size = 2; size <= npad; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = threadIdx.x; i < npad; i += blockDim.x) {
        const int j = i ^ stride;
        if (j > i) {
          const uint64_t a = keys[i], b = keys[j];
          const bool up = (i & size) == 0;
          if ((a > b) == up) { keys[i] = b; keys[j] = a; }
        }
      }
      __syncthreads();
    }
  }
}

__device__ __forceinline__ int next_pow2(int n) {
  int p = 2;
  while (p < n) p <<= 1;
  return p;
}

// grid: batch.  Low key word: parent slot (12 bits) << 20 | token (20 bits).
__global__ __launch_bounds__(1024) void select_topw(int n_parent, int k, int n_keep, float beta,
                                                    int parent_stride, int out_stride,
                                                    const float* __restrict__ parent_score,
                                                    const float* __restrict__ cand_logp,
                                                    const int32_t* __restrict__ cand_ids, int32_t* out_tok,
                                                    int32_t* out_par, float* out_score) {
  __shared__ uint64_t keys[kSortMax];
  const int q = blockIdx.x;
  const int n = n_parent * k;
  const int npad = next_pow2(n);
  const int64_t rbase = int64_t(q) * n_parent;
  for (int c = threadIdx.x; c < npad; c += blockDim.x) {
    uint64_t key = ~0ull;
    if (c < n) {
      const int j = c / k;
      const float sp = parent_score ? parent_score[int64_t(q) * parent_stride + j] : 0.f;
      const float s = (sp + cand_logp[rbase * k + c]) + beta;
      const uint32_t lo = (uint32_t(j) << 20) | uint32_t(cand_ids[rbase * k + c]);
      key = (uint64_t(score_desc_key(s)) << 32) | lo;
    }
    keys[c] = key;
  }
  __syncthreads();
  bitonic_sort(keys, npad);
  for (int i = threadIdx.x; i < n_keep; i += blockDim.x) {
    const uint64_t key = keys[i];
    const uint32_t lo = uint32_t(key);
    const int64_t o = int64_t(q) * out_stride + i;
    out_tok[o] = int32_t(lo & 0xFFFFFu);
    out_par[o] = int32_t(lo >> 20);
    out_score[o] = score_from_desc_key(uint32_t(key >> 32));
  }
}

// grid: batch * n_child rows.  Child row c = q * n_child + i is level entry
// q * lvl_stride + i; its parent row is q * n_parent + (its parent slot).
template <bool BF16>
__global__ __launch_bounds__(256) void state_update(int n_child, int n_parent, int hidden, int lvl_stride,
                                                    const int32_t* __restrict__ lvl_tok,
                                                    const int32_t* __restrict__ lvl_par,
                                                    const float* __restrict__ t, const void* __restrict__ U,
                                                    float e, void* r_out) {
  const int64_t c = blockIdx.x;
  const int64_t q = c / n_child;
  const int64_t li = q * lvl_stride + (c - q * n_child);
  const int64_t prow = q * n_parent + lvl_par[li];
  const int64_t tok = lvl_tok[li];
  const float* tp = t + prow * hidden;
  if constexpr (BF16) {
    const uint16_t* up = static_cast<const uint16_t*>(U) + tok * hidden;
    uint16_t* rp = static_cast<uint16_t*>(r_out) + c * hidden;
    for (int i = threadIdx.x * 8; i < hidden; i += blockDim.x * 8) {
      const f32x4 t0 = *reinterpret_cast<const f32x4*>(tp + i);
      const f32x4 t1 = *reinterpret_cast<const f32x4*>(tp + i + 4);
      typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
      const u16x8 u = *reinterpret_cast<const u16x8*>(up + i);
      u16x8 r;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        r[j] = f32_to_bf16(tanhf(t0[j] + e * bf16_to_f32(u[j])));
        r[j + 4] = f32_to_bf16(tanhf(t1[j] + e * bf16_to_f32(u[j + 4])));
      }
      *reinterpret_cast<u16x8*>(rp + i) = r;
    }
  } else {
    const float* up = static_cast<const float*>(U) + tok * hidden;
    float* rp = static_cast<float*>(r_out) + c * hidden;
    for (int i = threadIdx.x; i < hidden; i += blockDim.x) rp[i] = tanhf(tp[i] + e * up[i]);
  }
}

// grid: batch.  Level arrays are [L][batch][W]; node g of request q is slot
// g - off[d-1] of depth d.  Low key word of the prune: depth << 16 | slot.
__global__ __launch_bounds__(1024) void prune_emit(LevelShape shape, int budget, int batch,
                                                   const int32_t* __restrict__ lvl_tok,
                                                   const int32_t* __restrict__ lvl_par,
                                                   const float* __restrict__ lvl_score, dartree_tree out) {
  __shared__ uint64_t keys[kSortMax];
  __shared__ int32_t out_idx[kSortMax];   // per supertree node: output index, -1 if pruned
  __shared__ int32_t par_out[kSortMax];   // per output index: parent's output index
  __shared__ uint32_t rank_key[DARTREE_MAX_WIDTH];
  __shared__ int32_t kept_at_depth;

  const int q = blockIdx.x;
  const int L = shape.depth, W = shape.width;
  const int total = shape.off[L];
  const int n_out = min(budget, total);
  const int words = (budget + 63) / 64;
  const int npad = next_pow2(total);
  auto lvl_index = [&](int d, int slot) { return (int64_t(d - 1) * batch + q) * W + slot; };
  // supertree node index of the parent of level entry li at depth d >= 2
  // (slots outside S_{d-1} are clamped: malformed levels cannot index out of bounds)
  auto parent_node = [&](int d, int64_t li) {
    const int ps = min(max(lvl_par[li], 0), shape.n[d - 2] - 1);
    return shape.off[d - 2] + ps;
  };

  // 1. top-B of the supertree
  for (int g = threadIdx.x; g < npad; g += blockDim.x) {
    uint64_t key = ~0ull;
    if (g < total) {
      int d = 1;
      while (g >= shape.off[d]) ++d;
      const int slot = g - shape.off[d - 1];
      key = (uint64_t(score_desc_key(lvl_score[lvl_index(d, slot)])) << 32) |
            (uint32_t(d) << 16) | uint32_t(slot);
    }
    keys[g] = key;
    if (g < total) out_idx[g] = -1;
    if (g < kSortMax) par_out[g] = -1;
  }
  __syncthreads();
  bitonic_sort(keys, npad);
  for (int i = threadIdx.x; i < n_out; i += blockDim.x) {
    const uint32_t lo = uint32_t(keys[i]);
    const int d = int(lo >> 16), slot = int(lo & 0xFFFFu);
    out_idx[shape.off[d - 1] + slot] = 0;  // mark kept
  }
  __syncthreads();

  // 2. canonical order, one depth at a time: rank kept nodes of depth d by
  //    (parent's output index, token); siblings have distinct tokens.
  int base = 0;
  for (int d = 1; d <= L; ++d) {
    const int nd = shape.n[d - 1], od = shape.off[d - 1];
    if (threadIdx.x == 0) kept_at_depth = 0;
    for (int i = threadIdx.x; i < nd; i += blockDim.x) {
      uint32_t rk = ~0u;
      if (out_idx[od + i] >= 0) {
        const int64_t li = lvl_index(d, i);
        const uint32_t pidx = d == 1 ? 0u : uint32_t(out_idx[parent_node(d, li)]);
        rk = (pidx << 20) | (uint32_t(lvl_tok[li]) & 0xFFFFFu);
      }
      rank_key[i] = rk;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < nd; i += blockDim.x) {
      const uint32_t mine = rank_key[i];
      if (mine == ~0u) continue;
      int r = 0;
      for (int j = 0; j < nd; ++j) r += (rank_key[j] < mine) | ((rank_key[j] == mine) & (j < i));
      out_idx[od + i] = base + r;
      const int64_t li = lvl_index(d, i);
      par_out[base + r] = d == 1 ? -1 : out_idx[parent_node(d, li)];
      atomicAdd(&kept_at_depth, 1);
    }
    __syncthreads();
    base += kept_at_depth;
    __syncthreads();
  }

  // 3. emit node arrays (pad slots past n_out)
  const int64_t ob = int64_t(q) * budget;
  for (int o = threadIdx.x; o < budget; o += blockDim.x) {
    if (o >= n_out) {
      out.tokens[ob + o] = -1;
      out.parents[ob + o] = -1;
      out.depths[ob + o] = 0;
      out.scores[ob + o] = -INFINITY;
    }
  }
  for (int d = 1; d <= L; ++d) {
    const int nd = shape.n[d - 1], od = shape.off[d - 1];
    for (int i = threadIdx.x; i < nd; i += blockDim.x) {
      const int o = out_idx[od + i];
      if (o < 0) continue;
      const int64_t li = lvl_index(d, i);
      out.tokens[ob + o] = lvl_tok[li];
      out.parents[ob + o] = par_out[o];
      out.depths[ob + o] = d;
      out.scores[ob + o] = lvl_score[li];
    }
  }
  // 4. ancestor-or-self mask, one 64-bit word per thread
  const int64_t mb = int64_t(q) * budget * words;
  for (int w = threadIdx.x; w < budget * words; w += blockDim.x) {
    const int o = w / words, word = w % words;
    uint64_t bits = 0;
    if (o < n_out) {
      // parents precede children in the output order, so the walk strictly
      // decreases and ends at -1 after at most L steps
      for (int j = o; j >= 0;) {
        if (j / 64 == word) bits |= 1ull << (j % 64);
        const int nx = par_out[j];
        j = nx < j ? nx : -1;
      }
    }
    out.mask[mb + w] = bits;
  }
  if (threadIdx.x == 0) out.num_nodes[q] = n_out;
}

}  // namespace

hipError_t launch_select_topw(int batch, int n_parent, int k, int n_keep, float beta, int parent_stride,
                              int out_stride, const float* parent_score, const float* cand_logp,
                              const int32_t* cand_ids, int32_t* out_tok, int32_t* out_par, float* out_score,
                              hipStream_t s) {
  if (batch <= 0) return hipSuccess;
  const int n = n_parent * k;
  const int threads = n >= 1024 ? 1024 : (n >= 256 ? 256 : 64);
  hipLaunchKernelGGL(select_topw, dim3(batch), dim3(threads), 0, s, n_parent, k, n_keep, beta, parent_stride,
                     out_stride, parent_score,
                     cand_logp, cand_ids, out_tok, out_par, out_score);
  return hipGetLastError();
}

hipError_t launch_state_update(int precision, int batch, int n_child, int n_parent, int hidden, int lvl_stride,
                               const int32_t* lvl_tok, const int32_t* lvl_par, const float* t, const void* U,
                               float e, void* r_out, hipStream_t s) {
  const unsigned rows = unsigned(batch) * unsigned(n_child);
  if (rows == 0) return hipSuccess;
  if (precision == DARTREE_BF16)
    hipLaunchKernelGGL((state_update<true>), dim3(rows), dim3(256), 0, s, n_child, n_parent, hidden, lvl_stride, lvl_tok,
                       lvl_par, t, U, e, r_out);
  else
    hipLaunchKernelGGL((state_update<false>), dim3(rows), dim3(256), 0, s, n_child, n_parent, hidden, lvl_stride, lvl_tok,
                       lvl_par, t, U, e, r_out);
  return hipGetLastError();
}

hipError_t launch_prune_emit(int batch, const LevelShape& shape, int budget, const int32_t* lvl_tok,
                             const int32_t* lvl_par, const float* lvl_score, const dartree_tree& out,
                             hipStream_t s) {
  if (batch <= 0) return hipSuccess;
  hipLaunchKernelGGL(prune_emit, dim3(batch), dim3(1024), 0, s, shape, budget, batch, lvl_tok, lvl_par,
                     lvl_score, out);
  return hipGetLastError();
}

}  // namespace dartree
