// Selection and tree kernels of one round:
//  * select_level (Algorithm 1, scoring the children, keeping the global
//    top-W and updating their states): per request, the n_parent * k
//    candidates get s = (s_parent + log q~) + beta (eq. (5) one depth at a
//    time), the best n_keep by (s desc, parent slot asc, token asc) become
//    S_d in that order, and every kept child gets r = act(tanh(t_parent +
//    e U[token])).  The kernel also finishes the softmax pass when that pass
//    split its rows into segments.
//  * prune_emit   (Sec. 3.3, deferred best-first pruning): top-B of the whole
//    supertree by (s desc, depth asc, slot asc) - prefix-closed by Lemma 1 -
//    flattened in canonical breadth-first order (depth, parent's output index,
//    token) with parent indices and the ancestor-or-self mask.
// Every selection packs its order into one 64-bit key (score mapped to an
// ascending key in the high word, the tie-break fields in the low word) and
// sorts the keys with a bitonic network in LDS, one block per request, so the
// result does not depend on thread timing.
#include <float.h>

#include <algorithm>

#include "reduce.hpp"

namespace dartree {
namespace {

constexpr int kSortMax = DARTREE_MAX_SORT;

// grid: batch * S, block (q, sl): request q, state slice sl.  Three steps of
// one depth in one launch:
//  1. the candidate log-probabilities of request q's parent rows: read as
//     written by the softmax pass, or merged here from its per-segment
//     records, or (shared candidate set) computed here from the row's logits
//     over C_d (one wave per row; block 0 of the request also stores them);
//  2. s = (s_parent + log q~) + beta for every candidate and the best n_keep
//     by (s desc, parent slot asc, token asc), from one bitonic sort of 64-bit
//     keys (low word: parent slot (12 bits) << 20 | token (20 bits)); block 0
//     of the request writes the level;
//  3. the states r = act(tanh(t_parent + e U[token])) of kept children sl,
//     sl + S, ... (child i of request q is row q * n_keep + i).
// Steps 1-2 run in each of the S blocks of a request, which then need no
// further synchronisation.
template <int K>
constexpr int select_threads() { return K >= 32 ? 256 : K >= 16 ? 512 : 1024; }  // registers per lane for wide lists

template <int K>
__global__ __launch_bounds__(select_threads<K>()) void select_level(LevelArgs a, int S) {
  __shared__ uint64_t keys[kSortMax];
  __shared__ float c_logp[kSortMax];
  __shared__ int32_t c_ids[kSortMax];
  __shared__ float ps[kSortMax];   // parent scores (n_parent <= n_parent k <= kSortMax), fetched early
  const int q = blockIdx.x / S, sl = blockIdx.x - q * S;
  const int np = a.n_parent, k = a.k;
  int n = np * k;
  const int64_t rbase = int64_t(q) * np;
  if (a.stamp && blockIdx.x == 0 && threadIdx.x == 0) {   // the workspace's depth record
    a.stamp[0] = a.stamp_key_lo;
    a.stamp[1] = a.stamp_key_hi;
    a.stamp[2] = uint32_t(a.stamp_depth);
  }
  for (int j = threadIdx.x; j < np; j += blockDim.x)
    ps[j] = a.parent_score ? a.parent_score[int64_t(q) * a.parent_stride + j] : 0.f;
  if (a.shared_k > 0) {
    // shared candidate set: row j's K corrected logits over C_d -> log q~
    // normalised over C_d, and its k best by (z desc, id asc), ranked by
    // counting over the row (staged in this wave's LDS row)
    __shared__ __attribute__((aligned(16))) float rz[16][DARTREE_MAX_CANDIDATES];
    __shared__ __attribute__((aligned(16))) int32_t rid[16][DARTREE_MAX_CANDIDATES];
    const int nk = a.shared_k;
    const float scale = kLog2e / a.tau;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), nwaves = blockDim.x >> 6;
    const int32_t* set = a.cset + q * a.cset_stride;
    for (int j = wave; j < np; j += nwaves) {
      const float* zr = a.zsh + (rbase + j) * nk;
      float m = -INFINITY;
      for (int c = lane; c < nk; c += 64) {
        const float v = zr[c];
        rz[wave][c] = v;
        rid[wave][c] = min(max(set[c], 0), a.vocab - 1);   // workspace ids, clamped into U
        m = fmaxf(m, v);
      }
      m = wave_max(m);
      float sum = 0.f;
      for (int c = lane; c < nk; c += 64) sum += __builtin_amdgcn_exp2f((rz[wave][c] - m) * scale);
      const float log_s = logf(wave_sum(sum));
      __builtin_amdgcn_wave_barrier();
      for (int c = lane; c < nk; c += 64) {
        const float v = rz[wave][c];
        const int id = rid[wave][c];
        // 16-byte reads of four values and four ids at a time (every lane
        // reads the same address), then the tail
        typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
        const f32x4* rz4 = reinterpret_cast<const f32x4*>(rz[wave]);
        const i32x4* rid4 = reinterpret_cast<const i32x4*>(rid[wave]);
        const int nk4 = nk & ~3;
        int rank = 0;
#pragma unroll 4
        for (int o = 0; o < nk4; o += 4) {
          const f32x4 zv = rz4[o >> 2];
          const i32x4 iv = rid4[o >> 2];
          rank += int(better(zv[0], iv[0], v, id)) + int(better(zv[1], iv[1], v, id)) +
                  int(better(zv[2], iv[2], v, id)) + int(better(zv[3], iv[3], v, id));
        }
        for (int o = nk4; o < nk; ++o) rank += int(better(rz[wave][o], rid[wave][o], v, id));
        if (rank < k) {
          const float lp = (v - m) / a.tau - log_s;
          c_logp[j * k + rank] = lp;
          c_ids[j * k + rank] = id;
          if (sl == 0) {
            a.cand_logp[(rbase + j) * k + rank] = lp;
            a.cand_ids[(rbase + j) * k + rank] = id;
          }
        }
      }
      if (sl == 0 && lane == 0) a.lse[rbase + j] = m / a.tau + log_s;
      __builtin_amdgcn_wave_barrier();   // the LDS row is rewritten for the next row
    }
  } else if (a.nseg > 1) {
    constexpr int RF = record_floats<K>();
    const float scale = kLog2e / a.tau;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), nwaves = blockDim.x >> 6;
    for (int j = wave; j < np; j += nwaves) {
      uint64_t out[K];
      const Partial p = wave_merge_records<K>(a.part + (rbase + j) * a.nseg * RF, a.nseg, k, scale, out);
      const float log_s = logf(p.s);
#pragma unroll
      for (int r = 0; r < K; ++r) {
        if (r < k && lane == r) {
          const float lp = (key_value(out[r]) - p.m) / a.tau - log_s;
          const int id = key_id(out[r]);
          c_logp[j * k + r] = lp;
          c_ids[j * k + r] = id;
          if (sl == 0) {
            a.cand_logp[(rbase + j) * k + r] = lp;
            a.cand_ids[(rbase + j) * k + r] = id;
          }
        }
      }
      if (sl == 0 && lane == 0) a.lse[rbase + j] = p.m / a.tau + log_s;
    }
  } else {
    for (int c = threadIdx.x; c < n; c += blockDim.x) {
      c_logp[c] = a.cand_logp[rbase * k + c];
      c_ids[c] = a.cand_ids[rbase * k + c];
    }
  }
  __syncthreads();
  auto score_at = [&](int j, int r) {   // s of row j's candidate r, as in the keys below
    return (ps[j] + c_logp[j * k + r]) + a.beta;
  };
  // With rows in rank order, a row's candidates from position n_keep on have
  // scores <= its candidate n_keep's; if that is strictly below its candidate
  // n_keep - 1's in every row, each of them is beaten by n_keep children of its
  // own parent and can never be kept, so only the first n_keep of each row
  // compete.  (Equal fp32 scores order by token, not by rank, so a row with
  // such a tie keeps every candidate in play.)
  int kk = k;
  if (a.rows_ranked && a.n_keep < k) {
    __shared__ int tie;
    if (threadIdx.x == 0) tie = 0;
    __syncthreads();
    for (int j = threadIdx.x; j < np; j += blockDim.x)
      if (!(score_at(j, a.n_keep - 1) > score_at(j, a.n_keep))) tie = 1;
    __syncthreads();
    if (!tie) kk = a.n_keep;
  }
  n = np * kk;
  auto key_of = [&](int c) {
    const int j = c / kk;
    const int r = c - j * kk;
    const float sc = score_at(j, r);
    // ids < 2^20; the mask keeps a malformed id out of the parent-slot field
    return (uint64_t(score_desc_key(sc)) << 32) | (uint32_t(j) << 20) | (uint32_t(c_ids[j * k + r]) & 0xFFFFFu);
  };
  const uint64_t* kept = keys;   // the n_keep best, in order
  if (n <= int(blockDim.x)) {
    // few candidates: rank by counting (keys are distinct: (slot, token)
    // pairs are), one barrier instead of a sorting network
    uint64_t mine = ~0ull;
    if (int(threadIdx.x) < n) mine = key_of(threadIdx.x);
    keys[threadIdx.x] = mine;
    __syncthreads();
    int rank = 0;
    if (int(threadIdx.x) < n) {
      // 16-byte reads of key pairs, unrolled so that the reads overlap
      typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));
      const u64x2* kp = reinterpret_cast<const u64x2*>(keys);
      const int n2 = n >> 1;
#pragma unroll 8
      for (int j = 0; j < n2; ++j) {
        const u64x2 kk = kp[j];
        rank += int(kk.x < mine) + int(kk.y < mine);
      }
      if (n & 1) rank += int(keys[n - 1] < mine);
    }
    __syncthreads();
    // n <= 1024 and n_keep <= n: the ranked copy sits above the keys
    if (int(threadIdx.x) < n && rank < a.n_keep) keys[kSortMax / 2 + rank] = mine;
    kept = keys + kSortMax / 2;
    __syncthreads();
  } else {
    const int npad = next_pow2(n);
    for (int c = threadIdx.x; c < npad; c += blockDim.x) keys[c] = c < n ? key_of(c) : ~0ull;
    __syncthreads();
    bitonic_sort(keys, npad);
  }
  if (sl == 0) {
    for (int i = threadIdx.x; i < a.n_keep; i += blockDim.x) {
      const uint64_t key = kept[i];
      const uint32_t lo = uint32_t(key);
      const int64_t o = int64_t(q) * a.out_stride + i;
      a.out_tok[o] = int32_t(lo & 0xFFFFFu);
      a.out_par[o] = int32_t(lo >> 20);
      a.out_score[o] = score_from_desc_key(uint32_t(key >> 32));
    }
  }
  if (!a.state) return;
  const int h = a.hidden;
  for (int i = sl; i < a.n_keep; i += S) {
    const uint32_t lo = uint32_t(kept[i]);
    // an empty candidate (a row without finite values) is clamped into U
    const int64_t prow = rbase + (lo >> 20), tok = min(int(lo & 0xFFFFFu), a.vocab - 1);
    const int64_t c = int64_t(q) * a.n_keep + i;
    const float* tp = a.t + prow * h;
    if (a.precision == DARTREE_BF16) {
      typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
      const uint16_t* up = static_cast<const uint16_t*>(a.U) + tok * h;
      uint16_t* rp = static_cast<uint16_t*>(a.r_out) + c * h;
      for (int x = threadIdx.x * 8; x < h; x += blockDim.x * 8) {
        const f32x4 t0 = *reinterpret_cast<const f32x4*>(tp + x);
        const f32x4 t1 = *reinterpret_cast<const f32x4*>(tp + x + 4);
        const u16x8 u = *reinterpret_cast<const u16x8*>(up + x);
        u16x8 r;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float e0 = a.e * bf16_to_f32(u[j]), e1 = a.e * bf16_to_f32(u[j + 4]);
          r[j] = f32_to_bf16(a.markov ? e0 : tanhf(t0[j] + e0));
          r[j + 4] = f32_to_bf16(a.markov ? e1 : tanhf(t1[j] + e1));
        }
        *reinterpret_cast<u16x8*>(rp + x) = r;
      }
    } else {
      const float* up = static_cast<const float*>(a.U) + tok * h;
      float* rp = static_cast<float*>(a.r_out) + c * h;
      for (int x = threadIdx.x; x < h; x += blockDim.x) rp[x] = a.markov ? a.e * up[x] : tanhf(tp[x] + a.e * up[x]);
    }
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
  // per supertree node, staged once: token, parent slot, score
  __shared__ int32_t s_tok[kSortMax], s_par[kSortMax];
  __shared__ float s_score[kSortMax];
  __shared__ __attribute__((aligned(16))) uint32_t rank_key[DARTREE_MAX_WIDTH];
  __shared__ int32_t kept_at_depth;

  const int q = blockIdx.x;
  const int L = shape.depth, W = shape.width;
  const int total = shape.off[L];
  const int n_out = min(budget, total);
  const int words = (budget + 63) / 64;
  const int npad = next_pow2(total);
  auto lvl_index = [&](int d, int slot) { return (int64_t(d - 1) * batch + q) * W + slot; };
  // supertree node index of the parent of node g at depth d >= 2 (slots
  // outside S_{d-1} are clamped: malformed levels cannot index out of bounds)
  auto parent_node = [&](int d, int g) {
    const int ps = min(max(s_par[g], 0), shape.n[d - 2] - 1);
    return shape.off[d - 2] + ps;
  };

  // 0. stage the levels in LDS (one pass of independent loads) and build the
  // 1. top-B keys of the supertree
  for (int g = threadIdx.x; g < npad; g += blockDim.x) {
    uint64_t key = ~0ull;
    if (g < total) {
      int d = 1;
      while (g >= shape.off[d]) ++d;
      const int slot = g - shape.off[d - 1];
      const int64_t li = lvl_index(d, slot);
      const float sc = lvl_score[li];
      s_tok[g] = lvl_tok[li];
      s_par[g] = lvl_par[li];
      s_score[g] = sc;
      key = (uint64_t(score_desc_key(sc)) << 32) | (uint32_t(d) << 16) | uint32_t(slot);
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
        const uint32_t pidx = d == 1 ? 0u : uint32_t(out_idx[parent_node(d, od + i)]);
        rk = (pidx << 20) | (uint32_t(s_tok[od + i]) & 0xFFFFFu);
      }
      rank_key[i] = rk;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < nd; i += blockDim.x) {
      const uint32_t mine = rank_key[i];
      if (mine == ~0u) continue;
      // 16-byte reads of four keys at a time, then the tail
      typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
      const u32x4v* rk4 = reinterpret_cast<const u32x4v*>(rank_key);
      const int nd4 = nd & ~3;
      int r = 0;
      for (int j = 0; j < nd4; j += 4) {
        const u32x4v kv = rk4[j >> 2];
#pragma unroll
        for (int e = 0; e < 4; ++e) r += (kv[e] < mine) | ((kv[e] == mine) & (j + e < i));
      }
      for (int j = nd4; j < nd; ++j) r += (rank_key[j] < mine) | ((rank_key[j] == mine) & (j < i));
      out_idx[od + i] = base + r;
      par_out[base + r] = d == 1 ? -1 : out_idx[parent_node(d, od + i)];
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
      out.tokens[ob + o] = s_tok[od + i];
      out.parents[ob + o] = par_out[o];
      out.depths[ob + o] = d;
      out.scores[ob + o] = s_score[od + i];
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

int select_level_waves(int k) {
  switch (topk_bucket(k)) {
    case 1: return select_threads<1>() / 64;
    case 2: return select_threads<2>() / 64;
    case 4: return select_threads<4>() / 64;
    case 8: return select_threads<8>() / 64;
    case 16: return select_threads<16>() / 64;
    default: return select_threads<32>() / 64;
  }
}

hipError_t launch_select_level(const LevelArgs& a, hipStream_t s) {
  if (a.batch <= 0) return hipSuccess;
  // state slices: enough blocks to spread the state rows over the chip
  const int S = a.state ? std::max(1, std::min(a.n_keep, (256 + a.batch - 1) / a.batch)) : 1;
  const dim3 grid(unsigned(a.batch) * unsigned(S));
  // the top-k bucket only sizes the segment merge; without one the widest block serves
  switch ((a.shared_k > 0 || a.nseg <= 1) ? 1 : topk_bucket(a.k)) {
    case 1: hipLaunchKernelGGL((select_level<1>), grid, dim3(select_threads<1>()), 0, s, a, S); break;
    case 2: hipLaunchKernelGGL((select_level<2>), grid, dim3(select_threads<2>()), 0, s, a, S); break;
    case 4: hipLaunchKernelGGL((select_level<4>), grid, dim3(select_threads<4>()), 0, s, a, S); break;
    case 8: hipLaunchKernelGGL((select_level<8>), grid, dim3(select_threads<8>()), 0, s, a, S); break;
    case 16: hipLaunchKernelGGL((select_level<16>), grid, dim3(select_threads<16>()), 0, s, a, S); break;
    default: hipLaunchKernelGGL((select_level<32>), grid, dim3(select_threads<32>()), 0, s, a, S); break;
  }
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
