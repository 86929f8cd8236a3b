// The consumer of the emitted tree (Sec. 2.1, Sec. 2.3, Sec. 4.1):
//
//  * accept_walk: from the root, move to the child whose token equals the
//    target's token at the current position (its greedy prediction at T = 0,
//    its sample at T = 1) and stop at the first position without one; the
//    target's token there is the bonus.  One wavefront per request, the tree
//    staged in LDS; the loop is bounded by the path capacity and the node
//    count, so it ends on any input.
//  * tree_attention: one attention layer over the flattened tree.  Node i's
//    query attends to the verified context and to the nodes of mask row i.
//    On MFMA: a block owns 64 query rows of one key/value head (16 nodes x 4
//    query heads of a group share every K/V block it loads).  With few rows
//    (one request of a few dozen nodes: too few blocks for the chip) it is
//    flash-decoding: a block takes one key segment (a context slice, or the
//    tree's own B keys under the mask), partial (max, sum, unnormalised
//    output) go to the workspace and a second kernel merges the segments.
//    With many rows a block sweeps the whole context and then the tree keys
//    with one online softmax and writes the normalised output itself.  S = K Q^T leaves lane l with query
//    row l % 16 and keys 4 (l / 16) + i of every 16-key tile, which is exactly
//    the B operand layout of the P V product when the keys of each 32-key
//    chunk are taken in the order {4g..4g+3, 16+4g..16+4g+3} for lane group
//    g = l / 16; V is staged transposed in LDS and read in that same order, so
//    P never leaves the registers.
#include "internal.hpp"

namespace dartree {
namespace {

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// Acceptance walk
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void accept_walk(int budget, int max_len, const int32_t* __restrict__ tokens,
                                                  const int32_t* __restrict__ parents,
                                                  const int32_t* __restrict__ num_nodes,
                                                  const int32_t* __restrict__ target, int32_t* accepted,
                                                  int32_t* n_accepted, int32_t* bonus) {
  __shared__ int32_t tok[DARTREE_MAX_SORT], par[DARTREE_MAX_SORT];
  const int q = blockIdx.x, lane = threadIdx.x;
  const int n = min(max(num_nodes[q], 0), budget);
  const int64_t tb = int64_t(q) * budget;
  for (int j = lane; j < n; j += 64) {
    tok[j] = tokens[tb + j];
    par[j] = parents[tb + j];
  }
  __syncthreads();
  const int32_t* tgt = target + int64_t(q) * (budget + 1);
  int cur = -1, count = 0;
  const int steps = min(max_len, n);
  while (count < steps) {
    const int want = tgt[cur + 1];
    int found = INT32_MAX;
    for (int j = lane; j < n; j += 64)
      if (par[j] == cur && tok[j] == want) found = min(found, j);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) found = min(found, __shfl_xor(found, off));
    if (found == INT32_MAX) break;
    if (lane == 0) accepted[int64_t(q) * max_len + count] = found;
    cur = found;
    ++count;
  }
  for (int j = count + lane; j < max_len; j += 64) accepted[int64_t(q) * max_len + j] = -1;
  if (lane == 0) {
    n_accepted[q] = count;
    bonus[q] = tgt[cur + 1];
  }
}

// ---------------------------------------------------------------------------
// Tree attention (head_dim 128)
// ---------------------------------------------------------------------------
constexpr int kD = 128;
constexpr int kKeys = 64;                  // keys per block step
constexpr int kRows = 64;                  // query rows per block (4 waves x 16)
constexpr int kKS = kD + 8;                // padded LDS row of K (bf16)
constexpr int kVS = kKeys + 8;             // padded LDS row of V^T (bf16)
// With at least this many (request, key/value head, row tile) blocks (two
// per CU on 256 CUs) every block covers all keys: no segment split, no merge.
constexpr int kFusedMinBlocks = 512;

// grid: batch * Hkv * row tiles * segments (FUSED: batch * Hkv * row tiles).
// Segment s < nseg_ctx covers context keys [s * seg_len, +seg_len) (clipped to
// the request's length); segment nseg_ctx covers the tree's B keys under the
// mask.  FUSED: one block covers the context keys [0, ctx_len) and then the
// tree keys.
template <bool FUSED>
__global__ __launch_bounds__(256) void tree_attention_part(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t Ks[kKeys][kKS];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[kD][kVS];
  const int nseg = FUSED ? 1 : a.nseg_ctx + 1;
  const int rows = a.budget * a.group;
  const int ntile = (rows + kRows - 1) / kRows;
  int bid = blockIdx.x;
  const int seg = bid % nseg;
  bid /= nseg;
  const int rt = bid % ntile;
  bid /= ntile;
  const int kvh = bid % a.heads_kv;
  const int q = bid / a.heads_kv;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int clen = a.ctx_len ? min(max(a.ctx_len[q], 0), a.max_ctx) : a.max_ctx;
  const int words = (a.budget + 63) / 64;

  // this lane's query row (rows past the end are computed on the last row, never stored)
  const int row = rt * kRows + wave * 16 + r16;
  const int rowc = min(row, rows - 1);
  const int node = rowc / a.group, head = kvh * a.group + rowc % a.group;
  const uint16_t* qp = a.q + ((int64_t(q) * a.budget + node) * a.heads_q + head) * kD + g * 8;
  bf16x8 qf[kD / 32];
#pragma unroll
  for (int ks = 0; ks < kD / 32; ++ks) qf[ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const f32x4*>(qp + ks * 32));
  const uint64_t* mrow = a.mask + (int64_t(q) * a.budget + node) * words;

  float m_run = -INFINITY, l_run = 0.f;
  f32x4 o[kD / 16];
#pragma unroll
  for (int dt = 0; dt < kD / 16; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // keys [k0, k1) of one source (the context, or the tree under the mask)
  auto sweep = [&](const bool tree, const int k0, const int k1) {
    const uint16_t* kbase = tree ? a.k_tree + int64_t(q) * a.budget * a.heads_kv * kD
                                 : a.k_ctx + int64_t(q) * a.max_ctx * a.heads_kv * kD;
    const uint16_t* vbase = tree ? a.v_tree + int64_t(q) * a.budget * a.heads_kv * kD
                                 : a.v_ctx + int64_t(q) * a.max_ctx * a.heads_kv * kD;
    // this thread's share of a 64-key step: 4 chunks of K (a wave covers 4
    // whole rows) and 4 of V (a wave covers 64 keys of one 8-dim slice, so the
    // transposed 2-byte stores spread over the banks); keys past k1 are zero,
    // never read from memory.  The next step's share is loaded while the
    // current one is multiplied.
    typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
    constexpr int kChunks = kKeys * kD / 8 / 256;
    u16x8 kn[kChunks], vn[kChunks];
    auto load_step = [&](int kb) {
#pragma unroll
      for (int i = 0; i < kChunks; ++i) {
        const int c = threadIdx.x + 256 * i;
        const int kk = c / (kD / 8), kd = (c % (kD / 8)) * 8;
        const int vk = c % kKeys, vd = (c / kKeys) * 8;
        kn[i] = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
        vn[i] = kn[i];
        if (kb + kk < k1) kn[i] = *reinterpret_cast<const u16x8*>(kbase + (int64_t(kb + kk) * a.heads_kv + kvh) * kD + kd);
        if (kb + vk < k1) vn[i] = *reinterpret_cast<const u16x8*>(vbase + (int64_t(kb + vk) * a.heads_kv + kvh) * kD + vd);
      }
    };
    if (k0 < k1) load_step(k0);

    for (int kb = k0; kb < k1; kb += kKeys) {
      __syncthreads();   // every wave is done with the previous step's tiles
#pragma unroll
      for (int i = 0; i < kChunks; ++i) {
        const int c = threadIdx.x + 256 * i;
        *reinterpret_cast<u16x8*>(&Ks[c / (kD / 8)][(c % (kD / 8)) * 8]) = kn[i];
        const int vk = c % kKeys, vd = (c / kKeys) * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) Vt[vd + e][vk] = vn[i][e];
      }
      __syncthreads();
      if (kb + kKeys < k1) load_step(kb + kKeys);

      // S[key][query] for the 4 key tiles of 16
      f32x4 s[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        s[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < kD / 32; ++ks) {
          const bf16x8 kf =
              __builtin_bit_cast(bf16x8, *reinterpret_cast<const f32x4*>(&Ks[t * 16 + r16][ks * 32 + g * 8]));
          s[t] = mfma16(kf, qf[ks], s[t]);
        }
      }
      // visibility, scale (log2 domain) and the block's row maximum
      const uint64_t mw = tree ? mrow[kb / 64] : 0ull;
      float bmax = -INFINITY;
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int kl = t * 16 + g * 4 + i;   // key within the 64-key step
          const bool ok = kb + kl < k1 && (!tree || ((mw >> kl) & 1ull));
          s[t][i] = ok ? s[t][i] * a.scale_log2 : -INFINITY;
          bmax = fmaxf(bmax, s[t][i]);
        }
      bmax = fmaxf(bmax, __shfl_xor(bmax, 16));
      bmax = fmaxf(bmax, __shfl_xor(bmax, 32));
      // a row that has seen no visible key keeps m = -inf, l = 0, o = 0; the
      // arithmetic handles it (exp2(-inf) = 0), so control flow stays uniform
      // around the matrix-core instructions
      const float m_new = fmaxf(m_run, bmax);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
      float psum = 0.f;
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          s[t][i] = __builtin_amdgcn_exp2f(s[t][i] - m_use);
          psum += s[t][i];
        }
      psum += __shfl_xor(psum, 16);
      psum += __shfl_xor(psum, 32);
      l_run = l_run * alpha + psum;
      m_run = m_new;
#pragma unroll
      for (int dt = 0; dt < kD / 16; ++dt) o[dt] *= alpha;
      // O[dim][query] += V^T[dim][key] P[query][key] over the two 32-key chunks
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        bf16x8 pb;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          pb[i] = __bf16(s[2 * c][i]);
          pb[4 + i] = __bf16(s[2 * c + 1][i]);
        }
#pragma unroll
        for (int dt = 0; dt < kD / 16; ++dt) {
          typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
          const u16x4 lo = *reinterpret_cast<const u16x4*>(&Vt[dt * 16 + r16][c * 32 + g * 4]);
          const u16x4 hi = *reinterpret_cast<const u16x4*>(&Vt[dt * 16 + r16][c * 32 + 16 + g * 4]);
          const u16x8 vv = u16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
          o[dt] = mfma16(__builtin_bit_cast(bf16x8, vv), pb, o[dt]);
        }
      }
    }
  };

  if (FUSED) {
    sweep(false, 0, clen);
    sweep(true, 0, a.budget);
    if (row >= rows) return;
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;   // a row that sees nothing is zero
    float* op = a.out + ((int64_t(q) * a.budget + node) * a.heads_q + head) * kD;
#pragma unroll
    for (int dt = 0; dt < kD / 16; ++dt) *reinterpret_cast<f32x4*>(op + dt * 16 + g * 4) = o[dt] * inv;
    return;
  }
  const bool tree = seg == a.nseg_ctx;
  if (tree) sweep(true, 0, a.budget);
  else sweep(false, seg * a.seg_len, min(clen, seg * a.seg_len + a.seg_len));
  if (row >= rows) return;
  const int64_t pr = ((int64_t(seg) * a.batch + q) * a.heads_kv + kvh) * a.rows_pad + row;
  if (g == 0) {
    a.part_ml[pr * 2] = m_run;
    a.part_ml[pr * 2 + 1] = l_run;
  }
  float* op = a.part_o + pr * kD;
#pragma unroll
  for (int dt = 0; dt < kD / 16; ++dt) *reinterpret_cast<f32x4*>(op + dt * 16 + g * 4) = o[dt];
}

// grid: batch * budget * ceil(heads_q / 8), block 1024: merge the segments
// of 8 query heads of one node, one (head, dim) output per thread.  The
// per-head segment weights w_s = exp2(m_s - M) / L go to LDS first; then
// every output sums its segments' partial rows with independent loads.
constexpr int kMergeHeads = 8;
constexpr int kMergeThreads = kMergeHeads * kD;
constexpr int kMaxSegments = 1024;   // limit of nseg = context segments + 1 (checked on the host)
__global__ __launch_bounds__(kMergeThreads) void tree_attention_merge(AttnArgs a) {
  __shared__ float w[kMaxSegments * kMergeHeads];   // [nseg][kMergeHeads]
  const int nseg = a.nseg_ctx + 1;
  const int nhg = (a.heads_q + kMergeHeads - 1) / kMergeHeads;
  const int hg = blockIdx.x % nhg, node = (blockIdx.x / nhg) % a.budget, q = blockIdx.x / nhg / a.budget;
  auto part = [&](int s, int head) {
    const int kvh = head / a.group, row = node * a.group + head % a.group;
    return ((int64_t(s) * a.batch + q) * a.heads_kv + kvh) * a.rows_pad + row;
  };
  if (threadIdx.x < kMergeHeads) {
    const int head = hg * kMergeHeads + threadIdx.x;
    if (head < a.heads_q) {
      float M = -INFINITY;
      for (int s = 0; s < nseg; ++s) M = fmaxf(M, a.part_ml[part(s, head) * 2]);
      float L = 0.f;
      for (int s = 0; s < nseg; ++s) {
        const float m = a.part_ml[part(s, head) * 2];
        const float ws = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - M);
        w[s * kMergeHeads + threadIdx.x] = ws;
        L += ws * a.part_ml[part(s, head) * 2 + 1];
      }
      const float inv = L > 0.f ? 1.f / L : 0.f;   // a row that sees nothing is zero
      for (int s = 0; s < nseg; ++s) w[s * kMergeHeads + threadIdx.x] *= inv;
    }
  }
  __syncthreads();
  const int hl = threadIdx.x / kD, d = threadIdx.x % kD, head = hg * kMergeHeads + hl;
  if (head >= a.heads_q) return;
  float acc = 0.f;
  for (int s = 0; s < nseg; ++s) acc += w[s * kMergeHeads + hl] * a.part_o[part(s, head) * kD + d];
  a.out[((int64_t(q) * a.budget + node) * a.heads_q + head) * kD + d] = acc;
}

}  // namespace

int attention_segment_len() { return 4 * kKeys; }
int attention_max_segments() { return kMaxSegments; }
bool attention_fused(int batch, int budget, int heads_q, int heads_kv) {
  const int64_t rows = int64_t(budget) * (heads_q / heads_kv);
  return int64_t(batch) * heads_kv * ((rows + kRows - 1) / kRows) >= kFusedMinBlocks;
}

hipError_t launch_accept_walk(int batch, int budget, int max_len, const int32_t* tokens, const int32_t* parents,
                              const int32_t* num_nodes, const int32_t* target, int32_t* accepted,
                              int32_t* n_accepted, int32_t* bonus, hipStream_t s) {
  if (batch <= 0) return hipSuccess;
  hipLaunchKernelGGL(accept_walk, dim3(unsigned(batch)), dim3(64), 0, s, budget, max_len, tokens, parents,
                     num_nodes, target, accepted, n_accepted, bonus);
  return hipGetLastError();
}

hipError_t launch_tree_attention(const AttnArgs& a, hipStream_t s) {
  if (a.batch <= 0) return hipSuccess;
  const int rows = a.budget * a.group;
  const int ntile = (rows + kRows - 1) / kRows;
  if (attention_fused(a.batch, a.budget, a.heads_q, a.heads_kv)) {
    hipLaunchKernelGGL(tree_attention_part<true>, dim3(unsigned(a.batch) * a.heads_kv * ntile), dim3(256), 0, s, a);
    return hipGetLastError();
  }
  const unsigned parts = unsigned(a.batch) * a.heads_kv * ntile * (a.nseg_ctx + 1);
  hipLaunchKernelGGL(tree_attention_part<false>, dim3(parts), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const unsigned nhg = unsigned((a.heads_q + kMergeHeads - 1) / kMergeHeads);
  hipLaunchKernelGGL(tree_attention_merge, dim3(unsigned(a.batch) * a.budget * nhg), dim3(kMergeThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace dartree
