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
//    g = l / 16; V is transposed in registers (4 keys x 8 dims per thread)
//    and stored to LDS with its keys already in that order, so one 16-byte
//    read gives a lane its V operand and P never leaves the registers.
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
constexpr int kKS = kD + 8;                // padded LDS row of K (bf16)
constexpr int kRows = 64;                  // query rows per block (4 waves x 16)
constexpr int kVS = kKeys + 8;             // padded LDS row of V^T (bf16)
// With at least this many (request, key/value head, row tile) blocks (two
// per CU on 256 CUs) every block covers all keys: no segment split, no merge.
constexpr int kFusedMinBlocks = 512;

// Position of key group kg4 (keys 4 kg4 .. 4 kg4 + 3 of a 64-key step) in a
// V^T row: 32-key chunk c = kg4 / 8, lane group g = kg4 % 4, half
// (kg4 / 4) % 2; the chunk holds, per lane group, its 4 keys of the first
// 16-key tile and then its 4 of the second.
__device__ __forceinline__ int vt_pos(int kg4) { return (kg4 >> 3) * 32 + (kg4 & 3) * 8 + ((kg4 >> 2) & 1) * 4; }

// Blocks are dealt to the 8 XCDs round-robin: give XCD x the contiguous run
// of work items [x n / 8, (x + 1) n / 8) so that the row tiles of one
// (request, key/value head), which read the same keys and values, share its L2.
__device__ __forceinline__ int attn_xcd_order(int b, int n) {
  const int q8 = n / 8;
  return b < 8 * q8 ? (b % 8) * q8 + b / 8 : b;
}

// grid: batch * Hkv * row tiles * segments (FUSED: batch * Hkv * row tiles).
// A block has 4 waves, each with RG groups of 16 query rows (a row tile is
// 64 RG rows).  Segment s < nseg_ctx covers context keys [s * seg_len,
// +seg_len) (clipped to the request's length); segment nseg_ctx covers the
// tree's B keys under the mask.  FUSED: one block covers the context keys
// [0, ctx_len) and then the tree keys.
template <bool FUSED, int RG>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void tree_attention_part(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t Ks[kKeys][kKS];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[kD][kVS];
  constexpr int kTileRows = kRows * RG;
  const int nseg = FUSED ? 1 : a.nseg_ctx + 1;
  const int rows = a.budget * a.group;
  const int ntile = (rows + kTileRows - 1) / kTileRows;
  int bid = FUSED ? attn_xcd_order(blockIdx.x, gridDim.x) : int(blockIdx.x);
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

  // this lane's query rows (rows past the end are computed on the last row, never stored)
  int row[RG], node[RG], head[RG];
  bf16x8 qf[RG][kD / 32];
  const uint64_t* mrow[RG];
#pragma unroll
  for (int rg = 0; rg < RG; ++rg) {
    row[rg] = rt * kTileRows + (wave * RG + rg) * 16 + r16;
    const int rowc = min(row[rg], rows - 1);
    node[rg] = rowc / a.group;
    head[rg] = kvh * a.group + rowc % a.group;
    const uint16_t* qp = a.q + ((int64_t(q) * a.budget + node[rg]) * a.heads_q + head[rg]) * kD + g * 8;
#pragma unroll
    for (int ks = 0; ks < kD / 32; ++ks)
      qf[rg][ks] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const f32x4*>(qp + ks * 32));
    mrow[rg] = a.mask + (int64_t(q) * a.budget + node[rg]) * words;
  }

  float m_run[RG], l_run[RG];
  f32x4 o[RG][kD / 16];
#pragma unroll
  for (int rg = 0; rg < RG; ++rg) {
    m_run[rg] = -INFINITY;
    l_run[rg] = 0.f;
#pragma unroll
    for (int dt = 0; dt < kD / 16; ++dt) o[rg][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
  typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
  // this thread's share of a 64-key step: 4 chunks of K (chunk c = tid + 256 i:
  // key c / 16, dims 8 (c % 16)), and of V the 8 dims 8 (tid / 16) of the 4
  // keys 4 (tid % 16) .. +3.  They are read with buffer loads whose range ends
  // at the step's last valid key (k1), so keys past it read as zero with no
  // per-lane test; the byte offsets within a step are fixed per thread.  The
  // next step's share is loaded while the current one is multiplied.
  const int vkg = threadIdx.x & 15, vdc = threadIdx.x >> 4;
  constexpr int kChunks = kKeys * kD / 8 / 256;
  const int key_bytes = a.heads_kv * kD * 2;
  int koff[kChunks], voff[4];
#pragma unroll
  for (int i = 0; i < kChunks; ++i) {
    const int c = threadIdx.x + 256 * i;
    koff[i] = (c / (kD / 8)) * key_bytes + kvh * kD * 2 + (c % (kD / 8)) * 16;
    voff[i] = (4 * vkg + i) * key_bytes + kvh * kD * 2 + 16 * vdc;
  }
  // keys [k0, k1) of one source (the context, or the tree under the mask)
  auto sweep = [&](const bool tree, const int k0, const int k1) {
    const uint16_t* kbase = tree ? a.k_tree + int64_t(q) * a.budget * a.heads_kv * kD
                                 : a.k_ctx + int64_t(q) * a.max_ctx * a.heads_kv * kD;
    const uint16_t* vbase = tree ? a.v_tree + int64_t(q) * a.budget * a.heads_kv * kD
                                 : a.v_ctx + int64_t(q) * a.max_ctx * a.heads_kv * kD;
    u16x8 kn[kChunks], vn[4];
    auto load_step = [&](int kb) {
      const int bytes = min(k1 - kb, kKeys) * key_bytes;
      const int64_t first = int64_t(kb) * a.heads_kv * kD;
      const __amdgpu_buffer_rsrc_t rk =
          __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(kbase + first), (short)0, bytes, 0x00020000);
      const __amdgpu_buffer_rsrc_t rv =
          __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(vbase + first), (short)0, bytes, 0x00020000);
#pragma unroll
      for (int i = 0; i < kChunks; ++i) kn[i] = __builtin_bit_cast(u16x8, __builtin_amdgcn_raw_buffer_load_b128(rk, koff[i], 0, 0));
#pragma unroll
      for (int i = 0; i < 4; ++i) vn[i] = __builtin_bit_cast(u16x8, __builtin_amdgcn_raw_buffer_load_b128(rv, voff[i], 0, 0));
    };
    if (k0 < k1) load_step(k0);

    for (int kb = k0; kb < k1; kb += kKeys) {
      __syncthreads();   // every wave is done with the previous step's tiles
#pragma unroll
      for (int i = 0; i < kChunks; ++i) {
        const int c = threadIdx.x + 256 * i;
        *reinterpret_cast<u16x8*>(&Ks[c / (kD / 8)][(c % (kD / 8)) * 8]) = kn[i];
      }
#pragma unroll
      for (int e = 0; e < 8; ++e)
        *reinterpret_cast<u16x4*>(&Vt[8 * vdc + e][vt_pos(vkg)]) = u16x4{vn[0][e], vn[1][e], vn[2][e], vn[3][e]};
      __syncthreads();
      if (kb + kKeys < k1) load_step(kb + kKeys);

      // S[key][query] for the 4 key tiles of 16, every row group
      f32x4 s[RG][4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
#pragma unroll
        for (int rg = 0; rg < RG; ++rg) s[rg][t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < kD / 32; ++ks) {
          const bf16x8 kf =
              __builtin_bit_cast(bf16x8, *reinterpret_cast<const f32x4*>(&Ks[t * 16 + r16][ks * 32 + g * 8]));
#pragma unroll
          for (int rg = 0; rg < RG; ++rg) s[rg][t] = mfma16(kf, qf[rg][ks], s[rg][t]);
        }
      }
      // visibility: a context step wholly inside [k0, k1) needs no test
      if (tree || kb + kKeys > k1) {
#pragma unroll
        for (int rg = 0; rg < RG; ++rg) {
          const uint64_t mw = tree ? mrow[rg][kb / 64] : ~0ull;
#pragma unroll
          for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int kl = t * 16 + g * 4 + i;   // key within the 64-key step
              if (!(kb + kl < k1 && ((mw >> kl) & 1ull))) s[rg][t][i] = -INFINITY;
            }
        }
      }
      // online softmax on the unscaled scores (scale > 0 keeps the order);
      // p = exp2(scale log2(e) (s - m)).  The running maximum m moves only when
      // a row's new maximum exceeds it by more than 8 / (scale log2(e)), so
      // p <= 2^8 and the rescaling of l and O is skipped for most steps.  A
      // row that has seen no visible key keeps m = -inf, l = 0, O = 0; the
      // arithmetic handles it (exp2(-inf) = 0), so control flow stays uniform
      // around the matrix-core instructions.
      const float c2 = a.scale_log2;
      bf16x8 pb[RG][2];
#pragma unroll
      for (int rg = 0; rg < RG; ++rg) {
        float bmax = -INFINITY;
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) bmax = fmaxf(bmax, s[rg][t][i]);
        bmax = fmaxf(bmax, __shfl_xor(bmax, 16));
        bmax = fmaxf(bmax, __shfl_xor(bmax, 32));
        const bool grow = bmax * c2 > m_run[rg] * c2 + 8.f;
        if (__any(grow)) {
          const float m_new = grow ? bmax : m_run[rg];
          const float alpha = __builtin_amdgcn_exp2f((m_run[rg] - (m_new == -INFINITY ? 0.f : m_new)) * c2);
          l_run[rg] *= alpha;
#pragma unroll
          for (int dt = 0; dt < kD / 16; ++dt) o[rg][dt] *= alpha;
          m_run[rg] = m_new;
        }
        const float nmc = -(m_run[rg] == -INFINITY ? 0.f : m_run[rg]) * c2;
        float psum = 0.f;
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            s[rg][t][i] = __builtin_amdgcn_exp2f(fmaf(s[rg][t][i], c2, nmc));
            psum += s[rg][t][i];
          }
        psum += __shfl_xor(psum, 16);
        psum += __shfl_xor(psum, 32);
        l_run[rg] += psum;
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            pb[rg][c][i] = __bf16(s[rg][2 * c][i]);
            pb[rg][c][4 + i] = __bf16(s[rg][2 * c + 1][i]);
          }
      }
      // O[dim][query] += V^T[dim][key] P[query][key] over the two 32-key chunks
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int dt = 0; dt < kD / 16; ++dt) {
          const bf16x8 vv =
              __builtin_bit_cast(bf16x8, *reinterpret_cast<const f32x4*>(&Vt[dt * 16 + r16][c * 32 + g * 8]));
#pragma unroll
          for (int rg = 0; rg < RG; ++rg) o[rg][dt] = mfma16(vv, pb[rg][c], o[rg][dt]);
        }
    }
  };

  if (FUSED) {
    sweep(false, 0, clen);
    sweep(true, 0, a.budget);
#pragma unroll
    for (int rg = 0; rg < RG; ++rg) {
      if (row[rg] >= rows) continue;
      const float inv = l_run[rg] > 0.f ? 1.f / l_run[rg] : 0.f;   // a row that sees nothing is zero
      float* op = a.out + ((int64_t(q) * a.budget + node[rg]) * a.heads_q + head[rg]) * kD;
#pragma unroll
      for (int dt = 0; dt < kD / 16; ++dt) *reinterpret_cast<f32x4*>(op + dt * 16 + g * 4) = o[rg][dt] * inv;
    }
    return;
  }
  const bool tree = seg == a.nseg_ctx;
  if (tree) sweep(true, 0, a.budget);
  else sweep(false, seg * a.seg_len, min(clen, seg * a.seg_len + a.seg_len));
#pragma unroll
  for (int rg = 0; rg < RG; ++rg) {
    if (row[rg] >= rows) continue;
    const int64_t pr = ((int64_t(seg) * a.batch + q) * a.heads_kv + kvh) * a.rows_pad + row[rg];
    if (g == 0) {
      a.part_ml[pr * 2] = m_run[rg];
      a.part_ml[pr * 2 + 1] = l_run[rg];
    }
    float* op = a.part_o + pr * kD;
#pragma unroll
    for (int dt = 0; dt < kD / 16; ++dt) *reinterpret_cast<f32x4*>(op + dt * 16 + g * 4) = o[rg][dt];
  }
}

// grid: batch * budget * ceil(heads_q / 8), block 1024: merge the segments
// of 8 query heads of one node, one (head, dim) output per thread.  The
// per-head segment weights w_s = exp2(scale log2(e) (m_s - M)) / L (m_s the
// segment's unscaled row maximum, M their maximum) go to LDS first; then
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
        const float m = a.part_ml[part(s, head) * 2];   // unscaled row maximum of segment s
        const float ws = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((m - M) * a.scale_log2);
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
    const int ntile2 = (rows + 2 * kRows - 1) / (2 * kRows);   // 128-row tiles
    hipLaunchKernelGGL((tree_attention_part<true, 2>), dim3(unsigned(a.batch) * a.heads_kv * ntile2), dim3(256), 0, s,
                       a);
    return hipGetLastError();
  }
  const unsigned parts = unsigned(a.batch) * a.heads_kv * ntile * (a.nseg_ctx + 1);
  hipLaunchKernelGGL((tree_attention_part<false, 1>), dim3(parts), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const unsigned nhg = unsigned((a.heads_q + kMergeHeads - 1) / kMergeHeads);
  hipLaunchKernelGGL(tree_attention_merge, dim3(unsigned(a.batch) * a.budget * nhg), dim3(kMergeThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace dartree
