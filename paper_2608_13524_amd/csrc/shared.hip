// Shared candidate sets (Algorithm 1 as printed): C_d = TopK(L_d^base, K) for
// every request and depth, and the corrected logits of every node of a depth
// over C_d only, z_j[c] = L_d^base[C_d[c]] + U[C_d[c]] . a_j.
//  * cset_group_max / cset_select: theta = the least of the maxima of K
//    disjoint groups of a row bounds the K-th largest value from below; the
//    elements >= theta are compacted and sorted as 64-bit keys (score key << 32
//    | id, ascending = (value desc, id asc)), with an exact radix select when
//    too many qualify (heavy ties).
//  * shared_logits_bf16: a gather-product on MFMA.  Block (request, 16
//    candidates, up to 64 node rows); the A operand is 16 rows of U picked by
//    the set, the B operand 16 node rows of a; 16 waves split h and are
//    summed through LDS in wave order.  fp32 mode: one thread per (node,
//    candidate).
#include "reduce.hpp"

namespace dartree {
namespace {

// Orderable 32-bit key of a logit: larger key = larger value (-0 taken as +0).
__device__ __forceinline__ uint32_t ord_key(float x) {
  const uint32_t b = __float_as_uint(x + 0.0f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Group maxima: group g of a row is [g V / K, (g + 1) V / K); one wave per
// group.  grid: rows * ceil(K / 4), block 256.
__global__ __launch_bounds__(256) void cset_group_max(const float* __restrict__ logits, int vocab, int K, int gpb,
                                                      float* gmax) {
  const int64_t row = blockIdx.x / gpb;
  const int g = (blockIdx.x % gpb) * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (g >= K) return;   // whole waves only
  const int v0 = int(int64_t(g) * vocab / K), v1 = int(int64_t(g + 1) * vocab / K);
  const float* x = logits + row * int64_t(vocab);
  float m = -INFINITY;
#pragma unroll 8
  for (int v = v0 + lane; v < v1; v += 64) m = fmaxf(m, x[v]);
  m = wave_max(m);
  if (lane == 0) gmax[row * K + g] = m;
}

constexpr int kSelCap = 4096;   // candidates above the threshold sorted in LDS

// One row per block (1024 threads).  theta = min over the K group maxima is
// <= the K-th largest value, so every one of the K best is >= theta.  The
// elements >= theta (at least K) are compacted and sorted.  When more than
// kSelCap qualify (heavy ties), an exact radix select finds the K-th largest
// key T instead: the elements above T (fewer than K) are sorted, and the
// elements equal to T follow in id order.
__global__ __launch_bounds__(1024) void cset_select(const float* __restrict__ logits, int vocab, int K,
                                                    const float* __restrict__ gmax, int32_t* ids) {
  __shared__ uint64_t cand[kSelCap];
  __shared__ uint32_t hist[16][256];
  __shared__ int count, remaining_s, taken_s;
  __shared__ uint32_t prefix_s;
  __shared__ int wave_tot[16];
  const int64_t row = blockIdx.x;
  const float* x = logits + row * int64_t(vocab);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int32_t* out = ids + row * K;

  float theta = INFINITY;
  for (int g = tid; g < K; g += blockDim.x) theta = fminf(theta, gmax[row * K + g]);
  {  // block minimum
    __shared__ float red[16];
    theta = -wave_max(-theta);
    if (lane == 0) red[wave] = theta;
    if (tid == 0) count = 0;
    __syncthreads();
    theta = red[0];
    for (int w = 1; w < int(blockDim.x >> 6); ++w) theta = fminf(theta, red[w]);
  }
  // 8 loads in flight per thread before any check (the atomics below would
  // otherwise keep the loads from overlapping)
  constexpr int kBatch = 8;
  if ((vocab & 3) == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0) {
    // float4 loads: four times the bytes in flight of the scalar loop
    const f32x4* x4 = reinterpret_cast<const f32x4*>(x);
    const int n4 = vocab >> 2;
    for (int base = 0; base < n4; base += kBatch * int(blockDim.x)) {
      f32x4 xv[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int i = base + u * int(blockDim.x) + tid;
        xv[u] = i < n4 ? x4[i] : f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int i = base + u * int(blockDim.x) + tid;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (i < n4 && xv[u][e] >= theta) {
            const int pos = atomicAdd(&count, 1);
            if (pos < kSelCap) cand[pos] = (uint64_t(score_desc_key(xv[u][e])) << 32) | uint32_t(4 * i + e);
          }
      }
    }
  } else {
    for (int base = 0; base < vocab; base += kBatch * int(blockDim.x)) {
      float xv[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int v = base + u * int(blockDim.x) + tid;
        xv[u] = v < vocab ? x[v] : -INFINITY;
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int v = base + u * int(blockDim.x) + tid;
        if (v < vocab && xv[u] >= theta) {
          const int pos = atomicAdd(&count, 1);
          if (pos < kSelCap) cand[pos] = (uint64_t(score_desc_key(xv[u])) << 32) | uint32_t(v);
        }
      }
    }
  }
  __syncthreads();
  const int n = count;
  if (n <= kSelCap) {
    const int npad = next_pow2(n);
    for (int i = n + tid; i < npad; i += blockDim.x) cand[i] = ~0ull;
    __syncthreads();
    bitonic_sort(cand, npad);
    for (int r = tid; r < K; r += blockDim.x) out[r] = int32_t(uint32_t(cand[r]));
    return;
  }

  // exact radix select of the K-th largest orderable key, 8 bits at a time
  uint32_t prefix = 0, mask = 0;
  if (tid == 0) remaining_s = K;
  for (int pass = 3; pass >= 0; --pass) {
    for (int i = tid; i < 16 * 256; i += blockDim.x) (&hist[0][0])[i] = 0;
    __syncthreads();
    const int shift = 8 * pass;
    for (int v = tid; v < vocab; v += blockDim.x) {
      const uint32_t u = ord_key(x[v]);
      if ((u & mask) == prefix) atomicAdd(&hist[wave][(u >> shift) & 0xFF], 1u);
    }
    __syncthreads();
    if (tid == 0) {
      int rem = remaining_s;
      int bsel = 0;
      for (int bin = 255; bin >= 0; --bin) {
        int c = 0;
        for (int w = 0; w < int(blockDim.x >> 6); ++w) c += int(hist[w][bin]);
        if (c >= rem) { bsel = bin; break; }
        rem -= c;
      }
      remaining_s = rem;
      prefix_s = prefix | (uint32_t(bsel) << shift);
    }
    __syncthreads();
    prefix = prefix_s;
    mask |= 0xFFu << shift;
  }
  const uint32_t T = prefix;
  const int need_eq = remaining_s;   // elements equal to T to take, lowest ids first
  // elements above T: fewer than K, sorted
  if (tid == 0) count = 0;
  __syncthreads();
  for (int v = tid; v < vocab; v += blockDim.x) {
    const float xv = x[v];
    if (ord_key(xv) > T) cand[atomicAdd(&count, 1)] = (uint64_t(score_desc_key(xv)) << 32) | uint32_t(v);
  }
  __syncthreads();
  const int n_gt = count;   // = K - need_eq
  {
    const int npad = next_pow2(n_gt);
    for (int i = n_gt + tid; i < npad; i += blockDim.x) cand[i] = ~0ull;
    __syncthreads();
    bitonic_sort(cand, npad);
    for (int r = tid; r < n_gt; r += blockDim.x) out[r] = int32_t(uint32_t(cand[r]));
  }
  // elements equal to T in id order: block-wide prefix counts over tiles
  if (tid == 0) taken_s = 0;
  __syncthreads();
  for (int base = 0; base < vocab; base += blockDim.x) {
    const int v = base + tid;
    const bool eq = v < vocab && ord_key(x[v]) == T;
    const uint64_t bal = __ballot(eq);
    const int before_in_wave = __builtin_amdgcn_mbcnt_hi(uint32_t(bal >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(bal), 0));
    if (lane == 0) wave_tot[wave] = __popcll(bal);
    __syncthreads();
    int before = taken_s + before_in_wave;
    for (int w = 0; w < wave; ++w) before += wave_tot[w];
    if (eq && before < need_eq) out[n_gt + before] = v;
    __syncthreads();
    if (tid == 0) {
      int t = 0;
      for (int w = 0; w < int(blockDim.x >> 6); ++w) t += wave_tot[w];
      taken_s += t;
    }
    __syncthreads();
    if (taken_s >= need_eq) break;
  }
}

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

constexpr int kRowTiles = 4;  // node-row tiles of 16 per block

// grid: batch * ncb * nrb; block (q, cb, rb): candidates 16 cb .. 16 cb + 15,
// node rows 64 rb .. 64 rb + 63 of request q.  Rows past K or n_parent are
// clamped (computed, never stored).
__global__ __launch_bounds__(1024) void shared_logits_bf16(int np, int K, int hidden, int vocab, int ncb, int nrb,
                                                          const uint16_t* __restrict__ a,
                                                          const uint16_t* __restrict__ U,
                                                          const float* __restrict__ lb, int64_t lb_stride,
                                                          const int32_t* __restrict__ cset, int64_t cset_stride,
                                                          const int32_t* __restrict__ group_index, float* z) {
  constexpr int kWaves = 16;   // split h
  __shared__ f32x4 red[kWaves][kRowTiles][64];
  const int q = blockIdx.x / (ncb * nrb);
  const int rest = blockIdx.x - q * ncb * nrb;
  const int cb = rest / nrb, rb = rest % nrb;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int64_t g = group_index ? group_index[q] : q;   // L^base / C_d row of request q
  const int32_t* set = cset + g * cset_stride;
  const int c = min(16 * cb + r16, K - 1);
  // set ids come from the workspace: clamped into the vocabulary, so a set
  // that was never built (depths enqueued out of order) cannot index past U
  auto id_at = [&](int i) { return min(max(set[i], 0), vocab - 1); };
  const uint16_t* urow = U + int64_t(id_at(c)) * hidden + kg * 8;
  const uint16_t* arow[kRowTiles];
#pragma unroll
  for (int t = 0; t < kRowTiles; ++t) {
    const int j = min(64 * rb + 16 * t + r16, np - 1);
    arow[t] = a + (int64_t(q) * np + j) * hidden + kg * 8;
  }
  // node-row tiles this block needs (block-uniform)
  const int ntile = min(kRowTiles, (np - 64 * rb + 15) / 16);
  // wave 0 adds L^base at its lanes' four candidates: fetch them now, while
  // the products run, rather than after the reduction
  float lbv[4] = {0.f, 0.f, 0.f, 0.f};
  if (wave == 0) {
    const float* lbq = lb + g * lb_stride;
#pragma unroll
    for (int i = 0; i < 4; ++i) lbv[i] = lbq[id_at(min(16 * cb + 4 * kg + i, K - 1))];
  }
  f32x4 acc[kRowTiles];
#pragma unroll
  for (int t = 0; t < kRowTiles; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int k = wave * 32; k < hidden; k += kWaves * 32) {
    const bf16x8 av = __builtin_bit_cast(bf16x8, *reinterpret_cast<const f32x4*>(urow + k));
#pragma unroll
    for (int t = 0; t < kRowTiles; ++t) {
      if (t < ntile) {
        const bf16x8 bv = __builtin_bit_cast(bf16x8, *reinterpret_cast<const f32x4*>(arow[t] + k));
        acc[t] = mfma16(av, bv, acc[t]);
      }
    }
  }
#pragma unroll
  for (int t = 0; t < kRowTiles; ++t) red[wave][t][lane] = acc[t];
  __syncthreads();
  if (wave != 0) return;
  // lane holds D[candidate 4 kg + i][node row r16] of each tile; waves summed in order
#pragma unroll
  for (int t = 0; t < kRowTiles; ++t) {
    if (t >= ntile) continue;
    f32x4 v = red[0][t][lane];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) v += red[w][t][lane];
    const int j = 64 * rb + 16 * t + r16;
    if (j >= np) continue;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int cc = 16 * cb + 4 * kg + i;
      if (cc < K) z[(int64_t(q) * np + j) * K + cc] = v[i] + lbv[i];
    }
  }
}

// fp32: grid batch * ceil(np K / 256); thread (q, j, c) computes one dot product.
__global__ __launch_bounds__(256) void shared_logits_f32(int np, int K, int hidden, int vocab, int nblk,
                                                         const float* __restrict__ a,
                                                         const float* __restrict__ U, const float* __restrict__ lb,
                                                         int64_t lb_stride, const int32_t* __restrict__ cset,
                                                         int64_t cset_stride, const int32_t* __restrict__ group_index,
                                                         float* z) {
  const int q = blockIdx.x / nblk;
  const int e = (blockIdx.x % nblk) * blockDim.x + threadIdx.x;
  if (e >= np * K) return;
  const int j = e / K, cc = e % K;
  const int64_t g = group_index ? group_index[q] : q;
  const int tok = min(max(cset[g * cset_stride + cc], 0), vocab - 1);   // clamped as above
  const float* ar = a + (int64_t(q) * np + j) * hidden;
  const float* ur = U + int64_t(tok) * hidden;
  float acc = 0.f;
  for (int k = 0; k < hidden; ++k) acc = fmaf(ar[k], ur[k], acc);
  z[(int64_t(q) * np + j) * K + cc] = acc + lb[g * lb_stride + tok];
}

}  // namespace

size_t candidate_sets_scratch_bytes(int64_t rows, int64_t vocab, int K) {
  (void)vocab;
  return size_t(rows) * K * sizeof(float);   // the group maxima
}

bool candidate_sets_supported(int64_t vocab, int K) { return K >= 1 && K <= vocab && K <= DARTREE_MAX_CANDIDATES; }

hipError_t launch_candidate_sets(const float* logits, int64_t rows, int64_t vocab, int K, int32_t* ids,
                                 void* scratch, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  float* gmax = static_cast<float*>(scratch);
  const int gpb = (K + 3) / 4;
  hipLaunchKernelGGL(cset_group_max, dim3(unsigned(rows * gpb)), dim3(256), 0, s, logits, int(vocab), K, gpb, gmax);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(cset_select, dim3(unsigned(rows)), dim3(1024), 0, s, logits, int(vocab), K, gmax, ids);
  return hipGetLastError();
}

hipError_t launch_shared_logits(int precision, int batch, int np, int K, int hidden, int vocab, const void* a,
                                const void* U, const float* lb, int64_t lb_stride, const int32_t* cset,
                                int64_t cset_stride, const int32_t* group_index, float* z, hipStream_t s) {
  if (batch <= 0) return hipSuccess;
  if (precision == DARTREE_BF16) {
    const int ncb = (K + 15) / 16, nrb = (np + 16 * kRowTiles - 1) / (16 * kRowTiles);
    hipLaunchKernelGGL(shared_logits_bf16, dim3(unsigned(batch * ncb * nrb)), dim3(1024), 0, s, np, K, hidden, vocab,
                       ncb, nrb, static_cast<const uint16_t*>(a), static_cast<const uint16_t*>(U), lb, lb_stride, cset,
                       cset_stride, group_index, z);
  } else {
    const int nblk = (np * K + 255) / 256;
    hipLaunchKernelGGL(shared_logits_f32, dim3(unsigned(batch * nblk)), dim3(256), 0, s, np, K, hidden, vocab, nblk,
                       static_cast<const float*>(a), static_cast<const float*>(U), lb, lb_stride, cset, cset_stride,
                       group_index, z);
  }
  return hipGetLastError();
}

}  // namespace dartree
