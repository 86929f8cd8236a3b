// Shared candidate sets (Algorithm 1 as printed): C_d = TopK(L_d^base, K) for
// every request and depth, and the corrected logits of every node of a depth
// over C_d only, z_j[c] = L_d^base[C_d[c]] + U[C_d[c]] . a_j.
//  * cset_chunks / cset_merge: each block sorts one chunk of a logit row as
//    64-bit keys (score key << 32 | id, ascending = (value desc, id asc)) and
//    keeps its K best; one block per row then sorts the chunk winners.
//  * shared_logits_bf16: a gather-product on MFMA.  Block (request, 16
//    candidates, up to 64 node rows); the A operand is 16 rows of U picked by
//    the set, the B operand 16 node rows of a; the 4 waves split h and are
//    summed through LDS.  fp32 mode: one thread per (node, candidate).
#include "reduce.hpp"

namespace dartree {
namespace {

constexpr int kChunk = DARTREE_CSET_CHUNK;

__global__ __launch_bounds__(1024) void cset_chunks(const float* __restrict__ logits, int vocab, int nchunk, int K,
                                                     uint64_t* scratch) {
  __shared__ uint64_t keys[kChunk];
  const int64_t row = blockIdx.x / nchunk;
  const int ch = blockIdx.x % nchunk;
  const int v0 = ch * kChunk;
  const int n = min(kChunk, vocab - v0);
  const float* x = logits + row * int64_t(vocab);
  const int npad = next_pow2(n);
  for (int i = threadIdx.x; i < npad; i += blockDim.x)
    keys[i] = i < n ? (uint64_t(score_desc_key(x[v0 + i])) << 32) | uint32_t(v0 + i) : ~0ull;
  __syncthreads();
  bitonic_sort(keys, npad);
  uint64_t* out = scratch + (row * nchunk + ch) * K;
  for (int r = threadIdx.x; r < K; r += blockDim.x) out[r] = r < n ? keys[r] : ~0ull;
}

__global__ __launch_bounds__(1024) void cset_merge(int nchunk, int K, const uint64_t* __restrict__ scratch,
                                                    int32_t* ids) {
  __shared__ uint64_t keys[8192];
  const int64_t row = blockIdx.x;
  const int n = nchunk * K;
  const int npad = next_pow2(n);
  for (int i = threadIdx.x; i < npad; i += blockDim.x) keys[i] = i < n ? scratch[row * n + i] : ~0ull;
  __syncthreads();
  bitonic_sort(keys, npad);
  for (int r = threadIdx.x; r < K; r += blockDim.x) ids[row * K + r] = int32_t(uint32_t(keys[r]));
}

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

constexpr int kRowTiles = 4;  // node-row tiles of 16 per block

// grid: batch * ncb * nrb; block (q, cb, rb): candidates 16 cb .. 16 cb + 15,
// node rows 64 rb .. 64 rb + 63 of request q.  Rows past K or n_parent are
// clamped (computed, never stored).
__global__ __launch_bounds__(256) void shared_logits_bf16(int np, int K, int hidden, int ncb, int nrb,
                                                          const uint16_t* __restrict__ a,
                                                          const uint16_t* __restrict__ U,
                                                          const float* __restrict__ lb, int64_t lb_stride,
                                                          const int32_t* __restrict__ cset, int64_t cset_stride,
                                                          float* z) {
  __shared__ f32x4 red[4][kRowTiles][64];
  const int q = blockIdx.x / (ncb * nrb);
  const int rest = blockIdx.x - q * ncb * nrb;
  const int cb = rest / nrb, rb = rest % nrb;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int32_t* set = cset + q * cset_stride;
  const int c = min(16 * cb + r16, K - 1);
  const uint16_t* urow = U + int64_t(set[c]) * hidden + kg * 8;
  const uint16_t* arow[kRowTiles];
#pragma unroll
  for (int t = 0; t < kRowTiles; ++t) {
    const int j = min(64 * rb + 16 * t + r16, np - 1);
    arow[t] = a + (int64_t(q) * np + j) * hidden + kg * 8;
  }
  f32x4 acc[kRowTiles];
#pragma unroll
  for (int t = 0; t < kRowTiles; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int k = wave * 32; k < hidden; k += 4 * 32) {
    const bf16x8 av = __builtin_bit_cast(bf16x8, *reinterpret_cast<const f32x4*>(urow + k));
#pragma unroll
    for (int t = 0; t < kRowTiles; ++t) {
      const bf16x8 bv = __builtin_bit_cast(bf16x8, *reinterpret_cast<const f32x4*>(arow[t] + k));
      acc[t] = mfma16(av, bv, acc[t]);
    }
  }
#pragma unroll
  for (int t = 0; t < kRowTiles; ++t) red[wave][t][lane] = acc[t];
  __syncthreads();
  if (wave != 0) return;
  const float* lbq = lb + q * lb_stride;
  // lane holds D[candidate 4 kg + i][node row r16] of each tile
#pragma unroll
  for (int t = 0; t < kRowTiles; ++t) {
    const f32x4 v = red[0][t][lane] + red[1][t][lane] + red[2][t][lane] + red[3][t][lane];
    const int j = 64 * rb + 16 * t + r16;
    if (j >= np) continue;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int cc = 16 * cb + 4 * kg + i;
      if (cc < K) z[(int64_t(q) * np + j) * K + cc] = v[i] + lbq[set[cc]];
    }
  }
}

// fp32: grid batch * ceil(np K / 256); thread (q, j, c) computes one dot product.
__global__ __launch_bounds__(256) void shared_logits_f32(int np, int K, int hidden, int nblk, const float* __restrict__ a,
                                                         const float* __restrict__ U, const float* __restrict__ lb,
                                                         int64_t lb_stride, const int32_t* __restrict__ cset,
                                                         int64_t cset_stride, float* z) {
  const int q = blockIdx.x / nblk;
  const int e = (blockIdx.x % nblk) * blockDim.x + threadIdx.x;
  if (e >= np * K) return;
  const int j = e / K, cc = e % K;
  const int tok = cset[q * cset_stride + cc];
  const float* ar = a + (int64_t(q) * np + j) * hidden;
  const float* ur = U + int64_t(tok) * hidden;
  float acc = 0.f;
  for (int k = 0; k < hidden; ++k) acc = fmaf(ar[k], ur[k], acc);
  z[(int64_t(q) * np + j) * K + cc] = acc + lb[q * lb_stride + tok];
}

int cset_nchunk(int64_t vocab) { return int((vocab + kChunk - 1) / kChunk); }

}  // namespace

size_t candidate_sets_scratch_bytes(int64_t rows, int64_t vocab, int K) {
  return size_t(rows) * cset_nchunk(vocab) * K * sizeof(uint64_t);
}

bool candidate_sets_supported(int64_t vocab, int K) { return int64_t(cset_nchunk(vocab)) * K <= 8192; }

hipError_t launch_candidate_sets(const float* logits, int64_t rows, int64_t vocab, int K, int32_t* ids,
                                 void* scratch, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const int nchunk = cset_nchunk(vocab);
  uint64_t* sc = static_cast<uint64_t*>(scratch);
  hipLaunchKernelGGL(cset_chunks, dim3(unsigned(rows * nchunk)), dim3(1024), 0, s, logits, int(vocab), nchunk, K, sc);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(cset_merge, dim3(unsigned(rows)), dim3(1024), 0, s, nchunk, K, sc, ids);
  return hipGetLastError();
}

hipError_t launch_shared_logits(int precision, int batch, int np, int K, int hidden, const void* a, const void* U,
                                const float* lb, int64_t lb_stride, const int32_t* cset, int64_t cset_stride,
                                float* z, hipStream_t s) {
  if (batch <= 0) return hipSuccess;
  if (precision == DARTREE_BF16) {
    const int ncb = (K + 15) / 16, nrb = (np + 16 * kRowTiles - 1) / (16 * kRowTiles);
    hipLaunchKernelGGL(shared_logits_bf16, dim3(unsigned(batch * ncb * nrb)), dim3(256), 0, s, np, K, hidden, ncb, nrb,
                       static_cast<const uint16_t*>(a), static_cast<const uint16_t*>(U), lb, lb_stride, cset,
                       cset_stride, z);
  } else {
    const int nblk = (np * K + 255) / 256;
    hipLaunchKernelGGL(shared_logits_f32, dim3(unsigned(batch * nblk)), dim3(256), 0, s, np, K, hidden, nblk,
                       static_cast<const float*>(a), static_cast<const float*>(U), lb, lb_stride, cset, cset_stride,
                       z);
  }
  return hipGetLastError();
}

}  // namespace dartree
