// Log-softmax normaliser and per-row top-k of the corrected logits (Algorithm
// 1: log q~_d over the vocabulary, then the k best candidate children of each
// node).  One read of z:
//   * each thread streams float4s of its row segment, keeping an online
//     (max, sum of exp((z - max) / tau)) pair and a sorted top-K list in
//     registers (insertion only when a value beats the current K-th);
//   * the block merges with wavefront butterflies: (max, sum) pairs combine,
//     and the top-k is taken in k rounds of a (value desc, id asc) arg-max
//     across lanes, the winning lane shifting its list;
//   * rows are split into segments when there are too few rows to fill the
//     chip; a second kernel merges the per-segment partials in segment order.
// Ties: ids ascend along every thread's traversal, so "strictly greater"
// keeps the lower id first; every merge compares (value desc, id asc).
#include <float.h>

#include "internal.hpp"

namespace dartree {
namespace {

constexpr int kBlock = 256;
constexpr float kLog2e = 1.4426950408889634f;

struct Partial {
  float m;  // running max of z
  float s;  // sum of exp((z - m) / tau)
};

__device__ __forceinline__ bool better(float v, int i, float w, int j) {
  return v > w || (v == w && i < j);
}

__device__ __forceinline__ Partial combine(Partial a, Partial b, float scale) {
  // scale = log2(e) / tau.  exp2(-inf) = 0 handles an empty side.
  const float m = fmaxf(a.m, b.m);
  if (m == -INFINITY) return Partial{m, 0.f};
  return Partial{m, a.s * __builtin_amdgcn_exp2f((a.m - m) * scale) + b.s * __builtin_amdgcn_exp2f((b.m - m) * scale)};
}

template <int K>
__device__ __forceinline__ void insert(float v, int id, float (&tv)[K], int (&ti)[K]) {
  if (!better(v, id, tv[K - 1], ti[K - 1])) return;
  tv[K - 1] = v;
  ti[K - 1] = id;
#pragma unroll
  for (int j = K - 1; j > 0; --j) {
    if (better(tv[j], ti[j], tv[j - 1], ti[j - 1])) {
      const float fv = tv[j]; tv[j] = tv[j - 1]; tv[j - 1] = fv;
      const int fi = ti[j]; ti[j] = ti[j - 1]; ti[j - 1] = fi;
    }
  }
}

// Insertion along one thread's traversal, where ids only grow: a value equal
// to an entry already kept has a larger id and ranks after it, so comparing
// values alone gives the (value desc, id asc) order.
template <int K>
__device__ __forceinline__ void insert_ascending(float v, int id, float (&tv)[K], int (&ti)[K]) {
  tv[K - 1] = v;
  ti[K - 1] = id;
#pragma unroll
  for (int j = K - 1; j > 0; --j) {
    if (tv[j] > tv[j - 1]) {
      const float fv = tv[j]; tv[j] = tv[j - 1]; tv[j - 1] = fv;
      const int fi = ti[j]; ti[j] = ti[j - 1]; ti[j - 1] = fi;
    }
  }
}

// Ranking key of a candidate: a larger key ranks first, i.e. (value desc, id
// asc).  High word: the value's bits in unsigned order (-0 taken as +0, so
// equal values tie); low word: ~id.  The empty entry (-inf, INT32_MAX) has the
// smallest key any entry can have.
__device__ __forceinline__ uint64_t rank_key(float v, int id) {
  uint32_t b = __float_as_uint(v + 0.0f);
  b = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return (uint64_t(b) << 32) | uint32_t(~uint32_t(id));
}
__device__ __forceinline__ float key_value(uint64_t key) {
  const uint32_t b = uint32_t(key >> 32);
  return __uint_as_float((b & 0x80000000u) ? (b & 0x7FFFFFFFu) : ~b);
}
__device__ __forceinline__ int key_id(uint64_t key) { return int(~uint32_t(key)); }

// Wavefront reductions on DPP lane moves (no LDS round trip): two quad
// permutes and two row rotations leave every lane of a 16-lane row with the
// row's result; row broadcasts 15 and 31 carry it to lane 63, which is read
// back as a wave-uniform value.  Lanes whose row is masked off receive the
// identity.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp(uint32_t identity, uint32_t x) {
  return uint32_t(__builtin_amdgcn_update_dpp(int(identity), int(x), CTRL, ROW_MASK, 0xF, false));
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint64_t max_step(uint64_t x) {
  const uint64_t o = (uint64_t(dpp<CTRL, ROW_MASK>(0u, uint32_t(x >> 32))) << 32) | dpp<CTRL, ROW_MASK>(0u, uint32_t(x));
  return o > x ? o : x;
}
__device__ __forceinline__ uint64_t wave_max_key(uint64_t x) {
  x = max_step<0xB1, 0xF>(x);   // quad_perm [1,0,3,2]
  x = max_step<0x4E, 0xF>(x);   // quad_perm [2,3,0,1]
  x = max_step<0x124, 0xF>(x);  // row_ror:4
  x = max_step<0x128, 0xF>(x);  // row_ror:8
  x = max_step<0x142, 0xA>(x);  // row_bcast:15 into rows 1 and 3
  x = max_step<0x143, 0xC>(x);  // row_bcast:31 into rows 2 and 3
  const uint32_t hi = __builtin_amdgcn_readlane(uint32_t(x >> 32), 63);
  const uint32_t lo = __builtin_amdgcn_readlane(uint32_t(x), 63);
  return (uint64_t(hi) << 32) | lo;
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float fmax_step(float x) {
  return fmaxf(x, __uint_as_float(dpp<CTRL, ROW_MASK>(__float_as_uint(-INFINITY), __float_as_uint(x))));
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float add_step(float x) {
  return x + __uint_as_float(dpp<CTRL, ROW_MASK>(0u, __float_as_uint(x)));
}
__device__ __forceinline__ float wave_max(float x) {
  x = fmax_step<0xB1, 0xF>(x);
  x = fmax_step<0x4E, 0xF>(x);
  x = fmax_step<0x124, 0xF>(x);
  x = fmax_step<0x128, 0xF>(x);
  x = fmax_step<0x142, 0xA>(x);
  x = fmax_step<0x143, 0xC>(x);
  return __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(x), 63));
}
__device__ __forceinline__ float wave_sum(float x) {
  x = add_step<0xB1, 0xF>(x);
  x = add_step<0x4E, 0xF>(x);
  x = add_step<0x124, 0xF>(x);
  x = add_step<0x128, 0xF>(x);
  x = add_step<0x142, 0xA>(x);
  x = add_step<0x143, 0xC>(x);
  return __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(x), 63));
}

// (max, sum) of the wave: the sums are rescaled to the wave max, then added.
__device__ __forceinline__ Partial wave_partial(Partial p, float scale) {
  const float m = wave_max(p.m);
  if (m == -INFINITY) return Partial{m, 0.f};
  return Partial{m, wave_sum(p.s * __builtin_amdgcn_exp2f((p.m - m) * scale))};
}

// k rounds of a wave arg-max over the heads of the lanes' sorted key lists;
// the lane that supplied the winner shifts its list.  Keys are unique except
// the empty one, and shifting an empty list changes nothing.
template <int K>
__device__ __forceinline__ void wave_topk(uint64_t (&key)[K], int k, uint64_t (&out)[K]) {
#pragma unroll
  for (int r = 0; r < K; ++r) {
    if (r < k) {  // wave-uniform
      const uint64_t best = wave_max_key(key[0]);
      out[r] = best;
      if (key[0] == best) {
#pragma unroll
        for (int j = 0; j < K - 1; ++j) key[j] = key[j + 1];
        key[K - 1] = rank_key(-INFINITY, INT32_MAX);
      }
    }
  }
}

// Block-wide merge of the threads' (Partial, top-K).  Every wave reduces its
// own lists; the 4k wave winners are then ranked by counting (ties of equal
// keys by position), so each thread holding a block winner learns its output
// slot without another round of reductions.  Returns the block's Partial in
// every thread, and in threads with *slot in [0, k) the key of rank *slot.
template <int K>
__device__ __forceinline__ uint64_t block_merge(Partial& p, const float (&tv)[K], const int (&ti)[K], int k,
                                                float scale, int* slot) {
  constexpr int kWaves = kBlock / 64;
  __shared__ Partial sp[kWaves];
  __shared__ uint64_t sk[kWaves * K];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const Partial wp = wave_partial(p, scale);
  uint64_t key[K], out[K];
#pragma unroll
  for (int r = 0; r < K; ++r) key[r] = rank_key(tv[r], ti[r]);
  wave_topk<K>(key, k, out);
  if (lane == 0) {
    sp[wave] = wp;
#pragma unroll
    for (int r = 0; r < K; ++r)
      if (r < k) sk[wave * k + r] = out[r];
  }
  __syncthreads();
  Partial q{-INFINITY, 0.f};
#pragma unroll
  for (int w = 0; w < kWaves; ++w) q = combine(q, sp[w], scale);  // fixed order
  p = q;
  const int n = kWaves * k, t = threadIdx.x;
  *slot = -1;
  if (t >= n) return 0;
  const uint64_t e = sk[t];
  int rank = 0;
  for (int j = 0; j < n; ++j) {
    const uint64_t o = sk[j];
    rank += int(o > e) + int(o == e && j < t);
  }
  *slot = rank;
  return e;
}

// Outputs of the row from the merged result: lse once, and one candidate per
// thread holding a rank below k.
__device__ __forceinline__ void emit_row(int64_t row, Partial p, uint64_t key, int slot, int k, float tau,
                                         float* lse, float* cand_logp, int32_t* cand_ids) {
  if (slot < 0 || slot >= k) return;
  const float log_s = logf(p.s);
  if (slot == 0) lse[row] = p.m / tau + log_s;
  cand_logp[row * k + slot] = (key_value(key) - p.m) / tau - log_s;
  cand_ids[row * k + slot] = key_id(key);
}

constexpr int kChunk = 4;  // float4 loads in flight per thread

// Partial record of one row segment: m, s, two pad words, K values, K ids.
template <int K>
constexpr int record_floats() { return (4 + 2 * K + 3) & ~3; }

// Fold the nseg records of one row into each thread's (Partial, top-K):
// threads take single candidates, which keeps this tail small in registers.
template <int K>
__device__ void fold_records(const float* recs, int nseg, int k, float scale, Partial& p, float (&tv)[K],
                             int (&ti)[K]) {
  constexpr int RF = record_floats<K>();
  p = Partial{-INFINITY, 0.f};
  for (int sg = threadIdx.x; sg < nseg; sg += blockDim.x) p = combine(p, Partial{recs[sg * RF], recs[sg * RF + 1]}, scale);
#pragma unroll
  for (int r = 0; r < K; ++r) { tv[r] = -INFINITY; ti[r] = INT32_MAX; }
#pragma unroll 1
  for (int c = threadIdx.x; c < nseg * k; c += blockDim.x) {
    const int sg = c / k, r = c - sg * k;
    insert<K>(recs[sg * RF + 4 + r], __float_as_int(recs[sg * RF + 4 + K + r]), tv, ti);
  }
}

// grid: rows * nseg blocks, block = row * nseg + segment.  One segment per
// row writes the result directly; otherwise every block writes its segment's
// record for lse_topk_merge.
template <int K, bool VEC>
__global__ __launch_bounds__(kBlock) void lse_topk_rows(const float* __restrict__ z, int vocab,
                                                        int nseg, int seg_len, int k, float tau,
                                                        float* lse, float* cand_logp,
                                                        int32_t* cand_ids, float* part) {
  // per-thread staging row for the (rare) chunks that reach the top-K list
  __shared__ float stage[kBlock][4 * kChunk + 1];
  const int64_t row = blockIdx.x / nseg;
  const int seg = blockIdx.x % nseg;
  const int v0 = seg * seg_len;
  const int v1 = min(vocab, v0 + seg_len);
  const float* zr = z + row * int64_t(vocab);
  const float scale = kLog2e / tau;
  const int tid = threadIdx.x;

  Partial p{-INFINITY, 0.f};
  float tv[K];
  int ti[K];
#pragma unroll
  for (int r = 0; r < K; ++r) { tv[r] = -INFINITY; ti[r] = INT32_MAX; }

  if constexpr (VEC) {
    // Thread tid visits, per iteration, float4 c at base + 4 kBlock c: ids
    // ascend along the traversal.  The first float4 of an iteration is always
    // in range, so the running max is finite before any -inf padding is summed.
    for (int base = v0 + 4 * tid; base < v1; base += 4 * kBlock * kChunk) {
      f32x4 x[kChunk];
#pragma unroll
      for (int c = 0; c < kChunk; ++c) {
        const int v = base + 4 * kBlock * c;
        x[c] = v < v1 ? *reinterpret_cast<const f32x4*>(zr + v) : f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      }
      float mx = -INFINITY;
#pragma unroll
      for (int c = 0; c < kChunk; ++c) mx = fmaxf(mx, fmaxf(fmaxf(x[c][0], x[c][1]), fmaxf(x[c][2], x[c][3])));
      if (mx > p.m) {
        p.s *= __builtin_amdgcn_exp2f((p.m - mx) * scale);
        p.m = mx;
      }
      float acc = 0.f;
#pragma unroll
      for (int c = 0; c < kChunk; ++c)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc += __builtin_amdgcn_exp2f((x[c][i] - p.m) * scale);
      p.s += acc;
      if (mx > tv[K - 1]) {
        // only this lane's values above its current K-th are visited, in id order
        const float thr = tv[K - 1];
        uint32_t mask = 0;
#pragma unroll
        for (int c = 0; c < kChunk; ++c)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            stage[tid][4 * c + i] = x[c][i];
            mask |= uint32_t(x[c][i] > thr) << (4 * c + i);
          }
        while (mask) {
          const int j = __builtin_ctz(mask);
          mask &= mask - 1;
          const float xv = stage[tid][j];
          if (xv > tv[K - 1]) insert_ascending<K>(xv, base + 4 * kBlock * (j >> 2) + (j & 3), tv, ti);
        }
      }
    }
  } else {
#pragma unroll 1
    for (int v = v0 + tid; v < v1; v += kBlock) {
      const float x = zr[v];
      if (x > p.m) {
        p.s *= __builtin_amdgcn_exp2f((p.m - x) * scale);
        p.m = x;
      }
      p.s += __builtin_amdgcn_exp2f((x - p.m) * scale);
      if (x > tv[K - 1]) insert_ascending<K>(x, v, tv, ti);
    }
  }

  int slot;
  const uint64_t key = block_merge<K>(p, tv, ti, k, scale, &slot);
  if (nseg == 1) {
    emit_row(row, p, key, slot, k, tau, lse, cand_logp, cand_ids);
    return;
  }
  if (slot < 0 || slot >= k) return;
  constexpr int RF = record_floats<K>();
  float* rec = part + (row * nseg + seg) * RF;
  if (slot == 0) {
    rec[0] = p.m;
    rec[1] = p.s;
  }
  rec[4 + slot] = key_value(key);
  rec[4 + K + slot] = __int_as_float(key_id(key));
}

// grid: rows.  Merge the row's segment records, every thread folding single
// candidates (no thread waits on a chain of dependent loads).
template <int K>
__global__ __launch_bounds__(kBlock) void lse_topk_merge(int nseg, int k, float tau, const float* part, float* lse,
                                                         float* cand_logp, int32_t* cand_ids) {
  const int64_t row = blockIdx.x;
  const float scale = kLog2e / tau;
  Partial p;
  float tv[K];
  int ti[K];
  fold_records<K>(part + row * nseg * record_floats<K>(), nseg, k, scale, p, tv, ti);
  int slot;
  const uint64_t key = block_merge<K>(p, tv, ti, k, scale, &slot);
  emit_row(row, p, key, slot, k, tau, lse, cand_logp, cand_ids);
}

// Segments per row: enough blocks to fill 256 CUs a few times over, but no
// segment shorter than 2048 elements.
int num_segments(int64_t rows, int64_t vocab) {
  const int64_t want = (2048 + rows - 1) / rows;
  const int64_t most = (vocab + 2047) / 2048;
  return int(std::max<int64_t>(1, std::min(want, most)));
}

template <int K>
hipError_t launch_k(const float* z, int64_t rows, int64_t vocab, int k, float tau, float* lse,
                    float* cand_logp, int32_t* cand_ids, float* part, hipStream_t s) {
  const int nseg = num_segments(rows, vocab);
  const bool vec = (vocab % 4) == 0 && (reinterpret_cast<uintptr_t>(z) % 16) == 0;
  int seg_len = int((vocab + nseg - 1) / nseg);
  if (vec) seg_len = (seg_len + 3) & ~3;
  const dim3 grid(unsigned(rows * nseg));
  if (vec)
    hipLaunchKernelGGL((lse_topk_rows<K, true>), grid, dim3(kBlock), 0, s, z, int(vocab), nseg, seg_len, k, tau,
                       lse, cand_logp, cand_ids, part);
  else
    hipLaunchKernelGGL((lse_topk_rows<K, false>), grid, dim3(kBlock), 0, s, z, int(vocab), nseg, seg_len, k, tau,
                       lse, cand_logp, cand_ids, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || nseg == 1) return e;
  hipLaunchKernelGGL((lse_topk_merge<K>), dim3(unsigned(rows)), dim3(kBlock), 0, s, nseg, k, tau, part, lse,
                     cand_logp, cand_ids);
  return hipGetLastError();
}

}  // namespace

size_t lse_topk_scratch_bytes(int64_t rows, int64_t vocab, int k) {
  const int nseg = num_segments(rows, vocab);
  if (nseg == 1) return 0;
  const int K = k <= 1 ? 1 : k <= 2 ? 2 : k <= 4 ? 4 : k <= 8 ? 8 : k <= 16 ? 16 : 32;
  const size_t rf = size_t((4 + 2 * K + 3) & ~3);
  return size_t(rows) * nseg * rf * sizeof(float);
}

hipError_t launch_lse_topk(const float* z, int64_t rows, int64_t vocab, int k, float tau, float* lse,
                           float* cand_logp, int32_t* cand_ids, void* scratch, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  float* part = static_cast<float*>(scratch);
  if (k <= 1) return launch_k<1>(z, rows, vocab, k, tau, lse, cand_logp, cand_ids, part, s);
  if (k <= 2) return launch_k<2>(z, rows, vocab, k, tau, lse, cand_logp, cand_ids, part, s);
  if (k <= 4) return launch_k<4>(z, rows, vocab, k, tau, lse, cand_logp, cand_ids, part, s);
  if (k <= 8) return launch_k<8>(z, rows, vocab, k, tau, lse, cand_logp, cand_ids, part, s);
  if (k <= 16) return launch_k<16>(z, rows, vocab, k, tau, lse, cand_logp, cand_ids, part, s);
  return launch_k<32>(z, rows, vocab, k, tau, lse, cand_logp, cand_ids, part, s);
}

}  // namespace dartree
