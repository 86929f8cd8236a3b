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
// Ties: ids ascend along every thread's traversal, so a strictly-greater test
// keeps the lower id first; every merge compares (value desc, id asc).
#include <float.h>

#include <mutex>

#include "reduce.hpp"

namespace dartree {
namespace {

constexpr int kBlock = 256;
constexpr int kMidSegment = 4 * kBlock * 8;   // elements of a register-held segment at 8 float4 per thread

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
  __shared__ __attribute__((aligned(16))) uint64_t sk[kWaves * K];
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
  // 16-byte reads of two keys at a time (n = kWaves k is even)
  typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));
  const u64x2* sk2 = reinterpret_cast<const u64x2*>(sk);
  for (int j = 0; j < n; j += 2) {
    const u64x2 o = sk2[j >> 1];
    rank += int(o.x > e) + int(o.x == e && j < t) + int(o.y > e) + int(o.y == e && j + 1 < t);
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

// A segment of at most 4 kBlock CH values, held in registers after one pass
// of loads.  Every thread's best (value desc, id asc) is a distinct element,
// so the k-th best of those kBlock keys, T, is met or beaten by k elements of
// the segment and its k best are among the keys >= T.  Only the k threads
// whose best is >= T hold such keys, at most 4 CH each: they are compacted
// and ranked by counting.  The (max, sum) pair is merged as in block_merge.
// Writes the row's result (one segment) or the segment's record.
template <int K, int CH, bool NTL>
__device__ __forceinline__ void segment_in_registers(const float* zr, int v0, int v1, int nseg, int k, float tau,
                                                     float scale, int64_t row, int seg, float* lse, float* cand_logp,
                                                     int32_t* cand_ids, float* part) {
  constexpr int kWaves = kBlock / 64;
  constexpr int kCap = K * 4 * CH;
  __shared__ __attribute__((aligned(16))) uint64_t wkey[kWaves * K];
  __shared__ uint64_t cand[kCap];
  __shared__ Partial sp[kWaves];
  __shared__ uint64_t thr_s;
  __shared__ int count;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  f32x4 x[CH];
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int v = v0 + 4 * tid + 4 * kBlock * c;
    const f32x4* src = reinterpret_cast<const f32x4*>(zr + v);
    x[c] = v < v1 ? (NTL ? __builtin_nontemporal_load(src) : *src) : f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
  }
  float mx = -INFINITY;
  uint64_t best = rank_key(-INFINITY, INT32_MAX);
#pragma unroll
  for (int c = 0; c < CH; ++c)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int v = v0 + 4 * tid + 4 * kBlock * c + i;
      mx = fmaxf(mx, x[c][i]);
      if (v < v1) best = max(best, rank_key(x[c][i], v));
    }
  Partial p{mx, 0.f};
  if (mx > -INFINITY) {
#pragma unroll
    for (int c = 0; c < CH; ++c)
#pragma unroll
      for (int i = 0; i < 4; ++i) p.s += __builtin_amdgcn_exp2f((x[c][i] - mx) * scale);
  }
  const Partial wp = wave_partial(p, scale);
  if (lane == 0) sp[wave] = wp;
  // the k-th largest thread key (keys of threads holding values are distinct:
  // one id each; the others hold the empty key, the least of all): every
  // wave's k largest by k rounds of a wave arg-max, then the kWaves k wave
  // winners, which hold the block's k largest, ranked by counting (ranking
  // all kBlock keys against each other read 512 KB of LDS per block)
  {
    uint64_t one[K], wout[K];
    one[0] = best;
#pragma unroll
    for (int r = 1; r < K; ++r) one[r] = rank_key(-INFINITY, INT32_MAX);
    wave_topk<K>(one, k, wout);
    if (lane == 0) {
#pragma unroll
      for (int r = 0; r < K; ++r)
        if (r < k) wkey[wave * k + r] = wout[r];
    }
  }
  if (tid == 0) {
    count = 0;
    thr_s = rank_key(-INFINITY, INT32_MAX);   // fewer than k threads hold values: take them all
  }
  __syncthreads();
  if (tid < kWaves * k) {
    const uint64_t e = wkey[tid];
    int rank = 0;
    for (int j = 0; j < kWaves * k; ++j) rank += int(wkey[j] > e);
    if (rank == k - 1) thr_s = e;
  }
  __syncthreads();
  const uint64_t thr = thr_s;
#pragma unroll
  for (int c = 0; c < CH; ++c)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int v = v0 + 4 * tid + 4 * kBlock * c + i;
      if (v < v1) {
        const uint64_t key = rank_key(x[c][i], v);
        if (key >= thr) cand[atomicAdd(&count, 1)] = key;
      }
    }
  __syncthreads();
  Partial q{-INFINITY, 0.f};
#pragma unroll
  for (int w = 0; w < kWaves; ++w) q = combine(q, sp[w], scale);  // fixed order
  const int n = count;
  constexpr int RF = record_floats<K>();
  float* rec = part + (row * nseg + seg) * RF;
  if (nseg > 1 && tid == 0) {
    rec[0] = q.m;
    rec[1] = q.s;
  }
  for (int t = tid; t < n; t += kBlock) {
    const uint64_t key = cand[t];
    int slot = 0;
    for (int j = 0; j < n; ++j) slot += int(cand[j] > key);
    if (nseg == 1) {
      emit_row(row, q, key, slot, k, tau, lse, cand_logp, cand_ids);
    } else if (slot < k) {
      rec[4 + slot] = key_value(key);
      rec[4 + K + slot] = __int_as_float(key_id(key));
    }
  }
}

// grid: rows * nseg blocks, block = row * nseg + segment.  One segment per
// row writes the result directly; otherwise every block writes its segment's
// record for lse_topk_merge.
// CH float4 loads in flight per thread (at most 8: the candidate bitmask has
// 32 bits); NTL: non-temporal loads (many rows: z is far larger than the caches).
template <int K, bool VEC, int CH, bool NTL>
__global__ __launch_bounds__(kBlock) void lse_topk_rows(const float* __restrict__ z, int vocab,
                                                        int nseg, int seg_len, int k, float tau,
                                                        float* lse, float* cand_logp,
                                                        int32_t* cand_ids, float* part) {
  static_assert(CH >= 1 && CH <= 8, "bitmask holds 32 candidates");
  // per-thread staging row for the (rare) chunks that reach the top-K list
  __shared__ float stage[kBlock][4 * CH + 1];
  const int64_t row = blockIdx.x / nseg;
  const int seg = blockIdx.x % nseg;
  const int v0 = seg * seg_len;
  const int v1 = min(vocab, v0 + seg_len);
  const float* zr = z + row * int64_t(vocab);
  const float scale = kLog2e / tau;
  const int tid = threadIdx.x;

  Partial p{-INFINITY, 0.f};
  if constexpr (VEC && !NTL) {
    if (v1 - v0 <= 4 * kBlock * CH) {
      // the whole segment in one pass of loads (few rows: cache-resident z)
      segment_in_registers<K, CH, NTL>(zr, v0, v1, nseg, k, tau, scale, row, seg, lse, cand_logp, cand_ids, part);
      return;
    }
  }
  float tv[K];
  int ti[K];
#pragma unroll
  for (int r = 0; r < K; ++r) { tv[r] = -INFINITY; ti[r] = INT32_MAX; }

  if constexpr (VEC) {
    // Thread tid visits, per iteration, float4 c at base + 4 kBlock c: ids
    // ascend along the traversal.  The first float4 of an iteration is always
    // in range, so the running max is finite before any -inf padding is summed.
    for (int base = v0 + 4 * tid; base < v1; base += 4 * kBlock * CH) {
      f32x4 x[CH];
#pragma unroll
      for (int c = 0; c < CH; ++c) {
        const int v = base + 4 * kBlock * c;
        const f32x4* src = reinterpret_cast<const f32x4*>(zr + v);
        x[c] = v < v1 ? (NTL ? __builtin_nontemporal_load(src) : *src) : f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      }
      float mx = -INFINITY;
#pragma unroll
      for (int c = 0; c < CH; ++c) mx = fmaxf(mx, fmaxf(fmaxf(x[c][0], x[c][1]), fmaxf(x[c][2], x[c][3])));
      if (mx > p.m) {
        p.s *= __builtin_amdgcn_exp2f((p.m - mx) * scale);
        p.m = mx;
      }
      float acc = 0.f;
#pragma unroll
      for (int c = 0; c < CH; ++c)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc += __builtin_amdgcn_exp2f((x[c][i] - p.m) * scale);
      p.s += acc;
      if (mx > tv[K - 1]) {
        // only this lane's values above its current K-th are visited, in id order
        const float thr = tv[K - 1];
        uint32_t mask = 0;
#pragma unroll
        for (int c = 0; c < CH; ++c)
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

// The register-resident path alone, for segments known to fit one pass:
// without the streaming path's staging rows its LDS is a few KB, so more
// blocks fit on a compute unit (the 1216 segments of 64 rows x 151936 are
// resident at once instead of 1024 and a second wave).
template <int K, int CH>
__global__ __launch_bounds__(kBlock) void lse_topk_regs(const float* __restrict__ z, int vocab, int nseg,
                                                        int seg_len, int k, float tau, float* lse,
                                                        float* cand_logp, int32_t* cand_ids, float* part) {
  const int64_t row = blockIdx.x / nseg;
  const int seg = blockIdx.x % nseg;
  const int v0 = seg * seg_len;
  const int v1 = min(vocab, v0 + seg_len);
  segment_in_registers<K, CH, false>(z + row * int64_t(vocab), v0, v1, nseg, k, tau, kLog2e / tau, row, seg, lse,
                                     cand_logp, cand_ids, part);
}

// Segments per row (at most 64: one record per lane when a wave merges a
// row).  Up to 16 rows: about 1024 blocks (four per CU), no segment shorter
// than 2048 elements.  17..511 rows: segments of at most 8192 elements, each
// held in registers in one pass (measured at 32 and 64 rows x 151936: 19
// segments per row 15.4 / 21.6 us per launch, against 32 / 16 segments
// streamed in 4096-element passes, 19.0 / 24.0 us, and 38 segments of 4000
// in registers, 19.0 / 28.2 us).  From 512 rows one segment per row.
int num_segments(int64_t rows, int64_t vocab) {
  if (rows > 16 && rows < 512)
    return int(std::max<int64_t>(1, std::min<int64_t>((vocab + kMidSegment - 1) / kMidSegment, 64)));
  const int64_t want = (1024 + rows - 1) / rows;
  const int64_t most = std::min<int64_t>((vocab + 2047) / 2048, 64);
  return int(std::max<int64_t>(1, std::min(want, most)));
}

template <int K>
hipError_t launch_k(const float* z, int64_t rows, int64_t vocab, int k, float tau, float* lse,
                    float* cand_logp, int32_t* cand_ids, float* part, bool merge, hipStream_t s) {
  const int nseg = num_segments(rows, vocab);
  const bool vec = (vocab % 4) == 0 && (reinterpret_cast<uintptr_t>(z) % 16) == 0;
  int seg_len = int((vocab + nseg - 1) / nseg);
  if (vec) seg_len = (seg_len + 3) & ~3;
  const dim3 grid(unsigned(rows * nseg));
  if (vec && rows >= 512)  // z (R V floats) far exceeds the caches: stream it, 8 float4 per thread in flight
    hipLaunchKernelGGL((lse_topk_rows<K, true, 8, true>), grid, dim3(kBlock), 0, s, z, int(vocab), nseg, seg_len, k,
                       tau, lse, cand_logp, cand_ids, part);
  else if (vec && rows > 16 && seg_len <= kMidSegment)  // one pass of 8 float4 per thread, held in registers
    hipLaunchKernelGGL((lse_topk_regs<K, 8>), grid, dim3(kBlock), 0, s, z, int(vocab), nseg, seg_len, k, tau, lse,
                       cand_logp, cand_ids, part);
  else if (vec)
    hipLaunchKernelGGL((lse_topk_rows<K, true, 4, false>), grid, dim3(kBlock), 0, s, z, int(vocab), nseg, seg_len, k,
                       tau, lse, cand_logp, cand_ids, part);
  else
    hipLaunchKernelGGL((lse_topk_rows<K, false, 4, false>), grid, dim3(kBlock), 0, s, z, int(vocab), nseg, seg_len, k,
                       tau, lse, cand_logp, cand_ids, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || nseg == 1 || !merge) return e;
  hipLaunchKernelGGL((lse_topk_merge<K>), dim3(unsigned(rows)), dim3(kBlock), 0, s, nseg, k, tau, part, lse,
                     cand_logp, cand_ids);
  return hipGetLastError();
}

}  // namespace

int lse_topk_segments(int64_t rows, int64_t vocab) { return num_segments(rows, vocab); }

size_t lse_topk_scratch_bytes(int64_t rows, int64_t vocab, int k) {
  const int nseg = num_segments(rows, vocab);
  if (nseg == 1) return 0;
  return size_t(rows) * nseg * size_t(record_floats_of(topk_bucket(k))) * sizeof(float);
}

hipError_t launch_lse_topk(const float* z, int64_t rows, int64_t vocab, int k, float tau, float* lse,
                           float* cand_logp, int32_t* cand_ids, void* scratch, bool merge, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  float* part = static_cast<float*>(scratch);
  switch (topk_bucket(k)) {
    case 1: return launch_k<1>(z, rows, vocab, k, tau, lse, cand_logp, cand_ids, part, merge, s);
    case 2: return launch_k<2>(z, rows, vocab, k, tau, lse, cand_logp, cand_ids, part, merge, s);
    case 4: return launch_k<4>(z, rows, vocab, k, tau, lse, cand_logp, cand_ids, part, merge, s);
    case 8: return launch_k<8>(z, rows, vocab, k, tau, lse, cand_logp, cand_ids, part, merge, s);
    case 16: return launch_k<16>(z, rows, vocab, k, tau, lse, cand_logp, cand_ids, part, merge, s);
    default: return launch_k<32>(z, rows, vocab, k, tau, lse, cand_logp, cand_ids, part, merge, s);
  }
}

}  // namespace dartree

// ---------------------------------------------------------------------------
// dartree_lse_topk without a workspace argument and without allocating: the
// segment records live in `scratch`, a device array of the library that each
// GPU holds until the process ends.  Its address on a device comes from
// hipGetSymbolAddress, taken once per device with that device current (the
// array's name in host code is not a device address).
// ---------------------------------------------------------------------------
namespace {

// rows * segments <= 2047 whenever a row is split (a split needs fewer than
// 1024 rows, and then rows * ceil(1024 / rows) < 2048), times the largest
// record (68 floats at k <= 32): 556784 bytes of every valid call fit.
static_assert(2047 * dartree::record_floats_of(32) * 4 <= DARTREE_LSE_TOPK_STATIC_SCRATCH_BYTES,
              "static scratch too small for the largest split");
static __device__ __align__(256) float scratch[DARTREE_LSE_TOPK_STATIC_SCRATCH_BYTES / sizeof(float)];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// The current device's address of `scratch` (nullptr on failure).
void* scratch_on_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" dartree_status dartree_lse_topk_noalloc(const float* z, int32_t rows, int32_t vocab, int32_t k,
                                                   float temperature, float* lse, float* cand_logp,
                                                   int32_t* cand_ids, hipStream_t stream) {
  size_t need = 0;
  dartree_status v = dartree_lse_topk_workspace_size(rows, vocab, k, &need);
  if (v != DARTREE_OK) return v;
  if (!__builtin_isfinite(temperature) || temperature < 0.f) return DARTREE_ERR_INVALID_ARG;
  if (!z || !lse || !cand_logp || !cand_ids) return DARTREE_ERR_INVALID_ARG;
  if (need > DARTREE_LSE_TOPK_STATIC_SCRATCH_BYTES) return DARTREE_ERR_UNSUPPORTED;
  void* ptr = need > 0 ? scratch_on_current_device() : nullptr;
  if (need > 0 && !ptr) return DARTREE_ERR_HIP;
  const float tau = temperature > 0.f ? temperature : 1.f;
  return dartree::launch_lse_topk(z, rows, vocab, k, tau, lse, cand_logp, cand_ids, ptr, true, stream) == hipSuccess
             ? DARTREE_OK
             : DARTREE_ERR_HIP;
}
