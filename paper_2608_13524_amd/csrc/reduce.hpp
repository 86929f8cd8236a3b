// Device-side reduction helpers shared by the softmax/top-k kernels and the
// level-selection kernel: online (max, sum of exponentials) pairs, sorted
// per-lane top-K lists, 64-bit ranking keys and DPP wavefront reductions.
#pragma once

#include "internal.hpp"

namespace dartree {

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

// Top-K bucket of a branching factor k (the template instance serving it).
__host__ __device__ constexpr int topk_bucket(int k) {
  return k <= 1 ? 1 : k <= 2 ? 2 : k <= 4 ? 4 : k <= 8 ? 8 : k <= 16 ? 16 : 32;
}

// Partial record of one row segment: m, s, two pad words, K values, K ids.
__host__ __device__ constexpr int record_floats_of(int K) { return (4 + 2 * K + 3) & ~3; }
template <int K>
__host__ __device__ constexpr int record_floats() { return record_floats_of(K); }

// Top K of two lists of K ranking keys, each sorted descending, into `a`
// (sorted descending): the elementwise larger of a and reversed b is a
// bitonic sequence holding the K largest keys, which log2(K) half-cleaner
// stages sort.
template <int K>
__device__ __forceinline__ void merge_sorted_keys(uint64_t (&a)[K], const uint64_t (&b)[K]) {
#pragma unroll
  for (int i = 0; i < K; ++i) a[i] = a[i] > b[K - 1 - i] ? a[i] : b[K - 1 - i];
#pragma unroll
  for (int stride = K / 2; stride > 0; stride >>= 1)
#pragma unroll
    for (int i = 0; i < K; ++i)
      if ((i & stride) == 0) {
        const uint64_t x = a[i], y = a[i + stride];
        a[i] = x > y ? x : y;
        a[i + stride] = x > y ? y : x;
      }
}

// Merge the nseg records of one row over a wave: lane l takes records l,
// l + 64, ... (16-byte loads, all issued together); a record's list is
// already in rank order, so a lane keeps its first record's list and merges
// later ones into it.  Must be called by all 64 lanes of a wave; `recs` is
// 16-byte aligned.  Returns the row's Partial (wave-uniform) and its top-k
// keys in out[0 .. k) (wave-uniform).
template <int K>
__device__ __forceinline__ Partial wave_merge_records(const float* recs, int nseg, int k, float scale,
                                                      uint64_t (&out)[K]) {
  constexpr int RF = record_floats<K>();
  const int lane = threadIdx.x & 63;
  const uint64_t empty = rank_key(-INFINITY, INT32_MAX);
  Partial p{-INFINITY, 0.f};
  uint64_t key[K];
#pragma unroll
  for (int r = 0; r < K; ++r) key[r] = empty;
#pragma unroll 1
  for (int sg = lane; sg < nseg; sg += 64) {
    f32x4 rv[RF / 4];
    const f32x4* rp = reinterpret_cast<const f32x4*>(recs + int64_t(sg) * RF);
#pragma unroll
    for (int i = 0; i < RF / 4; ++i) rv[i] = rp[i];
    p = combine(p, Partial{rv[0][0], rv[0][1]}, scale);
    uint64_t rk[K];
#pragma unroll
    for (int r = 0; r < K; ++r)
      rk[r] = r < k ? rank_key(rv[(4 + r) / 4][(4 + r) % 4], __float_as_int(rv[(4 + K + r) / 4][(4 + K + r) % 4]))
                    : empty;
    merge_sorted_keys<K>(key, rk);
  }
  const Partial wp = wave_partial(p, scale);
  wave_topk<K>(key, k, out);
  return wp;
}

// Ascending bitonic sort of npad (a power of two, >= 2) keys in LDS by the
// whole block; returns after a barrier.
__device__ inline void bitonic_sort(uint64_t* keys, int npad) {
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

__host__ __device__ inline int next_pow2(int n) {
  int p = 2;
  while (p < n) p <<= 1;
  return p;
}

}  // namespace dartree
