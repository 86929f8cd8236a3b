// Correction-head products of one depth (Algorithm 1, "correct all prefixes
// in parallel"): for every node row m of S_{d-1}
//   head    : t[m] = A r[m],  a[m] = act(tanh(t[m] + H_d))      (N = h)
//   logits  : z[m] = L_d^base + U a[m]                            (N = V)
// Both are out[m][n] = f(sum_k x[m][k] w[n][k]) with w = A or U stored
// [N][K] row-major (K contiguous), so one family of kernels serves both.
//
// bf16 path, gfx950 MFMA v_mfma_f32_16x16x32_bf16 (fp32 accumulation):
//  * proj_bf16_stream: few rows (M <= 64; against the vocabulary M <= 16).
//    The product is a stream over the weight matrix (U is 0.78-1.56 GB per
//    depth, far beyond the caches), so every weight element is read once from
//    HBM with coalesced non-temporal loads and staged through LDS into MFMA
//    operand layout.
//  * proj_bf16_sweep: 17..64 rows against the vocabulary.  One wave per run
//    of weight tiles, accumulating them over the whole K loop; the weights
//    and node rows stream into the wave's own LDS by buffer loads.
//  * proj_bf16_hsplit: the head at 17..64 rows.  64 weight rows per block
//    and K split into pieces, the piece's node rows staged once in LDS for
//    the block's four tiles; a fix-up launch adds the pieces in order.
//  * proj_bf16_big: many rows (>= 512) against the vocabulary, and the head at
//    >= 512 rows when its tiles are too few to fill the chip.  256x256 tiles,
//    8 waves in two groups alternating LDS reads and MFMAs, buffer loads
//    straight to swizzled LDS, XCD-aware tile order; the tiles of a last
//    partial wave are split along K into pieces whose partial sums a fix-up
//    kernel adds in piece order.
//  * proj_bf16_tiled: other many-row products (the head, or a few hundred
//    rows).  128x128 output tiles, 64-deep K steps staged through
//    double-buffered, padded LDS tiles shared by 4 waves (64x64 each).
// fp32 path: plain FMA loop (small problems only).

#include <algorithm>
#include <type_traits>
#include <utility>

#include "internal.hpp"

namespace dartree {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct KArgs {
  const void* x;
  const void* w;
  int M, N, K;
  int rows_per_group;
  int64_t bias_stride;
  const float* bias_f32;
  const void* bias_act;
  const int32_t* group_index;
  float* out;
  void* act_out;
};

// first element of row m's bias row
__device__ __forceinline__ int64_t bias_base(const KArgs& a, int m) {
  const int g = m / a.rows_per_group;
  return int64_t(a.group_index ? a.group_index[g] : g) * a.bias_stride;
}

// NTS: logits stored with non-temporal stores (outputs far beyond the caches).
template <int EPI, bool BF16, bool NTS = false>
__device__ __forceinline__ void emit(const KArgs& a, int m, int n, float acc) {
  const int64_t bb = bias_base(a, m);
  const int64_t o = int64_t(m) * a.N + n;
  if constexpr (EPI == EPI_LOGITS) {
    if constexpr (NTS) __builtin_nontemporal_store(acc + a.bias_f32[bb + n], a.out + o);
    else a.out[o] = acc + a.bias_f32[bb + n];
  } else {
    a.out[o] = acc;
    float hb;
    if constexpr (BF16) hb = bf16_to_f32(static_cast<const uint16_t*>(a.bias_act)[bb + n]);
    else hb = static_cast<const float*>(a.bias_act)[bb + n];
    const float v = tanhf(acc + hb);
    if constexpr (BF16) static_cast<uint16_t*>(a.act_out)[o] = f32_to_bf16(v);
    else static_cast<float*>(a.act_out)[o] = v;
  }
}

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
typedef float f32x16 __attribute__((ext_vector_type(16)));
// v_mfma_f32_32x32x16_bf16: lane l supplies row l % 32 and the 8 consecutive
// k at 8 (l / 32) of each operand; element v of lane l's result is
// D[8 (v / 4) + 4 (l / 32) + v % 4][l % 32], D[i][j] = sum_k A[i][k] B[j][k].
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// Few rows: weight streaming through LDS-staged tiles.
//
// MFMA operand A = 16 weight rows (output n), operand B = 16 node rows
// (output m); lane l supplies row (l & 15) and the 8 consecutive k at
// (l >> 4) * 8 of each 32-deep step, so a direct operand load would touch 16
// rows x 64 B per instruction (half cache lines).  Instead each wave moves a
// 16*NT-row x 64-k chunk (128 B per row) with fully coalesced non-temporal
// loads (lane l: row l / 8, 16-byte piece l % 8) into its private LDS slot,
// XOR-swizzled by row so that both these writes and the operand reads are
// bank-conflict free, and reads the operands back from LDS.  Chunks are
// prefetched D ahead in registers.  The result lane l holds
// D[n = 4 (l >> 4) + i][m = l & 15], i = 0..3.
//
// A block owns 16*NT weight rows; its KW waves split K into contiguous ranges
// of 64-k chunks and are summed through LDS in wave order.  The node rows
// (the B operand, at most 64 x h) are small and stay in the caches.
// ---------------------------------------------------------------------------
__device__ __forceinline__ u32x4 ld_stream(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ u32x4 ld_cached(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ int lds_swizzle(int row) { return (row ^ (row >> 3)) & 7; }

typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));

// The four bias values of outputs (m, n..n+3) as fp32 (vector path only).
template <int EPI>
__device__ __forceinline__ f32x4 bias4(const KArgs& a, int m, int n) {
  const int64_t bb = bias_base(a, m) + n;
  if constexpr (EPI == EPI_LOGITS) return *reinterpret_cast<const f32x4*>(a.bias_f32 + bb);
  const u16x4 hb = *reinterpret_cast<const u16x4*>(static_cast<const uint16_t*>(a.bias_act) + bb);
  return f32x4{bf16_to_f32(hb[0]), bf16_to_f32(hb[1]), bf16_to_f32(hb[2]), bf16_to_f32(hb[3])};
}

// emit4's vector path with the bias already loaded (the same arithmetic).
template <int EPI>
__device__ __forceinline__ void emit4_bias(const KArgs& a, int m, int n, f32x4 v, f32x4 b) {
  const int64_t o = int64_t(m) * a.N + n;
  if constexpr (EPI == EPI_LOGITS) {
    *reinterpret_cast<f32x4*>(a.out + o) = v + b;
  } else {
    *reinterpret_cast<f32x4*>(a.out + o) = v;
    u16x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = f32_to_bf16(tanhf(v[i] + b[i]));
    *reinterpret_cast<u16x4*>(static_cast<uint16_t*>(a.act_out) + o) = r;
  }
}

template <int EPI, bool NTS = false>
__device__ __forceinline__ void emit4(const KArgs& a, int m, int n, f32x4 v, bool vec) {
  const int64_t bb = bias_base(a, m);
  const int64_t o = int64_t(m) * a.N + n;
  if (vec && n + 3 < a.N) {
    if constexpr (EPI == EPI_LOGITS) {
      const f32x4 b = *reinterpret_cast<const f32x4*>(a.bias_f32 + bb + n);
      if constexpr (NTS) __builtin_nontemporal_store(v + b, reinterpret_cast<f32x4*>(a.out + o));
      else *reinterpret_cast<f32x4*>(a.out + o) = v + b;
    } else {
      const u16x4 hb = *reinterpret_cast<const u16x4*>(static_cast<const uint16_t*>(a.bias_act) + bb + n);
      *reinterpret_cast<f32x4*>(a.out + o) = v;
      u16x4 r;
#pragma unroll
      for (int i = 0; i < 4; ++i) r[i] = f32_to_bf16(tanhf(v[i] + bf16_to_f32(hb[i])));
      *reinterpret_cast<u16x4*>(static_cast<uint16_t*>(a.act_out) + o) = r;
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (n + i < a.N) emit<EPI, true, NTS>(a, m, n + i, v[i]);
}

template <int MT, int NT, int KW, int D, int EPI>
__global__ __launch_bounds__(64 * KW) void proj_bf16_stream(KArgs a, int vec) {
  // staging slots during the stream, then the cross-wave partial sums
  constexpr int kSlotBytes = KW * 16 * NT * 64 * 2;
  constexpr int kRedBytes = KW * NT * MT * 64 * 16;
  __shared__ __attribute__((aligned(16))) uint8_t smem[kSlotBytes > kRedBytes ? kSlotBytes : kRedBytes];
  auto slot = reinterpret_cast<uint16_t(*)[16 * NT * 64]>(smem);
  auto red = reinterpret_cast<f32x4(*)[NT * MT][64]>(smem);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int lr = lane >> 3, lc = lane & 7;
  const int n0 = blockIdx.x * (16 * NT);
  const int M = a.M, N = a.N, K = a.K;
  const uint16_t* X = static_cast<const uint16_t*>(a.x);
  const uint16_t* Wt = static_cast<const uint16_t*>(a.w);

  // Rows past M or N are clamped to the last row: their sums are computed and
  // never stored.
  const uint16_t* wg[2 * NT];
  int woff[2 * NT];
#pragma unroll
  for (int i = 0; i < 2 * NT; ++i) {
    const int row = 8 * i + lr;
    wg[i] = Wt + int64_t(min(n0 + row, N - 1)) * K + lc * 8;
    woff[i] = row * 64 + (lc ^ lds_swizzle(row)) * 8;
  }
  int roff[2][NT];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int row = nt * 16 + r16;
      roff[j][nt] = row * 64 + ((4 * j + kg) ^ lds_swizzle(row)) * 8;
    }
  const uint16_t* xp[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) xp[mt] = X + int64_t(min(mt * 16 + r16, M - 1)) * K + kg * 8;

  // When every wave emits at most one 16x16 tile, its lanes fetch their
  // bias values now, so the epilogue does not wait on a last dependent load.
  constexpr bool kPre = NT * MT <= KW;
  f32x4 pre_b = f32x4{0.f, 0.f, 0.f, 0.f};
  bool pre_ok = false;
  if constexpr (kPre) {
    if (wave < NT * MT) {
      const int m = (wave % MT) * 16 + r16, n = n0 + (wave / MT) * 16 + kg * 4;
      pre_ok = vec != 0 && m < M && n + 3 < N;
      if (pre_ok) pre_b = bias4<EPI>(a, m, n);
    }
  }

  const int chunks = K >> 6;
  const int per = (chunks + KW - 1) / KW;
  const int c0 = min(chunks, wave * per);
  const int n = min(chunks, c0 + per) - c0;
  uint16_t* sl = slot[wave];

  f32x4 acc[NT][MT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[nt][mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 R[D][2 * NT], XR[D][2][MT];
  auto fetch = [&](int d, int k) {
#pragma unroll
    for (int i = 0; i < 2 * NT; ++i) R[d][i] = ld_stream(wg[i] + k);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      XR[d][0][mt] = ld_cached(xp[mt] + k);
      XR[d][1][mt] = ld_cached(xp[mt] + k + 32);
    }
  };
#pragma unroll
  for (int d = 0; d < D; ++d)
    if (d < n) fetch(d, (c0 + d) * 64);
  for (int c = 0; c < n; c += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      if (c + d < n) {
#pragma unroll
        for (int i = 0; i < 2 * NT; ++i) *reinterpret_cast<u32x4*>(sl + woff[i]) = R[d][i];
        u32x4 xv[2][MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) { xv[0][mt] = XR[d][0][mt]; xv[1][mt] = XR[d][1][mt]; }
        if (c + d + D < n) fetch(d, (c0 + c + d + D) * 64);
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            const bf16x8 av = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(sl + roff[j][nt]));
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
              acc[nt][mt] = mfma16(av, __builtin_bit_cast(bf16x8, xv[j][mt]), acc[nt][mt]);
          }
      }
    }
  }

  __syncthreads();  // every wave is done with its slot before the sums reuse the memory
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) red[wave][nt * MT + mt][lane] = acc[nt][mt];
  __syncthreads();

  for (int p = wave; p < NT * MT; p += KW) {
    const int nt = p / MT, mt = p % MT;
    f32x4 v = red[0][p][lane];
#pragma unroll
    for (int w = 1; w < KW; ++w) v += red[w][p][lane];
    const int m = mt * 16 + r16;
    if (m < M) {
      if (kPre && pre_ok) emit4_bias<EPI>(a, m, n0 + nt * 16 + kg * 4, v, pre_b);
      else emit4<EPI>(a, m, n0 + nt * 16 + kg * 4, v, vec != 0);
    }
  }
}

// ---------------------------------------------------------------------------
// At most 16 node rows against the vocabulary: blocks of 32 weight rows (two
// 16-row tiles), KW waves splitting K into ranges of 128-deep pairs, partial
// sums added through LDS in wave order.  A wave streams stages of 16 rows x
// 128 k (one tile of one pair, 4 KB: every load instruction covers 4 rows x
// 256 bytes, whole 256-byte row pieces, which stream from HBM faster than
// 128-byte ones), two stages in flight in registers, each written to the
// wave's private LDS slot (16 XOR-swizzled 16-byte positions per 256-byte
// row, conflict-free both ways) and read back in MFMA operand layout for
// v_mfma_f32_16x16x32_bf16 (A = 16 weight rows, B = the node rows).  The
// result lane l holds D[n = 4 (l >> 4) + i][m = l & 15], i = 0..3.
// ---------------------------------------------------------------------------
template <int KW, int EPI>
__global__ __launch_bounds__(64 * KW) void proj_bf16_pairs(KArgs a, int vec) {
  constexpr int NT = 2;
  constexpr int kSlotBytes = KW * 16 * 128 * 2;
  constexpr int kRedBytes = KW * NT * 64 * 16;
  __shared__ __attribute__((aligned(16))) uint8_t smem[kSlotBytes > kRedBytes ? kSlotBytes : kRedBytes];
  auto slot = reinterpret_cast<uint16_t(*)[16 * 128]>(smem);
  auto red = reinterpret_cast<f32x4(*)[NT][64]>(smem);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int n0 = blockIdx.x * (16 * NT);
  const int M = a.M, N = a.N, K = a.K;
  const uint16_t* X = static_cast<const uint16_t*>(a.x);
  const uint16_t* Wt = static_cast<const uint16_t*>(a.w);

  // load instruction i of a stage: tile row 4 i + l / 16, 16-byte piece
  // l % 16 of the row's 256 bytes, stored at position piece ^ row.  Rows
  // past N are clamped to the last row: computed, never stored.
  const uint16_t* wg[NT][4];
  int woff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 4 * i + kg;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) wg[nt][i] = Wt + int64_t(min(n0 + 16 * nt + row, N - 1)) * K + r16 * 8;
    woff[i] = row * 128 + ((r16 ^ row) * 8);
  }
  // operand j (k = 32 j .. 32 j + 31 of the pair) of lane l: row l % 16,
  // piece 4 j + l / 16
  int roff[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) roff[j] = r16 * 128 + (((4 * j + kg) ^ r16) * 8);
  const uint16_t* xp = X + int64_t(min(r16, M - 1)) * K + kg * 8;

  // When every wave emits at most one 16x16 tile, its lanes fetch their
  // bias values now, so the epilogue does not wait on a last dependent load.
  constexpr bool kPre = NT <= KW;
  f32x4 pre_b = f32x4{0.f, 0.f, 0.f, 0.f};
  bool pre_ok = false;
  if constexpr (kPre) {
    if (wave < NT) {
      const int m = r16, n = n0 + wave * 16 + kg * 4;
      pre_ok = vec != 0 && m < M && n + 3 < N;
      if (pre_ok) pre_b = bias4<EPI>(a, m, n);
    }
  }

  // pairs [q0, q0 + np) of this wave
  const int pairs = K >> 7;
  const int per = (pairs + KW - 1) / KW;
  const int q0 = min(pairs, wave * per);
  const int np = min(pairs, q0 + per) - q0;
  uint16_t* sl = slot[wave];

  f32x4 acc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 R[NT][4], XN[4], XR[4];
  // stage (q, nt): tile nt's rows of pair q (and with tile 0, the pair's node rows)
  auto fetch = [&](int q, auto NTc) __attribute__((always_inline)) {
    constexpr int nt = decltype(NTc)::value;
    const int k = q * 128;
#pragma unroll
    for (int i = 0; i < 4; ++i) R[nt][i] = ld_stream(wg[nt][i] + k);
    if constexpr (nt == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) XN[j] = ld_cached(xp + k + 32 * j);
    }
  };
  auto stage = [&](int q, auto NTc, bool more) __attribute__((always_inline)) {
    constexpr int nt = decltype(NTc)::value;
#pragma unroll
    for (int i = 0; i < 4; ++i) *reinterpret_cast<u32x4*>(sl + woff[i]) = R[nt][i];
    if constexpr (nt == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) XR[j] = XN[j];
    }
    if (more) fetch(q + 1, NTc);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bf16x8 av = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(sl + roff[j]));
      acc[nt] = mfma16(av, __builtin_bit_cast(bf16x8, XR[j]), acc[nt]);
    }
  };
  if (np > 0) {
    fetch(q0, std::integral_constant<int, 0>{});
    fetch(q0, std::integral_constant<int, 1>{});
    // every pair but the last fetches the next one (the loads are the same
    // on every pass, so the compiler's waits keep two stages in flight)
#pragma unroll 1
    for (int q = q0; q + 1 < q0 + np; ++q) {
      stage(q, std::integral_constant<int, 0>{}, true);
      stage(q, std::integral_constant<int, 1>{}, true);
    }
    stage(q0 + np - 1, std::integral_constant<int, 0>{}, false);
    stage(q0 + np - 1, std::integral_constant<int, 1>{}, false);
  }

  __syncthreads();  // every wave is done with its slot before the sums reuse the memory
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) red[wave][nt][lane] = acc[nt];
  __syncthreads();

  for (int nt = wave; nt < NT; nt += KW) {
    f32x4 v = red[0][nt][lane];
#pragma unroll
    for (int w = 1; w < KW; ++w) v += red[w][nt][lane];
    const int m = r16;
    if (m < M) {
      if (kPre && pre_ok) emit4_bias<EPI>(a, m, n0 + nt * 16 + kg * 4, v, pre_b);
      else emit4<EPI>(a, m, n0 + nt * 16 + kg * 4, v, vec != 0);
    }
  }
}

// ---------------------------------------------------------------------------
// Many rows: 128x128 output tile per block, K in steps of 64 through
// double-buffered LDS.  Rows are padded to 72 bf16 (144 B) so that the 16-byte
// operand reads of 16 consecutive rows fall in distinct LDS banks.
// ---------------------------------------------------------------------------
constexpr int TBM = 128, TBN = 128, TBK = 64, TLD = TBK + 8;

template <int EPI>
__global__ __launch_bounds__(256) void proj_bf16_tiled(KArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t Xs[2][TBM][TLD];
  __shared__ __attribute__((aligned(16))) uint16_t Ws[2][TBN][TLD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int wm = wave & 1, wn = wave >> 1;
  const int m0 = blockIdx.x * TBM, n0 = blockIdx.y * TBN;
  const int M = a.M, N = a.N, K = a.K;
  const uint16_t* X = static_cast<const uint16_t*>(a.x);
  const uint16_t* Wt = static_cast<const uint16_t*>(a.w);

  // Global -> LDS: thread t moves 16-byte chunk (t & 7) of rows (t >> 3) + 32 i.
  const int lc = (tid & 7) * 8;
  const int lr = tid >> 3;
  const uint16_t* xg[4];
  const uint16_t* wg[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    xg[i] = X + int64_t(min(m0 + lr + 32 * i, M - 1)) * K + lc;
    wg[i] = Wt + int64_t(min(n0 + lr + 32 * i, N - 1)) * K + lc;
  }
  u32x4 xr[4], wr[4];
  auto gload = [&](int kt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      xr[i] = *reinterpret_cast<const u32x4*>(xg[i] + kt * TBK);
      wr[i] = *reinterpret_cast<const u32x4*>(wg[i] + kt * TBK);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *reinterpret_cast<u32x4*>(&Xs[buf][lr + 32 * i][lc]) = xr[i];
      *reinterpret_cast<u32x4*>(&Ws[buf][lr + 32 * i][lc]) = wr[i];
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = K / TBK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
    for (int ks = 0; ks < TBK; ks += 32) {
      bf16x8 av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        av[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(&Ws[buf][wn * 64 + i * 16 + r16][ks + kg * 8]));
#pragma unroll
      for (int j = 0; j < 4; ++j)
        bv[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(&Xs[buf][wm * 64 + j * 16 + r16][ks + kg * 8]));
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma16(av[i], bv[j], acc[i][j]);
    }
    if (kt + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + wm * 64 + j * 16 + r16;
      if (m >= M) continue;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = n0 + wn * 64 + i * 16 + kg * 4 + q;
        if (n < N) emit<EPI, true>(a, m, n, acc[i][j][q]);
      }
    }
}

// ---------------------------------------------------------------------------
// Many rows, long weight matrix (>= 512 node rows): 256x256 output tile per
// block, 8 waves, two per SIMD.  Wave w belongs to group w / 4 (each SIMD runs
// one wave of each group) and owns weight rows [64 (w % 4), +64) x node rows
// [128 (w / 4), +128) of the tile as 2 x 4 tiles of 32x32 (the 32x32x16 MFMA
// reads half the operand bytes per flop of the 16x16x32 one, measured 4-6%
// faster under the power-limited clock).  The groups
// alternate between a memory phase (reading the operand fragments of one
// 64-deep K step from LDS) and a compute phase (the 64 MFMAs of that step),
// one phase apart, so each SIMD always has one wave issuing MFMAs; a barrier
// ends every phase.  Group 0 moves the K steps into LDS with buffer loads
// straight to LDS (XOR-swizzled rows: conflict-free for the MFMA-layout
// reads).  The weight rows stream from HBM and get three LDS stages: step
// s + 2 is issued at the start of the memory phase for step s, into the stage
// of step s - 1, which both groups have finished reading, so each load has two
// steps to land.  The node rows (cache-resident: every weight tile reuses
// them) get two stages and are issued one step ahead.  3 x 32 KB + 2 x 32 KB
// fill the 160 KB of LDS.  Every wave executes the same number of barriers
// (2 nk + 2).  The ragged
// last tile along M or N is shifted back to end at the matrix edge, so every
// loaded row exists; that block stores only the rows the previous tile did
// not cover.  Tiles are ordered so that the blocks of one XCD (blocks are
// dealt to the 8 XCDs round-robin) cover the M-tiles of one weight tile,
// which then stays in that XCD's L2.
//
// One block per CU fits (160 KB of LDS), so T tiles run in ceil(T / CUs)
// waves and a last partial wave of r tiles leaves the other CUs idle.  Those
// r tiles are split along K into S = min(CUs / r, steps / 4) pieces: block
// (tile, piece) multiplies its contiguous range of K steps and stores the raw
// 256x256 fp32 partial sum; proj_big_fixup then adds the S partials of every
// element in piece order (deterministic) and applies the epilogue.
// ---------------------------------------------------------------------------
constexpr int GBM = 256, GBN = 256, GBK = 64;
#define LDS_AS __attribute__((address_space(3)))

__device__ __forceinline__ int swz16(int r) { return (r ^ (r >> 3)) & 7; }  // r in 0..15

// Tiles [0, full) whole; tiles [full, full + rem) in `pieces` K pieces whose
// partial sums go to split[(r * pieces + piece) * 256 * 256 ..] (row-major
// 256 x 256 fp32 relative to the tile's loaded origin).
struct BigPlan {
  int full, rem, pieces;
  float* split;
};

// Output origin (m0, n0) of tile t (N-tile major, M-tile minor) and the origin
// (ml, nl) of the rows it loads: the ragged last tile is shifted back to end
// at the matrix edge (M, N >= 256).
struct BigTile {
  int m0, n0, ml, nl;
};
__device__ __forceinline__ BigTile big_tile(int M, int N, int t) {
  const int ntm = (M + GBM - 1) / GBM;
  BigTile b;
  b.n0 = (t / ntm) * GBN;
  b.m0 = (t % ntm) * GBM;
  b.nl = min(b.n0, N - GBN);
  b.ml = min(b.m0, M - GBM);
  return b;
}

// Work item of block b among n: XCD x (b % 8) gets the contiguous run
// [x q8, (x + 1) q8), q8 = n / 8, so its blocks share operand rows in its L2.
__device__ __forceinline__ int xcd_order(int b, int n) {
  const int q8 = n / 8;
  return b < 8 * q8 ? (b % 8) * q8 + b / 8 : b;
}

template <int EPI>
__global__ __launch_bounds__(512) void proj_bf16_big(KArgs a, int vec, BigPlan pl) {
  constexpr int kStage = GBN * GBK;  // elements of one 256-row, 64-deep stage
  __shared__ __attribute__((aligned(16))) uint16_t smem[5 * kStage];  // W stages 0..2, X stages 0..1
  const int lane = threadIdx.x & 63, r32 = lane & 31, kh = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int grp = wave >> 2, q = wave & 3;
  const int M = a.M, N = a.N, K = a.K;
  const int nk_all = K / GBK;
  int t, ks = 0, nk = nk_all, slot = -1;  // K steps [ks, ks + nk); slot >= 0: a piece of a split tile
  if (int(blockIdx.x) < pl.full) {
    t = xcd_order(blockIdx.x, pl.full);
  } else {
    // pieces ordered piece-major, so the M-tiles of one weight tile at one
    // piece are consecutive items (and land on one XCD)
    const int item = xcd_order(int(blockIdx.x) - pl.full, pl.rem * pl.pieces);
    const int piece = item / pl.rem, r = item % pl.rem;
    t = pl.full + r;
    ks = piece * nk_all / pl.pieces;
    nk = (piece + 1) * nk_all / pl.pieces - ks;
    slot = r * pl.pieces + piece;
  }
  const BigTile tl = big_tile(M, N, t);
  const int m0 = tl.m0, n0 = tl.n0, ml = tl.ml, nl = tl.nl;
  const uint16_t* X = static_cast<const uint16_t*>(a.x);
  const uint16_t* Wt = static_cast<const uint16_t*>(a.w);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(Wt + int64_t(nl) * K), (short)0, GBN * K * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(X + int64_t(ml) * K), (short)0, GBM * K * 2, 0x00020000);
  const bool wload = q < 2;
  const __amdgpu_buffer_rsrc_t rs = wload ? rw : rx;
  // group 0 wave q moves rows [128 (q % 2), +128) of the weight stage (q < 2)
  // or of the node stage, 8 rows per load: lane / 8 is the row, LDS chunk
  // lane % 8 holds global chunk (lane % 8) ^ swizzle(row)
  const int lrow = lane >> 3, lcp = lane & 7;
  const unsigned vo0 = unsigned(lrow * K * 2 + ((lcp ^ swz16(lrow)) * 16));
  const unsigned vo1 = unsigned(lrow * K * 2 + ((lcp ^ swz16(8 + lrow)) * 16));
  const int sw = swz16(r32 & 15);

  // wave tile: weight rows 64 q + 32 i + (0..31) x node rows 128 grp + 32 j +
  // (0..31); each MFMA takes the node rows as its first operand, so that it
  // produces out[m][n] with n = the lane (see the epilogue)
  f32x16 acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  auto dma = [&](int kt) {
    const int stage = wload ? kt % 3 : 3 + (kt & 1);
    LDS_AS uint16_t* base = (LDS_AS uint16_t*)smem + stage * kStage + 128 * (q & 1) * GBK;  // generic -> LDS
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const unsigned so = unsigned((128 * (q & 1) + 8 * i) * K * 2 + (ks + kt) * GBK * 2);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (LDS_AS void*)(base + 8 * i * GBK), 16, (i & 1) ? vo1 : vo0, so, 0,
                                               0);
    }
  };
  // four 16-deep sub-steps per 64-deep step: lane l reads row l % 32, chunk
  // 2 sub + l / 32 of the swizzled LDS row
  bf16x8 A[4][2], B[4][4];
  auto fetch = [&](int st) {
    const LDS_AS uint16_t* Sw = (const LDS_AS uint16_t*)smem + (st % 3) * kStage;
    const LDS_AS uint16_t* Sx = (const LDS_AS uint16_t*)smem + (3 + (st & 1)) * kStage;
#pragma unroll
    for (int sub = 0; sub < 4; ++sub) {
      const int c = ((2 * sub + kh) ^ sw) * 8;
#pragma unroll
      for (int i = 0; i < 2; ++i)
        A[sub][i] =
            __builtin_bit_cast(bf16x8, *reinterpret_cast<const LDS_AS u32x4*>(Sw + (64 * q + 32 * i + r32) * GBK + c));
#pragma unroll
      for (int j = 0; j < 4; ++j)
        B[sub][j] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const LDS_AS u32x4*>(Sx + (128 * grp + 32 * j + r32) * GBK + c));
    }
  };
  auto compute = [&]() {
#pragma unroll
    for (int sub = 0; sub < 4; ++sub)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma32(B[sub][j], A[sub][i], acc[i][j]);
  };
  // A bare barrier: the workgroup fence of __syncthreads would also wait for
  // the loads still in flight for the next step.  The waits that the data
  // dependencies need are explicit.
  auto barrier = [] { asm volatile("s_barrier" ::: "memory"); };
  auto wait_lds_reads = [] { __builtin_amdgcn_s_waitcnt(0xC07F); };  // lgkmcnt(0)
  auto wait_loads = [] { __builtin_amdgcn_s_waitcnt(0x0F70); };      // vmcnt(0)

  if (grp == 0) {
    // weights: steps 0..2 into their three stages, nodes: steps 0..1; wait for
    // step 0 with the later ones (16 loads each) still in flight
    const int ahead = min(wload ? 2 : 1, nk - 1);
    for (int kt = 0; kt <= ahead; ++kt) dma(kt);
    if (ahead == 2) __builtin_amdgcn_s_waitcnt(0x8F70);       // vmcnt(32)
    else if (ahead == 1) __builtin_amdgcn_s_waitcnt(0x4F70);  // vmcnt(16)
    else wait_loads();
  }
  barrier();  // step 0 in LDS
  if (grp == 0) {
    for (int st = 0; st < nk; ++st) {
      if (st >= 1) {
        const int kt = st + (wload ? 2 : 1);
        if (kt < nk) dma(kt);
      }
      fetch(st);
      wait_lds_reads();
      barrier();  // end of phase 2 st
      __builtin_amdgcn_sched_barrier(0);
      compute();
      __builtin_amdgcn_sched_barrier(0);
      // this wave's share of step st + 1 landed (a weight wave may keep step st + 2 in flight)
      if (wload && st + 2 < nk) __builtin_amdgcn_s_waitcnt(0x4F70);  // vmcnt(16)
      else if (st + 1 < nk) wait_loads();
      barrier();  // end of phase 2 st + 1
    }
    barrier();  // phase 2 nk: group 1 multiplies the last step
  } else {
    barrier();  // phase 0: group 0 reads step 0
    for (int st = 0; st < nk; ++st) {
      fetch(st);
      wait_lds_reads();
      barrier();  // end of phase 2 st + 1
      __builtin_amdgcn_sched_barrier(0);
      compute();
      __builtin_amdgcn_sched_barrier(0);
      barrier();  // end of phase 2 st + 2
    }
  }

  // element v of acc[i][j] in lane l is out[m][n] at node row m = 128 grp +
  // 32 j + 8 (v / 4) + 4 (l / 32) + v % 4 and weight row n = 64 q + 32 i +
  // l % 32: the 32 lanes of a half-wave hold 32 consecutive n of one m, so
  // every store instruction writes whole 128-byte lines.  The logits, far
  // beyond the caches and read back right away by the softmax pass, are
  // stored non-temporally (whole lines written around the caches read back
  // at the rate of data not written recently).
  (void)vec;
  if (slot >= 0) {
    float* P = pl.split + size_t(slot) * (GBM * GBN);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          P[(128 * grp + 32 * j + 8 * (v >> 2) + 4 * kh + (v & 3)) * GBN + 64 * q + 32 * i + r32] = acc[i][j][v];
    return;
  }
  // one bias row per 32-row block when the row groups are multiples of 32
  const bool block_bias = a.rows_per_group % 32 == 0;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int n = nl + 64 * q + 32 * i + r32;
    const bool n_new = n >= n0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int mb = ml + 128 * grp + 32 * j;
      if (mb + 31 < m0) continue;
      if (block_bias) {
        const int64_t bb = bias_base(a, mb) + n;
        if constexpr (EPI == EPI_LOGITS) {
          const float b = n_new ? a.bias_f32[bb] : 0.f;
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int m = mb + 8 * (v >> 2) + 4 * kh + (v & 3);
            if (m >= m0 && n_new) __builtin_nontemporal_store(acc[i][j][v] + b, a.out + int64_t(m) * N + n);
          }
        } else {
          const float hb = n_new ? bf16_to_f32(static_cast<const uint16_t*>(a.bias_act)[bb]) : 0.f;
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int m = mb + 8 * (v >> 2) + 4 * kh + (v & 3);
            if (m >= m0 && n_new) {
              const int64_t o = int64_t(m) * N + n;
              a.out[o] = acc[i][j][v];
              static_cast<uint16_t*>(a.act_out)[o] = f32_to_bf16(tanhf(acc[i][j][v] + hb));
            }
          }
        }
      } else {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int m = mb + 8 * (v >> 2) + 4 * kh + (v & 3);
          if (m >= m0 && n_new) emit<EPI, true, EPI == EPI_LOGITS>(a, m, n, acc[i][j][v]);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Many rows, wide node tiles: 512 node rows x 128 weight rows per block (the
// same 256 KB of accumulators as 256 x 256), 8 waves, two per SIMD, each
// 64 node rows x 128 weight rows (2 x 4 tiles of 32x32).  Only the weights go
// through LDS: 16 KB per 64-deep step, a ring of WAHEAD + WBAR stages filled
// WAHEAD steps ahead with buffer loads straight to swizzled LDS, one barrier
// every WBAR steps.  Each wave loads its own node-row fragments into registers
// one step ahead, from a copy of the node rows rearranged into fragment order
// (1 KB contiguous per load).  Per step the LDS carries 16 KB of fills and
// 128 KB of fragment reads (the 256x256 kernel: 64 KB and 192 KB).
// ---------------------------------------------------------------------------
constexpr int WBM = 512, WBN = 128;
constexpr int WAHEAD = 6, WBAR = 2;

// N-tile major: the node tiles of one weight tile are consecutive tiles, so
// they run at the same time on one XCD and share the weights in its L2.
__device__ __forceinline__ BigTile wide_tile(int M, int N, int t) {
  const int ntm = (M + WBM - 1) / WBM;
  BigTile b;
  b.n0 = (t / ntm) * WBN;
  b.m0 = (t % ntm) * WBM;
  b.nl = min(b.n0, N - WBN);
  b.ml = min(b.m0, M - WBM);
  return b;
}

constexpr int vmcnt_imm(int n) { return ((n >> 4) << 14) | (n & 15) | 0x0F70; }

// Node rows in MFMA-fragment order: 16-byte chunk c (k = 8c..8c+7) of row
// 32 rb + r at element ((rb * (K / 8) + c) * 32 + r) * 8, so the 64 lanes of
// one operand load (32 rows, two adjacent chunks) read 1 KB contiguously.
__global__ __launch_bounds__(256) void pack_x_frag(const uint16_t* __restrict__ x, int M, int K,
                                                   uint16_t* __restrict__ xp) {
  const int64_t t = int64_t(blockIdx.x) * 256 + threadIdx.x;
  const int kc = K / 8;
  const int64_t total = int64_t(M) * kc;
  if (t >= total) return;
  const int r = int(t & 31);
  const int64_t rc = t >> 5;                 // (rb, c)
  const int c = int(rc % kc);
  const int rb = int(rc / kc);
  const int m = 32 * rb + r;
  *reinterpret_cast<u32x4*>(xp + t * 8) = *reinterpret_cast<const u32x4*>(x + int64_t(m) * K + 8 * c);
}

template <int EPI>
__global__ __launch_bounds__(512, 2) void proj_bf16_wide(KArgs a, int vec, BigPlan pl, const uint16_t* xpk) {
  constexpr int BAR = WBAR;
  constexpr int kWStage = WAHEAD + BAR;   // a fill never overwrites a stage read since the last barrier
  constexpr int kStage = WBN * GBK;       // 8192 elements = 16 KB
  __shared__ __attribute__((aligned(16))) uint16_t smem[kWStage * kStage];
  const int lane = threadIdx.x & 63, r32 = lane & 31, kh = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int M = a.M, N = a.N, K = a.K;
  const int nk_all = K / GBK;
  int t, ks = 0, nk = nk_all, slot = -1;
  if (int(blockIdx.x) < pl.full) {
    t = xcd_order(blockIdx.x, pl.full);
  } else {
    const int item = xcd_order(int(blockIdx.x) - pl.full, pl.rem * pl.pieces);
    const int piece = item / pl.rem, r = item % pl.rem;
    t = pl.full + r;
    ks = piece * nk_all / pl.pieces;
    nk = (piece + 1) * nk_all / pl.pieces - ks;
    slot = r * pl.pieces + piece;
  }
  const BigTile tl = wide_tile(M, N, t);
  const int m0 = tl.m0, n0 = tl.n0, ml = tl.ml, nl = tl.nl;
  const uint16_t* Wt = static_cast<const uint16_t*>(a.w);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(Wt + int64_t(nl) * K), (short)0, WBN * K * 2, 0x00020000);
  const int lrow = lane >> 3, lcp = lane & 7;
  const unsigned vo0 = unsigned(lrow * K * 2 + ((lcp ^ swz16(lrow)) * 16));
  const unsigned vo1 = unsigned(lrow * K * 2 + ((lcp ^ swz16(8 + lrow)) * 16));
  const int sw = swz16(r32 & 15);
  // packed node rows: row block (ml + 64 wave + 32 j) / 32, chunk 8 step + 2 sub + kh, row r32
  const uint16_t* xr[2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
    xr[j] = xpk + ((int64_t((ml + 64 * wave + 32 * j) >> 5) * (K / 8) + ks * 8 + kh) * 32 + r32) * 8;

  f32x16 acc[2][4];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[j][i][v] = 0.f;

  // Every step issues the same loads (past the last step they repeat it into
  // a stage or buffer nothing reads), so the compiler's wait counts never
  // have to assume a path with fewer loads in flight.
  auto dma = [&](int kt) {
    LDS_AS uint16_t* base = (LDS_AS uint16_t*)smem + (kt % kWStage) * kStage + 16 * wave * GBK;
    const int ksrc = min(kt, nk - 1);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const unsigned so = unsigned((16 * wave + 8 * i) * K * 2 + (ks + ksrc) * GBK * 2);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (LDS_AS void*)(base + 8 * i * GBK), 16, i ? vo1 : vo0, so, 0, 0);
    }
  };
  u32x4 xf[2][4][2];   // [step parity][sub][node tile]
  auto load_x = [&](int kt, int buf) {
    kt = min(kt, nk - 1);
#pragma unroll
    for (int sub = 0; sub < 4; ++sub)
#pragma unroll
      for (int j = 0; j < 2; ++j) xf[buf][sub][j] = *reinterpret_cast<const u32x4*>(xr[j] + (kt * 8 + 2 * sub) * 256);
  };
  bf16x8 wf[2][4];     // [sub parity][weight tile]
  auto read_w = [&](int kt, int sub, int buf) {
    const LDS_AS uint16_t* Sw = (const LDS_AS uint16_t*)smem + (kt % kWStage) * kStage;
    const int c = ((2 * sub + kh) ^ sw) * 8;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      wf[buf][i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const LDS_AS u32x4*>(Sw + (32 * i + r32) * GBK + c));
  };
  auto barrier = [] { asm volatile("s_barrier" ::: "memory"); };

  // prologue: weight stages of steps 0 .. WAHEAD - 1 and node rows of step 0
  for (int kt = 0; kt < WAHEAD; ++kt) dma(kt);
  load_x(0, 0);
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  barrier();
  read_w(0, 0, 0);
  // one 64-deep step; the node rows of step s2 sit in buffer `half`
  auto step = [&](int s2, int half) __attribute__((always_inline)) {
    load_x(s2 + 1, half ^ 1);
    dma(s2 + WAHEAD);
    __builtin_amdgcn_sched_barrier(0);   // the step's loads go out before its products
#pragma unroll
    for (int sub = 0; sub < 4; ++sub) {
      if (sub < 3) {
        read_w(s2, sub + 1, (sub + 1) & 1);
      } else if (s2 + 1 < nk) {
        if ((s2 + 1) % BAR == 0) {
          // the next BAR steps' weights landed (this wave's share; the last
          // of them was issued WAHEAD - BAR steps ago, and each step since
          // issued 8 node-row loads and 2 fills) and every wave is done
          // reading the stages the fills after this barrier reuse
          __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
          __builtin_amdgcn_s_waitcnt(vmcnt_imm(10 * (WAHEAD - BAR)));
          barrier();
        }
        read_w(s2 + 1, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);   // the next weights' reads overlap these products
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc[j][i] = mfma32(__builtin_bit_cast(bf16x8, xf[half][sub][j]), wf[sub & 1][i], acc[j][i]);
    }
  };
  // steps in pairs (buffers alternate), both halves unconditional so that
  // every path around the loop carries the same loads in flight
#pragma unroll 1
  for (int st = 0; st + 1 < nk; st += 2) {
    step(st, 0);
    step(st + 1, 1);
  }
  if (nk & 1) step(nk - 1, 0);

  // the repeated loads past the last step land before the block's LDS goes
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));

  // element v of acc[j][i] in lane l is out[m][n] at node row m = 64 wave +
  // 32 j + 8 (v / 4) + 4 (l / 32) + v % 4 and weight row n = 32 i + l % 32
  // (whole 128-byte lines per store instruction)
  (void)vec;
  if (slot >= 0) {
    float* P = pl.split + size_t(slot) * (WBM * WBN);
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          P[(64 * wave + 32 * j + 8 * (v >> 2) + 4 * kh + (v & 3)) * WBN + 32 * i + r32] = acc[j][i][v];
    return;
  }
  const bool block_bias = a.rows_per_group % 32 == 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int n = nl + 32 * i + r32;
    const bool n_new = n >= n0;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int mb = ml + 64 * wave + 32 * j;
      if (mb + 31 < m0) continue;
      if (block_bias) {
        const int64_t bb = bias_base(a, mb) + n;
        if constexpr (EPI == EPI_LOGITS) {
          const float b = n_new ? a.bias_f32[bb] : 0.f;
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int m = mb + 8 * (v >> 2) + 4 * kh + (v & 3);
            if (m >= m0 && n_new) __builtin_nontemporal_store(acc[j][i][v] + b, a.out + int64_t(m) * N + n);
          }
        } else {
          const float hb = n_new ? bf16_to_f32(static_cast<const uint16_t*>(a.bias_act)[bb]) : 0.f;
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int m = mb + 8 * (v >> 2) + 4 * kh + (v & 3);
            if (m >= m0 && n_new) {
              const int64_t o = int64_t(m) * N + n;
              a.out[o] = acc[j][i][v];
              static_cast<uint16_t*>(a.act_out)[o] = f32_to_bf16(tanhf(acc[j][i][v] + hb));
            }
          }
        }
      } else {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int m = mb + 8 * (v >> 2) + 4 * kh + (v & 3);
          if (m >= m0 && n_new) emit<EPI, true, EPI == EPI_LOGITS>(a, m, n, acc[j][i][v]);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// 17..64 rows against the vocabulary: a sweep.  One wave per block; wave w
// owns TPW consecutive 16-row weight tiles (rows 16 TPW w ..) and keeps their
// accumulators over the whole K loop.  Every operand goes memory -> LDS by
// buffer loads (nothing held in registers while in flight) into LDS private
// to the wave: the weights through a ring of AHEAD + 1 stages of 16 rows x
// 128 k (4 KB; each load instruction covers 4 rows x 256 bytes, whole
// 256-byte row pieces, which stream from HBM faster than 128-byte ones), in
// chunk-major order (c, t) = (0, 0) .. (0, TPW - 1), (1, 0) .., AHEAD < TPW
// stages in flight; the node rows of a chunk (MT x 16 rows x 128 k) into one
// slot, read into registers at the chunk's first stage (they serve its TPW
// tiles) and refilled with the next chunk's at step TPW - AHEAD.  Only the
// owning wave reads its LDS, so each wait is the wave's own vmcnt: no
// barriers, and no cross-wave reduction (the wave owns whole outputs).
// The waits count only LDS fills: register loads can complete ahead of older
// fills, so none is in flight during the stream.  Every fill reads memory
// (rows past N or M repeat the last row), and the last chunk issues only the
// fills of its own stages, with its waits counted to match.
// LDS rows are 256 bytes, 16-byte piece p of row r stored at position p ^ r
// (conflict-free both ways).  v_mfma_f32_16x16x32_bf16 with A = 16 weight
// rows, B = 16 node rows: lane l holds D[n = 4 (l >> 4) + i][m = l & 15].
// ---------------------------------------------------------------------------
// f(integral_constant<int, I>) for each I of the sequence, in order
template <class F, int... I>
__device__ __forceinline__ void each_index(std::integer_sequence<int, I...>, F&& f) {
  (f(std::integral_constant<int, I>{}), ...);
}

constexpr int kAuxNT = 2;   // cache policy of the weight fills: non-temporal
// LDS of one wave: the weight ring and the node-row slot
constexpr int sweep_lds_bytes(int MT, int AHEAD) { return (AHEAD + 1) * 4096 + MT * 4096; }

template <int MT, int TPW, int AHEAD>
__global__ __launch_bounds__(64) void proj_bf16_sweep(KArgs a) {
  constexpr int S = AHEAD + 1;       // the fill of stage s + AHEAD reuses stage s - 1's slot
  constexpr int TX = TPW - AHEAD;    // step of a chunk that fills the next chunk's node rows
  static_assert(TX >= 1, "the node-row slot is refilled after its chunk's first step");
  static_assert(4 * AHEAD + 4 * MT <= 63, "vmcnt range");
  __shared__ __attribute__((aligned(16))) uint16_t lds[sweep_lds_bytes(MT, AHEAD) / 2];
  LDS_AS uint16_t* const ring = (LDS_AS uint16_t*)lds;
  LDS_AS uint16_t* const xslot = ring + S * 2048;
  const int lane = threadIdx.x, r16 = lane & 15, kg = lane >> 4;
  const int M = a.M, N = a.N, K = a.K;
  const int nk = K >> 7;
  const int row0 = int(blockIdx.x) * (16 * TPW);
  const int rows = min(16 * TPW, N - row0);
  const unsigned rowb = unsigned(K * 2);
  const uint16_t* Wt = static_cast<const uint16_t*>(a.w);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(Wt + int64_t(row0) * K), (short)0, rows * K * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(a.x), (short)0, M * K * 2, 0x00020000);
  // fill instruction i of a 16-row block: LDS row 4 i + l / 16, position
  // l % 16, holding the row's piece (l % 16) ^ row; source rows clamped to
  // the last valid one
  const unsigned pz = unsigned((r16 ^ kg) * 16);   // for row 4 i + kg: (l % 16) ^ (4 i + kg) = pz ^ 4 i
  // operand j (k = 32 j .. 32 j + 31 of a chunk) of lane l: row l % 16,
  // piece 4 j + l / 16
  int roff[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) roff[j] = r16 * 128 + (((4 * j + kg) ^ r16) * 8);

  f32x4 acc[TPW][MT];
#pragma unroll
  for (int t = 0; t < TPW; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[t][mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // fill of the weight stage (c, t) into ring slot `slot`
  auto fill = [&](int c, int t, int slot) __attribute__((always_inline)) {
    const unsigned last = unsigned(rows - 1) * rowb;
    LDS_AS uint16_t* base = ring + slot * 2048;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const unsigned r = unsigned(16 * t + 4 * i + kg) * rowb;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (LDS_AS void*)(base + 512 * i), 16,
                                               min(r, last) + (pz ^ unsigned(64 * i)) + unsigned(c) * 256u, 0, 0, kAuxNT);
    }
  };
  // fill of chunk c's node rows into the slot
  auto fill_x = [&](int c) __attribute__((always_inline)) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (LDS_AS void*)(xslot + mt * 2048 + 512 * i), 16,
                                                 unsigned(min(16 * mt + 4 * i + kg, M - 1)) * rowb +
                                                     (pz ^ unsigned(64 * i)) + unsigned(c) * 256u, 0, 0, 0);
  };

  // chunk 0's node rows, then its first AHEAD stages into slots 0 .. AHEAD - 1
  fill_x(0);
#pragma unroll
  for (int t = 0; t < AHEAD; ++t) fill(0, t, t);

  u32x4 xf[MT][4];
  int slot = 0;   // ring slot of the current stage
  // LAST: the last chunk, which fills only its own stages
  auto chunk = [&](int c, auto LAST) __attribute__((always_inline)) {
    constexpr bool last = decltype(LAST)::value;
    each_index(std::make_integer_sequence<int, TPW>{}, [&](auto T) __attribute__((always_inline)) {
      constexpr int t = decltype(T)::value;
      __builtin_amdgcn_sched_barrier(0);   // the last step's operand reads stay ahead of this step's fills
      if constexpr (!last) {
        if constexpr (t == TX) {
          __builtin_amdgcn_s_waitcnt(0xC07F);   // chunk c's node rows are in registers: lgkmcnt(0)
          fill_x(c + 1);
        }
        fill(c + (t + AHEAD) / TPW, (t + AHEAD) % TPW, slot == 0 ? S - 1 : slot - 1);
      } else if constexpr (t + AHEAD < TPW) {
        fill(c, t + AHEAD, slot == 0 ? S - 1 : slot - 1);
      }
      // stage (c, t) (and chunk c's node rows, filled before it) landed: only
      // the fills issued after it may be in flight
      constexpr int after = last ? 4 * (AHEAD < TPW - 1 - t ? AHEAD : TPW - 1 - t)
                                 : 4 * AHEAD + (t >= TX ? 4 * MT : 0);
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(after));
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (t == 0) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            xf[mt][j] = *reinterpret_cast<const LDS_AS u32x4*>(xslot + mt * 2048 + roff[j]);
      }
      const LDS_AS uint16_t* Sw = ring + slot * 2048;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bf16x8 uf = __builtin_bit_cast(bf16x8, *reinterpret_cast<const LDS_AS u32x4*>(Sw + roff[j]));
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[t][mt] = mfma16(uf, __builtin_bit_cast(bf16x8, xf[mt][j]), acc[t][mt]);
      }
      slot = slot == S - 1 ? 0 : slot + 1;
    });
  };
#pragma unroll 1
  for (int c = 0; c + 1 < nk; ++c) chunk(c, std::false_type{});
  chunk(nk - 1, std::true_type{});

  // lane l holds, of tile t and node tile mt, node row m = 16 mt + l % 16
  // and weight rows n = row0 + 16 t + 4 (l / 16) + 0..3; the bias values of
  // a half of the tiles are loaded together, then that half is stored (with
  // ordinary stores: the 19-39 MB of logits at 32-64 rows measured 4.6 us
  // per launch faster than with non-temporal ones, and the softmax pass reads
  // them back sooner)
  auto store = [&](auto T0, auto T1) __attribute__((always_inline)) {
    constexpr int t0 = decltype(T0)::value, t1 = decltype(T1)::value;
    const bool vec = reinterpret_cast<uintptr_t>(a.bias_f32) % 16 == 0 && a.bias_stride % 4 == 0 && N % 4 == 0 &&
                     reinterpret_cast<uintptr_t>(a.out) % 16 == 0;
    int64_t bb[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) bb[mt] = bias_base(a, min(16 * mt + r16, M - 1));
    f32x4 bz[t1 - t0][MT];
#pragma unroll
    for (int t = t0; t < t1; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int n = min(row0 + 16 * t + 4 * kg, N - 4);
        bz[t - t0][mt] = vec ? *reinterpret_cast<const f32x4*>(a.bias_f32 + bb[mt] + n) : f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
    for (int t = t0; t < t1; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int m = 16 * mt + r16, n = row0 + 16 * t + 4 * kg;
        if (m >= M || n >= N) continue;
        const f32x4 v = acc[t][mt];
        if (vec && n + 3 < N) {
          *reinterpret_cast<f32x4*>(a.out + int64_t(m) * N + n) = v + bz[t - t0][mt];
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (n + i < N) a.out[int64_t(m) * N + n + i] = v[i] + a.bias_f32[bb[mt] + n + i];
        }
      }
  };
  constexpr int H = (TPW + 1) / 2;
  store(std::integral_constant<int, 0>{}, std::integral_constant<int, H>{});
  store(std::integral_constant<int, H>{}, std::integral_constant<int, TPW>{});
}

// The split wide tiles: 16 blocks per tile, each 32 rows x 128 columns.
template <int EPI>
__global__ __launch_bounds__(256) void proj_wide_fixup(KArgs a, int vec, BigPlan pl) {
  const int r = blockIdx.x / 16, row0 = (blockIdx.x % 16) * 32;
  const BigTile tl = wide_tile(a.M, a.N, pl.full + r);
  const float* P = pl.split + size_t(r) * pl.pieces * (WBM * WBN);
  const int c4 = threadIdx.x & 31;
  const int n = tl.nl + 4 * c4;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int row = row0 + (threadIdx.x >> 5) + 8 * u;
    const int m = tl.ml + row;
    if (m < tl.m0) continue;
    const size_t e = size_t(row) * WBN + 4 * c4;
    f32x4 v = *reinterpret_cast<const f32x4*>(P + e);
    for (int pc = 1; pc < pl.pieces; ++pc) v += *reinterpret_cast<const f32x4*>(P + size_t(pc) * (WBM * WBN) + e);
    if (n >= tl.n0) {
      emit4<EPI, EPI == EPI_LOGITS>(a, m, n, v, vec != 0);
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (n + k >= tl.n0) emit<EPI, true, EPI == EPI_LOGITS>(a, m, n + k, v[k]);
    }
  }
}

// The split tiles: 16 blocks per tile, each 16 rows x 256 columns; every
// thread sums the pieces of 4 float4s in piece order and applies the epilogue.
template <int EPI>
__global__ __launch_bounds__(256) void proj_big_fixup(KArgs a, int vec, BigPlan pl) {
  const int r = blockIdx.x / 16, row0 = (blockIdx.x % 16) * 16;
  const BigTile tl = big_tile(a.M, a.N, pl.full + r);
  const float* P = pl.split + size_t(r) * pl.pieces * (GBM * GBN);
  const int c4 = threadIdx.x & 63;
  const int n = tl.nl + 4 * c4;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int row = row0 + (threadIdx.x >> 6) + 4 * u;
    const int m = tl.ml + row;
    if (m < tl.m0) continue;
    const size_t e = size_t(row) * GBN + 4 * c4;
    f32x4 v = *reinterpret_cast<const f32x4*>(P + e);
    for (int pc = 1; pc < pl.pieces; ++pc) v += *reinterpret_cast<const f32x4*>(P + size_t(pc) * (GBM * GBN) + e);
    if (n >= tl.n0) {
      emit4<EPI, EPI == EPI_LOGITS>(a, m, n, v, vec != 0);
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (n + k >= tl.n0) emit<EPI, true, EPI == EPI_LOGITS>(a, m, n + k, v[k]);
    }
  }
}

// ---------------------------------------------------------------------------
// The head (A: h x h) at 17..64 node rows, split along K.  A block per 16-row
// weight tile over the whole K re-reads all node rows in every block (at 64
// rows x 4096 that is four times the weight bytes, and the launch is bound by
// it).  Here a block owns 64 weight rows (one 16-row tile per wave) and one K
// piece of KC: the piece's node rows are read once into LDS and serve all
// four tiles, each wave loads its tile's MFMA operand fragments straight from
// memory (all of the piece in flight at once), and the block stores its
// partial sums [piece][M][N]; proj_hsplit_fixup adds the pieces in piece
// order (deterministic) and applies the epilogue.  LDS rows of the staged
// node rows are 256-byte pieces with 16-byte chunk c of row r at c ^ (r % 16)
// (conflict-free writes and operand reads).
// ---------------------------------------------------------------------------
constexpr int HSG = 64;   // weight rows per block

template <int MT, int KC>
__global__ __launch_bounds__(256) void proj_bf16_hsplit(KArgs a, float* __restrict__ part) {
  constexpr int NS = KC / 32;          // 32-deep MFMA steps per piece
  constexpr int XR = 16 * MT;          // staged node rows
  constexpr int XC = KC / 8;           // 16-byte chunks per staged row
  constexpr int XPT = XR * XC / 256;   // chunks per thread
  static_assert(XR * XC % 256 == 0, "whole chunks per thread");
  __shared__ __attribute__((aligned(16))) uint16_t xs[XR * KC];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int M = a.M, N = a.N, K = a.K;
  const int n0 = blockIdx.x * HSG, piece = blockIdx.y;
  const int kb = piece * KC;   // K % KC == 0
  const uint16_t* X = static_cast<const uint16_t*>(a.x);
  const uint16_t* Wt = static_cast<const uint16_t*>(a.w);
  // LDS element of node row `row`, 16-byte chunk c of the piece
  auto xoff = [](int row, int c) { return (c >> 4) * (XR * 128) + row * 128 + (((c & 15) ^ (row & 15)) << 3); };

  // node rows of the piece (rows past M repeat the last row; never stored)
  u32x4 xv[XPT];
#pragma unroll
  for (int i = 0; i < XPT; ++i) {
    const int idx = threadIdx.x + 256 * i, row = idx / XC, c = idx % XC;
    xv[i] = ld_cached(X + int64_t(min(row, M - 1)) * K + kb + 8 * c);
  }
  // this wave's weight tile, as operand fragments (rows past N repeat the last)
  u32x4 R[NS];
  const uint16_t* wp = Wt + int64_t(min(n0 + 16 * w + r16, N - 1)) * K + kb + 8 * kg;
#pragma unroll
  for (int s = 0; s < NS; ++s) R[s] = ld_cached(wp + 32 * s);
  __builtin_amdgcn_sched_barrier(0);   // every load of the piece in flight before the first LDS write
#pragma unroll
  for (int i = 0; i < XPT; ++i) {
    const int idx = threadIdx.x + 256 * i, row = idx / XC, c = idx % XC;
    *reinterpret_cast<u32x4*>(xs + xoff(row, c)) = xv[i];
  }
  __syncthreads();

  f32x4 acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const bf16x8 av = __builtin_bit_cast(bf16x8, R[s]);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const bf16x8 bv = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(xs + xoff(16 * mt + r16, 4 * s + kg)));
      acc[mt] = mfma16(av, bv, acc[mt]);
    }
  }
  // lane (r16, kg) holds node row 16 mt + r16, weight rows n .. n + 3
  const int n = n0 + 16 * w + 4 * kg;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = 16 * mt + r16;
    if (m < M && n < N) *reinterpret_cast<f32x4*>(part + (size_t(piece) * M + m) * N + n) = acc[mt];
  }
}

// The pieces summed in piece order, then the epilogue.  Block b takes column
// group b % G (the 64 weight rows of one main-kernel group) and rows
// 16 (b / G) .. + 15, a thread 4 outputs (with G a multiple of 8 on the XCD
// whose main-kernel blocks wrote that group: about 1% faster per round than
// a row per block, though the counters show the partial sums still fetched
// from beyond the L2).  The loads go out BATCH pieces at a time (8, or 16
// past 8 pieces), unconditionally (pieces past the last repeat it and are not
// added): a loop of one load per piece would wait a memory round trip per
// piece.
template <int BATCH>
__device__ __forceinline__ f32x4 sum_pieces(const float* pp, size_t stride, int pieces) {
  f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int p0 = 0; p0 < pieces; p0 += BATCH) {
    f32x4 q[BATCH];
#pragma unroll
    for (int i = 0; i < BATCH; ++i) q[i] = *reinterpret_cast<const f32x4*>(pp + size_t(min(p0 + i, pieces - 1)) * stride);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < BATCH; ++i)
      if (p0 + i < pieces) v = p0 + i == 0 ? q[i] : v + q[i];
  }
  return v;
}

template <int EPI>
__global__ __launch_bounds__(256) void proj_hsplit_fixup(KArgs a, const float* __restrict__ part, int pieces, int vec) {
  const int G = (a.N + HSG - 1) / HSG;
  const int g = blockIdx.x % G, r16 = blockIdx.x / G;
  const int m = 16 * r16 + (threadIdx.x >> 4), n = HSG * g + 4 * (threadIdx.x & 15);
  if (m >= a.M || n >= a.N) return;
  const size_t stride = size_t(a.M) * a.N;
  const float* pp = part + size_t(m) * a.N + n;
  const f32x4 v = pieces <= 8 ? sum_pieces<8>(pp, stride, pieces) : sum_pieces<16>(pp, stride, pieces);
  emit4<EPI>(a, m, n, v, vec != 0);
}

// ---------------------------------------------------------------------------
// fp32: one thread per output element, sequential K.
// ---------------------------------------------------------------------------
template <int EPI>
__global__ __launch_bounds__(256) void proj_f32(KArgs a, int nblk_n) {
  const int m = blockIdx.x / nblk_n;
  const int n = (blockIdx.x % nblk_n) * 256 + threadIdx.x;
  if (n >= a.N) return;
  const float* xr = static_cast<const float*>(a.x) + int64_t(m) * a.K;
  const float* wr = static_cast<const float*>(a.w) + int64_t(n) * a.K;
  float acc = 0.f;
  for (int k = 0; k < a.K; ++k) acc = fmaf(xr[k], wr[k], acc);
  emit<EPI, false>(a, m, n, acc);
}

// vec: every group of 4 outputs and its bias are 16-byte aligned
bool epilogue_vec_ok(const KArgs& k, int epi) {
  if (k.N % 4 != 0 || k.bias_stride % 4 != 0) return false;
  const uintptr_t bias = epi == EPI_LOGITS ? reinterpret_cast<uintptr_t>(k.bias_f32)
                                           : reinterpret_cast<uintptr_t>(k.bias_act);
  const size_t bias_align = epi == EPI_LOGITS ? 16 : 8;
  return bias % bias_align == 0 && reinterpret_cast<uintptr_t>(k.out) % 16 == 0 &&
         (epi == EPI_LOGITS || reinterpret_cast<uintptr_t>(k.act_out) % 8 == 0);
}

template <int MT, int NT, int KW, int D>
hipError_t launch_stream(const KArgs& k, int epi, hipStream_t s) {
  const dim3 grid((k.N + 16 * NT - 1) / (16 * NT));
  const int vec = epilogue_vec_ok(k, epi);
  if (epi == EPI_LOGITS)
    hipLaunchKernelGGL((proj_bf16_stream<MT, NT, KW, D, EPI_LOGITS>), grid, dim3(64 * KW), 0, s, k, vec);
  else
    hipLaunchKernelGGL((proj_bf16_stream<MT, NT, KW, D, EPI_HEAD>), grid, dim3(64 * KW), 0, s, k, vec);
  return hipGetLastError();
}

template <int KW>
hipError_t launch_pairs(const KArgs& k, hipStream_t s) {
  const dim3 grid((k.N + 31) / 32);
  hipLaunchKernelGGL((proj_bf16_pairs<KW, EPI_LOGITS>), grid, dim3(64 * KW), 0, s, k, epilogue_vec_ok(k, EPI_LOGITS));
  return hipGetLastError();
}

template <int MT>
hipError_t launch_stream_nt(const KArgs& k, int epi, hipStream_t s) {
  // Long weight matrices (the vocabulary): 32-row blocks, 8 waves over K at
  // 16 node rows; from 17 node rows on, 128-row blocks and 4 waves over K, so
  // that every node-row operand a wave loads serves 8 weight tiles (measured
  // at 32 and 64 rows: 1.36x and 1.47x the 32-row blocks' stream rate).
  // Short ones (A, h rows): 16-row blocks, 8 waves over K (16 at 17-32 rows;
  // measured at 8 rows x 2560: 8 waves 129.7 us of head per round against
  // 135.8 with 16).
  if (k.N >= 32 * 2048) {
    if constexpr (MT >= 2) return launch_stream<MT, 8, 4, 1>(k, epi, s);
    if (k.K % 128 == 0 && epi == EPI_LOGITS) return launch_pairs<4>(k, s);
    return launch_stream<MT, 2, 8, 2>(k, epi, s);
  }
  if constexpr (MT == 2) return launch_stream<MT, 1, 16, 2>(k, epi, s);
  return launch_stream<MT, 1, 8, 2>(k, epi, s);
}

// Split plan limits: at most kSplitMaxBlocks pieces (one 256 KB partial each),
// and at least kMinPieceSteps 64-deep K steps per piece.
constexpr int kSplitMaxBlocks = 256;
constexpr int kMinPieceSteps = 4;
// one partial tile per split block; the two many-row tilings hold the same
constexpr size_t kSplitBytes = size_t(kSplitMaxBlocks) * GBM * GBN * sizeof(float);
static_assert(WBM * WBN == GBM * GBN, "split partial slots");

// Compute units of the current device (cached per device).
int device_cus() {
  static int cached[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return kSplitMaxBlocks;
  if (dev < 64 && cached[dev] > 0) return cached[dev];
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    n = kSplitMaxBlocks;
  if (dev < 64) cached[dev] = n;
  return n;
}

// Shapes the 256x256-tile kernel takes: the vocabulary at >= 512 rows, and
// (only when split) the head at >= 512 rows.
bool big_logits(const KArgs& k) { return k.M >= 2 * GBM && k.N >= 64 * GBN; }
// The 512-row tiles where they compute no more rows than the 256-row ones
// (their node-row blocks are 32 rows, so also M % 32 == 0).
bool wide_logits(const KArgs& k) {
  return big_logits(k) && k.M % 32 == 0 && (k.M + WBM - 1) / WBM * WBM == (k.M + GBM - 1) / GBM * GBM;
}
bool big_head_candidate(const KArgs& k) { return k.M >= 2 * GBM && k.N >= GBN && k.K >= 2 * kMinPieceSteps * GBK; }

// The split head: 17..64 node rows against a short weight matrix (fewer than
// 32 * 2048 rows), K a multiple of 128, N of 4.  The piece length is the
// longest of 512 / 256 / 128 dividing K that still gives about 384
// blocks (1.5 per CU of a 256-CU device; fixed, so that the workspace size
// does not depend on the device), else the shortest; a single piece takes the
// unsplit kernel.
bool hsplit_shape(const KArgs& k) {
  return k.M > 16 && k.M <= 64 && k.N < 32 * 2048 && k.K % 128 == 0 && k.N % 4 == 0;
}
int hsplit_kc(const KArgs& k) {
  const int groups = (k.N + HSG - 1) / HSG;
  for (int kc : {512, 256})
    if (k.K % kc == 0 && groups * (k.K / kc) >= 384) return kc;
  return 128;
}
int hsplit_pieces(const KArgs& k) { return k.K / hsplit_kc(k); }

template <int MT, int KC>
void launch_hsplit_mt(const KArgs& k, float* part, hipStream_t s) {
  const dim3 grid(unsigned((k.N + HSG - 1) / HSG), unsigned(k.K / KC));
  hipLaunchKernelGGL((proj_bf16_hsplit<MT, KC>), grid, dim3(256), 0, s, k, part);
}

template <int KC>
void launch_hsplit_kc(const KArgs& k, float* part, hipStream_t s) {
  if (k.M <= 32) launch_hsplit_mt<2, KC>(k, part, s);
  else if (k.M <= 48) launch_hsplit_mt<3, KC>(k, part, s);
  else launch_hsplit_mt<4, KC>(k, part, s);
}

hipError_t launch_hsplit(const KArgs& k, int epi, float* part, hipStream_t s) {
  const int kc = hsplit_kc(k);
  if (kc == 512) launch_hsplit_kc<512>(k, part, s);
  else if (kc == 256) launch_hsplit_kc<256>(k, part, s);
  else launch_hsplit_kc<128>(k, part, s);
  const int vec = epilogue_vec_ok(k, epi);
  const dim3 grid(unsigned(((k.N + HSG - 1) / HSG) * ((k.M + 15) / 16)));
  if (epi == EPI_LOGITS)
    hipLaunchKernelGGL((proj_hsplit_fixup<EPI_LOGITS>), grid, dim3(256), 0, s, k, part, hsplit_pieces(k), vec);
  else
    hipLaunchKernelGGL((proj_hsplit_fixup<EPI_HEAD>), grid, dim3(256), 0, s, k, part, hsplit_pieces(k), vec);
  return hipGetLastError();
}

BigPlan big_plan(const KArgs& k, float* split) {
  const int T = ((k.M + GBM - 1) / GBM) * ((k.N + GBN - 1) / GBN);
  BigPlan pl{T, 0, 1, nullptr};
  if (!split) return pl;
  const int ncu = std::min(device_cus(), kSplitMaxBlocks);
  const int rem = T % ncu;
  if (rem == 0) return pl;
  const int pieces = std::min(ncu / rem, (k.K / GBK) / kMinPieceSteps);
  if (pieces < 2) return pl;
  return BigPlan{T - rem, rem, pieces, split};
}

// The sweep: three waves per compute unit (measured at 32 rows x 151936:
// 13 tiles per wave with 9 stages ahead 128.3-128.9 us, 10 tiles with four
// waves per CU 131-133 us), tiles per wave (of the instantiated counts) so
// that all waves are resident at once, stages ahead as the LDS of three
// waves allows.
constexpr int sweep_waves_per_cu(int) { return 3; }
constexpr int sweep_ahead(int MT, int TPW) { return (MT == 2 ? 9 : 8) < TPW - 1 ? (MT == 2 ? 9 : 8) : TPW - 1; }

template <int MT, int TPW>
hipError_t launch_sweep(const KArgs& k, hipStream_t s) {
  constexpr int AHEAD = sweep_ahead(MT, TPW);
  static_assert(sweep_waves_per_cu(MT) * sweep_lds_bytes(MT, AHEAD) <= 160 * 1024, "LDS of the resident waves");
  const int tiles = (k.N + 15) / 16;
  hipLaunchKernelGGL((proj_bf16_sweep<MT, TPW, AHEAD>), dim3((tiles + TPW - 1) / TPW), dim3(64), 0, s, k);
  return hipGetLastError();
}

// The instantiated tile count to use (the least one not below the need), 0
// where none is large enough.
int sweep_tpw(const KArgs& k, int MT) {
  const int tiles = (k.N + 15) / 16;
  const int slots = sweep_waves_per_cu(MT) * device_cus();
  const int need = (tiles + slots - 1) / slots;
  for (int t : {4, 6, 8, 10, 13, 16})
    if (t >= need) return t;
  return 0;
}

template <int MT>
hipError_t launch_sweep_tpw(const KArgs& k, int tpw, hipStream_t s) {
  switch (tpw) {
    case 4: return launch_sweep<MT, 4>(k, s);
    case 6: return launch_sweep<MT, 6>(k, s);
    case 8: return launch_sweep<MT, 8>(k, s);
    case 10: return launch_sweep<MT, 10>(k, s);
    case 13: return launch_sweep<MT, 13>(k, s);
    default: return launch_sweep<MT, 16>(k, s);
  }
}

template <int EPI>
hipError_t launch_big(const KArgs& k, const BigPlan& pl, hipStream_t s) {
  const int vec = epilogue_vec_ok(k, EPI);
  hipLaunchKernelGGL((proj_bf16_big<EPI>), dim3(pl.full + pl.rem * pl.pieces), dim3(512), 0, s, k, vec, pl);
  if (pl.rem > 0) hipLaunchKernelGGL((proj_big_fixup<EPI>), dim3(pl.rem * 16), dim3(256), 0, s, k, vec, pl);
  return hipGetLastError();
}

BigPlan wide_plan(const KArgs& k, float* split) {
  const int T = ((k.M + WBM - 1) / WBM) * ((k.N + WBN - 1) / WBN);
  BigPlan pl{T, 0, 1, nullptr};
  if (!split) return pl;
  const int ncu = std::min(device_cus(), kSplitMaxBlocks);
  const int rem = T % ncu;
  if (rem == 0) return pl;
  const int pieces = std::min(ncu / rem, (k.K / GBK) / kMinPieceSteps);
  if (pieces < 2) return pl;
  return BigPlan{T - rem, rem, pieces, split};
}

template <int EPI>
hipError_t launch_wide(const KArgs& k, const BigPlan& pl, uint16_t* xpk, hipStream_t s) {
  const int vec = epilogue_vec_ok(k, EPI);
  const int64_t chunks = int64_t(k.M) * (k.K / 8);
  hipLaunchKernelGGL(pack_x_frag, dim3(unsigned((chunks + 255) / 256)), dim3(256), 0, s,
                     static_cast<const uint16_t*>(k.x), k.M, k.K, xpk);
  const dim3 grid(pl.full + pl.rem * pl.pieces);
  hipLaunchKernelGGL((proj_bf16_wide<EPI>), grid, dim3(512), 0, s, k, vec, pl, static_cast<const uint16_t*>(xpk));
  if (pl.rem > 0) hipLaunchKernelGGL((proj_wide_fixup<EPI>), dim3(pl.rem * 16), dim3(256), 0, s, k, vec, pl);
  return hipGetLastError();
}

}  // namespace

size_t proj_split_bytes(int precision, int epilogue, int64_t M, int64_t N, int64_t K) {
  if (precision != DARTREE_BF16 || M <= 0 || N <= 0 || K <= 0 || M > INT32_MAX || N > INT32_MAX) return 0;
  KArgs k{};
  k.M = int(M);
  k.N = int(N);
  k.K = int(K);
  if (epilogue == EPI_HEAD && hsplit_shape(k) && hsplit_pieces(k) > 1)
    return size_t(hsplit_pieces(k)) * size_t(M) * size_t(N) * sizeof(float);
  const bool big = epilogue == EPI_LOGITS ? big_logits(k) : big_head_candidate(k);
  // the split partials, then (512-row tiles) the node rows in fragment order
  const size_t packed = epilogue == EPI_LOGITS && wide_logits(k) ? size_t(M) * size_t(K) * 2 : 0;
  return big ? kSplitBytes + packed : 0;
}

hipError_t launch_project(const ProjArgs& p, hipStream_t s) {
  KArgs k;
  k.x = p.x;
  k.w = p.w;
  k.M = int(p.M);
  k.N = int(p.N);
  k.K = int(p.K);
  k.rows_per_group = int(p.rows_per_group);
  k.bias_stride = p.bias_stride;
  k.bias_f32 = p.bias_f32;
  k.bias_act = p.bias_act;
  k.group_index = p.group_index;
  k.out = p.out;
  k.act_out = p.act_out;
  if (k.M <= 0 || k.N <= 0) return hipSuccess;

  if (p.precision == DARTREE_FP32) {
    const int nblk_n = (k.N + 255) / 256;
    const dim3 grid(nblk_n * k.M);
    if (p.epilogue == EPI_LOGITS) hipLaunchKernelGGL((proj_f32<EPI_LOGITS>), grid, dim3(256), 0, s, k, nblk_n);
    else hipLaunchKernelGGL((proj_f32<EPI_HEAD>), grid, dim3(256), 0, s, k, nblk_n);
    return hipGetLastError();
  }
  if (p.epilogue == EPI_LOGITS && k.M > 16 && k.M <= 64 && k.N >= 32 * 2048 && k.K % 128 == 0) {
    const int mt = k.M <= 32 ? 2 : 4;
    const int tpw = sweep_tpw(k, mt);
    if (tpw > 0) return mt == 2 ? launch_sweep_tpw<2>(k, tpw, s) : launch_sweep_tpw<4>(k, tpw, s);
  }
  if (p.epilogue == EPI_HEAD && p.split && hsplit_shape(k) && hsplit_pieces(k) > 1)
    return launch_hsplit(k, p.epilogue, p.split, s);
  if (k.M <= 16) return launch_stream_nt<1>(k, p.epilogue, s);
  if (k.M <= 32) return launch_stream_nt<2>(k, p.epilogue, s);
  if (k.M <= 48) return launch_stream_nt<3>(k, p.epilogue, s);
  if (k.M <= 64) return launch_stream_nt<4>(k, p.epilogue, s);
  if (p.epilogue == EPI_LOGITS && big_logits(k)) {
    if (wide_logits(k) && p.split)
      return launch_wide<EPI_LOGITS>(k, wide_plan(k, p.split),
                                     reinterpret_cast<uint16_t*>(reinterpret_cast<char*>(p.split) + kSplitBytes), s);
    return launch_big<EPI_LOGITS>(k, big_plan(k, p.split), s);
  }
  if (p.epilogue == EPI_HEAD && big_head_candidate(k)) {
    const BigPlan pl = big_plan(k, p.split);
    if (pl.rem > 0) return launch_big<EPI_HEAD>(k, pl, s);
  }
  const dim3 grid((k.M + TBM - 1) / TBM, (k.N + TBN - 1) / TBN);
  if (p.epilogue == EPI_LOGITS) hipLaunchKernelGGL((proj_bf16_tiled<EPI_LOGITS>), grid, dim3(256), 0, s, k);
  else hipLaunchKernelGGL((proj_bf16_tiled<EPI_HEAD>), grid, dim3(256), 0, s, k);
  return hipGetLastError();
}

}  // namespace dartree
