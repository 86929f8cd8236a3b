// Correction-head products of one depth (Algorithm 1, "correct all prefixes
// in parallel"): for every node row m of S_{d-1}
//   head    : t[m] = A r[m],  a[m] = act(tanh(t[m] + H_d))      (N = h)
//   logits  : z[m] = L_d^base + U a[m]                            (N = V)
// Both are out[m][n] = f(sum_k x[m][k] w[n][k]) with w = A or U stored
// [N][K] row-major (K contiguous), so one family of kernels serves both.
//
// bf16 path, gfx950 MFMA v_mfma_f32_16x16x32_bf16 (fp32 accumulation):
//  * proj_bf16_stream: few rows (M <= 64).  The product is a stream over the
//    weight matrix (U is 0.78-1.56 GB per depth, far beyond the caches), so
//    every weight element is read once from HBM with coalesced non-temporal
//    loads and staged through LDS into MFMA operand layout.
//  * proj_bf16_big: many rows (>= 512) against the vocabulary.  256x256 tiles,
//    buffer loads straight to swizzled LDS, XCD-aware tile order.
//  * proj_bf16_tiled: other many-row products (the head, or a few hundred
//    rows).  128x128 output tiles, 64-deep K steps staged through
//    double-buffered, padded LDS tiles shared by 4 waves (64x64 each).
// fp32 path: plain FMA loop (small problems only).
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
  float* out;
  void* act_out;
};

template <int EPI, bool BF16>
__device__ __forceinline__ void emit(const KArgs& a, int m, int n, float acc) {
  const int64_t g = m / a.rows_per_group;
  const int64_t o = int64_t(m) * a.N + n;
  if constexpr (EPI == EPI_LOGITS) {
    a.out[o] = acc + a.bias_f32[g * a.bias_stride + n];
  } else {
    a.out[o] = acc;
    float hb;
    if constexpr (BF16) hb = bf16_to_f32(static_cast<const uint16_t*>(a.bias_act)[g * a.bias_stride + n]);
    else hb = static_cast<const float*>(a.bias_act)[g * a.bias_stride + n];
    const float v = tanhf(acc + hb);
    if constexpr (BF16) static_cast<uint16_t*>(a.act_out)[o] = f32_to_bf16(v);
    else static_cast<float*>(a.act_out)[o] = v;
  }
}

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
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

template <int EPI>
__device__ __forceinline__ void emit4(const KArgs& a, int m, int n, f32x4 v, bool vec) {
  const int64_t g = m / a.rows_per_group;
  const int64_t o = int64_t(m) * a.N + n;
  if (vec && n + 3 < a.N) {
    if constexpr (EPI == EPI_LOGITS) {
      const f32x4 b = *reinterpret_cast<const f32x4*>(a.bias_f32 + g * a.bias_stride + n);
      *reinterpret_cast<f32x4*>(a.out + o) = v + b;
    } else {
      typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
      const u16x4 hb = *reinterpret_cast<const u16x4*>(static_cast<const uint16_t*>(a.bias_act) + g * a.bias_stride + n);
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
    if (n + i < a.N) emit<EPI, true>(a, m, n + i, v[i]);
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
    if (m < M) emit4<EPI>(a, m, n0 + nt * 16 + kg * 4, v, vec != 0);
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
// block, 4 waves of 128x128 (64 MFMA accumulators each, held in AGPRs).
// Both operand tiles move 64-k slices with buffer loads straight into LDS
// (no VGPR staging; rows past the matrix read as zero through the buffer
// resource's range), XOR-swizzled by row so that the MFMA-layout reads are
// bank-conflict free, double-buffered over K.  Tiles are ordered so that
// consecutive blocks on one XCD (blocks are dealt to the 8 XCDs round-robin)
// cover the M-tiles of one weight tile, which then stays in that XCD's L2.
// ---------------------------------------------------------------------------
constexpr int GBM = 256, GBN = 256, GBK = 64;
#define LDS_AS __attribute__((address_space(3)))

__device__ __forceinline__ int swz16(int r) { return (r ^ (r >> 3)) & 7; }  // r in 0..15

__global__ __launch_bounds__(256) void proj_bf16_big(KArgs a, int vec) {
  __shared__ __attribute__((aligned(16))) uint16_t smem[2][(GBN + GBM) * GBK];  // [buf][W rows | X rows]
  const int lane = threadIdx.x & 63, r16 = lane & 15, kg = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int M = a.M, N = a.N, K = a.K;
  const int ntm = (M + GBM - 1) / GBM, ntn = (N + GBN - 1) / GBN, T = ntm * ntn;
  int t = blockIdx.x;
  const int q8 = T / 8;
  if (t < 8 * q8) t = (t % 8) * q8 + t / 8;
  const int n0 = (t / ntm) * GBN, m0 = (t % ntm) * GBM;
  const int wm = wave & 1, wn = wave >> 1;
  const uint16_t* X = static_cast<const uint16_t*>(a.x);
  const uint16_t* Wt = static_cast<const uint16_t*>(a.w);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(Wt + int64_t(n0) * K), (short)0, min(GBN, N - n0) * K * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(X + int64_t(m0) * K), (short)0, min(GBM, M - m0) * K * 2, 0x00020000);
  // load i of wave w moves rows 64 w + 8 i + lane / 8; LDS chunk lane % 8 holds
  // global chunk (lane % 8) ^ swizzle(row).  The row offset is part of the
  // per-lane offset, which the buffer range check covers (rows past the
  // matrix read as zero); the scalar offset carries only the k position.
  const int lrow = lane >> 3, lcp = lane & 7;
  const unsigned vrow = unsigned((64 * wave + lrow) * K * 2);
  const unsigned vc0 = unsigned((lcp ^ swz16(lrow)) * 16), vc1 = unsigned((lcp ^ swz16(8 + lrow)) * 16);
  const int ax0 = (wn * 128 + r16) * GBK + ((kg ^ swz16(r16)) * 8);
  const int ax1 = (wn * 128 + r16) * GBK + (((4 + kg) ^ swz16(r16)) * 8);
  const int bx0 = GBN * GBK + (wm * 128 + r16) * GBK + ((kg ^ swz16(r16)) * 8);
  const int bx1 = GBN * GBK + (wm * 128 + r16) * GBK + (((4 + kg) ^ swz16(r16)) * 8);

  f32x4 acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto load = [&](int buf, int kt) {
    LDS_AS uint16_t* base = (LDS_AS uint16_t*)smem[buf];  // generic -> LDS address space
    const unsigned so = unsigned(kt * GBK * 2);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const unsigned vo = vrow + unsigned(8 * i * K * 2) + ((i & 1) ? vc1 : vc0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (LDS_AS void*)(base + (64 * wave + 8 * i) * GBK), 16, vo, so, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (LDS_AS void*)(base + GBN * GBK + (64 * wave + 8 * i) * GBK), 16, vo,
                                               so, 0, 0);
    }
  };
  auto rd = [&](const LDS_AS uint16_t* S, int off) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const LDS_AS u32x4*>(S + off));
  };
  auto block = [&](const bf16x8 (&av)[8], const bf16x8 (&bv)[4], int h) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][4 * h + j] = mfma16(av[i], bv[j], acc[i][4 * h + j]);
  };

  const int nk = K / GBK;
  load(0, 0);
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    __builtin_amdgcn_s_waitcnt(0);  // this wave's share of tile kt has landed
    __syncthreads();                // ... every wave's; buffer cur ^ 1 is no longer read
    const LDS_AS uint16_t* S = (const LDS_AS uint16_t*)smem[cur];
    bf16x8 A0[8], A1[8], B00[4], B01[4], B10[4], B11[4];
#pragma unroll
    for (int i = 0; i < 8; ++i) A0[i] = rd(S, ax0 + i * 16 * GBK);
#pragma unroll
    for (int j = 0; j < 4; ++j) B00[j] = rd(S, bx0 + j * 16 * GBK);
    if (kt + 1 < nk) load(cur ^ 1, kt + 1);
#pragma unroll
    for (int j = 0; j < 4; ++j) B01[j] = rd(S, bx0 + (4 + j) * 16 * GBK);
    // operand reads for the next quarter are issued ahead of each MFMA group
    __builtin_amdgcn_sched_barrier(0);
    block(A0, B00, 0);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 8; ++i) A1[i] = rd(S, ax1 + i * 16 * GBK);
#pragma unroll
    for (int j = 0; j < 4; ++j) B10[j] = rd(S, bx1 + j * 16 * GBK);
    __builtin_amdgcn_sched_barrier(0);
    block(A0, B01, 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < 4; ++j) B11[j] = rd(S, bx1 + (4 + j) * 16 * GBK);
    __builtin_amdgcn_sched_barrier(0);
    block(A1, B10, 0);
    __builtin_amdgcn_sched_barrier(0);
    block(A1, B11, 1);
  }

  // lane holds D[n = 4 kg + q][m = r16] of each 16x16 sub-tile
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int m = m0 + wm * 128 + j * 16 + r16;
      if (m < M) emit4<EPI_LOGITS>(a, m, n0 + wn * 128 + i * 16 + kg * 4, acc[i][j], vec != 0);
    }
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

template <int MT>
hipError_t launch_stream_nt(const KArgs& k, int epi, hipStream_t s) {
  // Long weight matrices (the vocabulary): 32-row blocks, 8 waves over K.
  // Short ones (A, h rows): 16-row blocks, 16 waves over K (8 when the node
  // rows need more registers), so that even h = 2560 rows give enough waves
  // to keep HBM busy.
  if (k.N >= 32 * 2048) return launch_stream<MT, 2, 8, 2>(k, epi, s);
  if constexpr (MT <= 2) return launch_stream<MT, 1, 16, 2>(k, epi, s);
  return launch_stream<MT, 1, 8, 2>(k, epi, s);
}

}  // namespace

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
  if (k.M <= 16) return launch_stream_nt<1>(k, p.epilogue, s);
  if (k.M <= 32) return launch_stream_nt<2>(k, p.epilogue, s);
  if (k.M <= 48) return launch_stream_nt<3>(k, p.epilogue, s);
  if (k.M <= 64) return launch_stream_nt<4>(k, p.epilogue, s);
  if (p.epilogue == EPI_LOGITS && k.M >= 2 * GBM && k.N >= 64 * GBN) {
    const int tiles = ((k.M + GBM - 1) / GBM) * ((k.N + GBN - 1) / GBN);
    hipLaunchKernelGGL(proj_bf16_big, dim3(tiles), dim3(256), 0, s, k, int(epilogue_vec_ok(k, EPI_LOGITS)));
    return hipGetLastError();
  }
  const dim3 grid((k.M + TBM - 1) / TBM, (k.N + TBN - 1) / TBN);
  if (p.epilogue == EPI_LOGITS) hipLaunchKernelGGL((proj_bf16_tiled<EPI_LOGITS>), grid, dim3(256), 0, s, k);
  else hipLaunchKernelGGL((proj_bf16_tiled<EPI_HEAD>), grid, dim3(256), 0, s, k);
  return hipGetLastError();
}

}  // namespace dartree
