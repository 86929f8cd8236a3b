// Correction-head products of one depth (Algorithm 1, "correct all prefixes
// in parallel"): for every node row m of S_{d-1}
//   head    : t[m] = A r[m],  a[m] = act(tanh(t[m] + H_d))      (N = h)
//   logits  : z[m] = L_d^base + U a[m]                            (N = V)
// Both are out[m][n] = f(sum_k x[m][k] w[n][k]) with w = A or U stored
// [N][K] row-major (K contiguous), so one family of kernels serves both.
//
// bf16 path, gfx950 MFMA v_mfma_f32_16x16x32_bf16 (fp32 accumulation):
//  * proj_bf16_skinny: few rows (M <= 64).  The product is a stream over the
//    weight matrix (U is 0.78-1.56 GB per depth), so every weight element is
//    loaded once, straight from HBM into MFMA operand registers; the 4 waves
//    of a block split K and are summed through LDS.
//  * proj_bf16_tiled: many rows.  128x128 output tiles, 64-deep K steps staged
//    through double-buffered, padded LDS tiles shared by 4 waves (64x64 each).
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

__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// Few rows: weight streaming.  MFMA operand A = 16 weight rows (output n),
// operand B = 16 node rows (output m); lane l supplies row (l & 15) and the
// 8 consecutive k at (l >> 4) * 8 of each 32-deep step.  The result lane l
// holds D[n = 4 (l >> 4) + i][m = l & 15], i = 0..3.
// ---------------------------------------------------------------------------
constexpr int kSkinnyWaves = 4;

template <int MT, int NT, int EPI>
__global__ __launch_bounds__(256) void proj_bf16_skinny(KArgs a) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int n0 = blockIdx.x * (16 * NT);
  const int M = a.M, N = a.N, K = a.K;
  const uint16_t* X = static_cast<const uint16_t*>(a.x);
  const uint16_t* Wt = static_cast<const uint16_t*>(a.w);

  // Rows past M or N are clamped to the last row: their sums are computed and
  // never stored.
  const uint16_t* xp[MT];
  const uint16_t* wp[NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) xp[mt] = X + int64_t(min(mt * 16 + r16, M - 1)) * K + kg * 8;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) wp[nt] = Wt + int64_t(min(n0 + nt * 16 + r16, N - 1)) * K + kg * 8;

  const int steps = K >> 5;
  const int per = (steps + kSkinnyWaves - 1) / kSkinnyWaves;
  const int s0 = wave * per;
  const int s1 = min(steps, s0 + per);

  f32x4 acc[NT][MT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[nt][mt] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll 4
  for (int s = s0; s < s1; ++s) {
    const int k = s << 5;
    bf16x8 xv[MT], wv[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) wv[nt] = load_bf16x8(wp[nt] + k);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) xv[mt] = load_bf16x8(xp[mt] + k);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[nt][mt] = mfma16(wv[nt], xv[mt], acc[nt][mt]);
  }

  __shared__ f32x4 red[kSkinnyWaves][NT * MT][64];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) red[wave][nt * MT + mt][lane] = acc[nt][mt];
  __syncthreads();

  for (int p = wave; p < NT * MT; p += kSkinnyWaves) {
    const int nt = p / MT, mt = p % MT;
    f32x4 v = red[0][p][lane];
#pragma unroll
    for (int w = 1; w < kSkinnyWaves; ++w) v += red[w][p][lane];
    const int m = mt * 16 + r16;
    if (m < M) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int n = n0 + nt * 16 + kg * 4 + i;
        if (n < N) emit<EPI, true>(a, m, n, v[i]);
      }
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

template <int MT, int NT>
hipError_t launch_skinny(const KArgs& k, int epi, hipStream_t s) {
  const dim3 grid((k.N + 16 * NT - 1) / (16 * NT));
  if (epi == EPI_LOGITS) hipLaunchKernelGGL((proj_bf16_skinny<MT, NT, EPI_LOGITS>), grid, dim3(256), 0, s, k);
  else hipLaunchKernelGGL((proj_bf16_skinny<MT, NT, EPI_HEAD>), grid, dim3(256), 0, s, k);
  return hipGetLastError();
}

template <int MT>
hipError_t launch_skinny_nt(const KArgs& k, int epi, hipStream_t s) {
  // Widest weight strip per block that still gives >= 1024 blocks.
  if ((k.N + 63) / 64 >= 1024) return launch_skinny<MT, 4>(k, epi, s);
  if ((k.N + 31) / 32 >= 1024) return launch_skinny<MT, 2>(k, epi, s);
  return launch_skinny<MT, 1>(k, epi, s);
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
  if (k.M <= 16) return launch_skinny_nt<1>(k, p.epilogue, s);
  if (k.M <= 32) return launch_skinny_nt<2>(k, p.epilogue, s);
  if (k.M <= 48) return launch_skinny_nt<3>(k, p.epilogue, s);
  if (k.M <= 64) return launch_skinny_nt<4>(k, p.epilogue, s);
  const dim3 grid((k.M + TBM - 1) / TBM, (k.N + TBN - 1) / TBN);
  if (p.epilogue == EPI_LOGITS) hipLaunchKernelGGL((proj_bf16_tiled<EPI_LOGITS>), grid, dim3(256), 0, s, k);
  else hipLaunchKernelGGL((proj_bf16_tiled<EPI_HEAD>), grid, dim3(256), 0, s, k);
  return hipGetLastError();
}

}  // namespace dartree
