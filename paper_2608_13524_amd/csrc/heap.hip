// Sequential correction with a best-first heap (Sec. 3.1, the node-at-a-time
// construction that Table 2 measures against DARTree), on the device.
//
// The correction head makes a prefix's children scoreable only after the
// head has run on that prefix, so pops and head evaluations alternate: pop
// the best prefix, run the head on it, offer its children, pop again.  One
// step per pop; the head, the logits and the softmax pass of the popped
// prefix (one row per request) run as ordinary launches before the step, and
// nothing returns to the host, so a whole round can be captured in a graph.
//
//  * heap_step: finishes the popped row's softmax/top-k (merging its segment
//    records, or the softmax over C_d with a shared candidate set), stores its
//    children in rank order, pops the best candidate and writes the popped
//    prefix's state r = act(tanh(t_parent + e U[token])) for the next step.
//    The heap is kept lazily: a prefix's children have non-increasing scores
//    in rank order, so each expanded prefix exposes only its next unpopped
//    child and a pop is one wavefront arg-min over at most budget + 1 keys
//    (the order (s desc, depth asc, parent slot asc, rank asc) is unchanged).
//  * heap_emit: flattens the popped prefixes in canonical breadth-first order
//    (depth, parent's output index, token) with the ancestor-or-self mask.
#include "reduce.hpp"

namespace dartree {
namespace {

constexpr int kHeapThreads = 256;
constexpr int kEmitThreads = 1024;
constexpr uint64_t kNone = ~0ull;

// Ascending pop key of the next child of slot `slot`: (s desc, depth asc,
// slot asc); depth < 256 and slot < 2^24, so a real key is never kNone.
__device__ __forceinline__ uint64_t heap_key(float s, int depth, int slot) {
  return (uint64_t(score_desc_key(s)) << 32) | (uint32_t(depth) << 24) | uint32_t(slot);
}
__device__ __forceinline__ int key_slot(uint64_t key) { return int(uint32_t(key) & 0xFFFFFFu); }
__device__ __forceinline__ int key_depth(uint64_t key) { return int((uint32_t(key) >> 24) & 0xFFu); }
__device__ __forceinline__ uint64_t wave_min_key(uint64_t x) { return ~wave_max_key(~x); }

// grid: batch, block (q): step a.step of request q.  Slot i = a.step was popped
// at the previous step (i = 0: the root) and, if above depth L, expanded by the
// launches in between.
template <int KB>
__global__ __launch_bounds__(kHeapThreads) void heap_step(HeapArgs a) {
  __shared__ float c_lp[DARTREE_MAX_CANDIDATES];   // slot i's children in rank order
  __shared__ int32_t c_tok[DARTREE_MAX_CANDIDATES];
  __shared__ __attribute__((aligned(16))) float rz[DARTREE_MAX_CANDIDATES];     // the row over C_d (shared set)
  __shared__ __attribute__((aligned(16))) int32_t rid[DARTREE_MAX_CANDIDATES];
  __shared__ int s_slot, s_tok;
  const int q = blockIdx.x, i = a.step;
  const int B = a.budget, L = a.depth, k = a.k, b = a.batch;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t sb = int64_t(q) * (B + 1);
  if (i > 0 && a.n_pop[q] != i) return;   // an earlier pop found the heap empty (block-uniform)
  const int d_i = i == 0 ? 0 : a.slot_depth[sb + i];
  const float s_i = i == 0 ? 0.f : a.slot_score[sb + i];
  const bool expand = d_i < L;
  const int64_t ci = int64_t(i) * b + q;  // step-major row of slot i's children

  // 1. slot i's children: log q~ and ids in rank order (z desc, id asc)
  if (expand && wave == 0) {
    const float scale = kLog2e / a.tau;
    if (a.shared_k > 0) {
      const int K = a.shared_k;
      const float* zr = a.zsh + int64_t(q) * K;
      const int32_t* set = a.cset + (int64_t(q) * L + d_i) * K;
      float m = -INFINITY;
      for (int c = lane; c < K; c += 64) {
        const float v = zr[c];
        rz[c] = v;
        rid[c] = min(max(set[c], 0), a.vocab - 1);   // workspace ids, clamped into U
        m = fmaxf(m, v);
      }
      m = wave_max(m);
      float sum = 0.f;
      for (int c = lane; c < K; c += 64) sum += __builtin_amdgcn_exp2f((rz[c] - m) * scale);
      const float log_s = logf(wave_sum(sum));
      __builtin_amdgcn_wave_barrier();
      for (int c = lane; c < K; c += 64) {
        const float v = rz[c];
        const int id = rid[c];
        // 16-byte reads of four values and four ids at a time (every lane
        // reads the same address), then the tail
        typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
        const f32x4* rz4 = reinterpret_cast<const f32x4*>(rz);
        const i32x4* rid4 = reinterpret_cast<const i32x4*>(rid);
        const int K4 = K & ~3;
        int rank = 0;
#pragma unroll 4
        for (int o = 0; o < K4; o += 4) {
          const f32x4 zv = rz4[o >> 2];
          const i32x4 iv = rid4[o >> 2];
          rank += int(better(zv[0], iv[0], v, id)) + int(better(zv[1], iv[1], v, id)) +
                  int(better(zv[2], iv[2], v, id)) + int(better(zv[3], iv[3], v, id));
        }
        for (int o = K4; o < K; ++o) rank += int(better(rz[o], rid[o], v, id));
        if (rank < k) {
          const float lp = (v - m) / a.tau - log_s;
          c_lp[rank] = lp;
          c_tok[rank] = id;
          a.ch_lp[ci * k + rank] = lp;
          a.ch_tok[ci * k + rank] = id;
        }
      }
      if (lane == 0) a.ch_lse[ci] = m / a.tau + log_s;
    } else if (a.nseg > 1) {
      uint64_t out[KB];
      const Partial p = wave_merge_records<KB>(a.part + int64_t(q) * a.nseg * record_floats<KB>(), a.nseg, k,
                                                scale, out);
      const float log_s = logf(p.s);
#pragma unroll
      for (int r = 0; r < KB; ++r) {
        if (r < k && lane == r) {
          const float lp = (key_value(out[r]) - p.m) / a.tau - log_s;
          const int id = key_id(out[r]);
          c_lp[r] = lp;
          c_tok[r] = id;
          a.ch_lp[ci * k + r] = lp;
          a.ch_tok[ci * k + r] = id;
        }
      }
      if (lane == 0) a.ch_lse[ci] = p.m / a.tau + log_s;
    } else {  // the softmax pass wrote the row in place
      for (int r = lane; r < k; r += 64) {
        c_lp[r] = a.ch_lp[ci * k + r];
        c_tok[r] = a.ch_tok[ci * k + r];
      }
    }
  }
  __syncthreads();

  // 2. pop the least key among the next children of slots 0 .. i
  if (wave == 0) {
    const uint64_t key_i = expand ? heap_key((s_i + c_lp[0]) + a.beta, d_i + 1, i) : kNone;
    uint64_t mine = lane == 0 ? key_i : kNone;
    for (int j = lane; j < i; j += 64) {
      const uint64_t kj = a.cand_key[sb + j];
      mine = kj < mine ? kj : mine;
    }
    const uint64_t best = wave_min_key(mine);
    if (lane == 0) {
      a.slot_nch[sb + i] = expand ? k : 0;
      a.slot_next[sb + i] = 0;
      a.cand_key[sb + i] = key_i;
      int next_slot = -1, tok = -1;
      if (i == 0) {  // the root
        a.slot_tok[sb] = -1;
        a.slot_par[sb] = -1;
        a.slot_depth[sb] = 0;
        a.slot_score[sb] = 0.f;
      }
      if (best != kNone) {
        const int p = key_slot(best), d = key_depth(best);
        const float s = score_from_desc_key(uint32_t(best >> 32));
        const int64_t cp = int64_t(p) * b + q;
        const int r = p == i ? 0 : a.slot_next[sb + p];
        const int nch = p == i ? k : a.slot_nch[sb + p];
        const float sp = p == i ? s_i : a.slot_score[sb + p];
        tok = p == i ? c_tok[r] : a.ch_tok[cp * k + r];
        uint64_t nk = kNone;
        if (r + 1 < nch) nk = heap_key((sp + (p == i ? c_lp[r + 1] : a.ch_lp[cp * k + r + 1])) + a.beta, d, p);
        a.slot_next[sb + p] = r + 1;
        a.cand_key[sb + p] = nk;
        a.slot_tok[sb + i + 1] = tok;
        a.slot_par[sb + i + 1] = p;
        a.slot_depth[sb + i + 1] = d;
        a.slot_score[sb + i + 1] = s;
        a.n_pop[q] = i + 1;
        a.group_index[q] = q * L + (d < L ? d : 0);
        if (d < L && i + 1 < B) next_slot = p;   // the last pop's children are never popped
      }
      s_slot = next_slot;
      s_tok = tok;
    }
  }
  __syncthreads();

  // 3. state of the popped prefix (slot i + 1), the next step's head input
  const int p = s_slot;
  if (p < 0) return;
  const int64_t tok = min(max(s_tok, 0), a.vocab - 1);   // an empty candidate (non-finite row) stays in U
  const int h = a.hidden;
  const float* tp = a.t_store + (int64_t(p) * b + q) * h;
  const int64_t ro = (int64_t(i + 1) * b + q) * h;
  if (a.precision == DARTREE_BF16) {
    typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
    const uint16_t* up = static_cast<const uint16_t*>(a.U) + tok * h;
    uint16_t* rp = static_cast<uint16_t*>(a.r_store) + ro;
    for (int x = threadIdx.x * 8; x < h; x += kHeapThreads * 8) {
      const f32x4 t0 = *reinterpret_cast<const f32x4*>(tp + x);
      const f32x4 t1 = *reinterpret_cast<const f32x4*>(tp + x + 4);
      const u16x8 u = *reinterpret_cast<const u16x8*>(up + x);
      u16x8 r;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float e0 = a.e * bf16_to_f32(u[j]), e1 = a.e * bf16_to_f32(u[j + 4]);
        r[j] = f32_to_bf16(a.markov ? e0 : tanhf(t0[j] + e0));
        r[j + 4] = f32_to_bf16(a.markov ? e1 : tanhf(t1[j] + e1));
      }
      *reinterpret_cast<u16x8*>(rp + x) = r;
    }
  } else {
    const float* up = static_cast<const float*>(a.U) + tok * h;
    float* rp = static_cast<float*>(a.r_store) + ro;
    for (int x = threadIdx.x; x < h; x += kHeapThreads) rp[x] = a.markov ? a.e * up[x] : tanhf(tp[x] + a.e * up[x]);
  }
}

// grid: batch.  Slots 1 .. n of request q are its popped prefixes; parents
// precede children, so output indices are assigned one depth at a time.
__global__ __launch_bounds__(kEmitThreads) void heap_emit(HeapArgs a, dartree_tree out) {
  constexpr int N = DARTREE_MAX_HEAP_BUDGET + 1;
  __shared__ int32_t tok[N], par[N], dep[N], oidx[N];
  __shared__ uint32_t rkey[N];
  __shared__ int32_t pout[DARTREE_MAX_HEAP_BUDGET];   // per output index: the parent's output index
  __shared__ int32_t per_depth[DARTREE_MAX_DEPTH + 1];
  const int q = blockIdx.x, B = a.budget, L = a.depth;
  const int64_t sb = int64_t(q) * (B + 1);
  const int n = min(max(a.n_pop[q], 0), B);
  for (int d = threadIdx.x; d <= L; d += blockDim.x) per_depth[d] = 0;
  for (int x = threadIdx.x; x <= n; x += blockDim.x) oidx[x] = -1;
  __syncthreads();
  // malformed parents or depths are clamped: nothing can index out of bounds
  for (int x = 1 + threadIdx.x; x <= n; x += blockDim.x) {
    tok[x] = a.slot_tok[sb + x];
    par[x] = min(max(a.slot_par[sb + x], 0), x - 1);
    dep[x] = min(max(a.slot_depth[sb + x], 1), L);
    atomicAdd(&per_depth[dep[x]], 1);
  }
  __syncthreads();
  int base = 0;
  for (int d = 1; d <= L; ++d) {
    const int nd = per_depth[d];
    if (nd == 0) break;   // popped prefixes are prefix-closed
    for (int x = 1 + threadIdx.x; x <= n; x += blockDim.x)
      if (dep[x] == d) rkey[x] = (uint32_t(d == 1 ? 0 : oidx[par[x]]) << 20) | (uint32_t(tok[x]) & 0xFFFFFu);
    __syncthreads();
    for (int x = 1 + threadIdx.x; x <= n; x += blockDim.x) {
      if (dep[x] != d) continue;
      const uint32_t mine = rkey[x];
      int r = 0;
      for (int y = 1; y <= n; ++y) r += int(dep[y] == d) & int(rkey[y] < mine);
      const int o = base + min(r, nd - 1);
      oidx[x] = o;
      pout[o] = d == 1 ? -1 : oidx[par[x]];
    }
    __syncthreads();
    base += nd;
  }
  const int64_t ob = int64_t(q) * B;
  for (int o = n + threadIdx.x; o < B; o += blockDim.x) {
    out.tokens[ob + o] = -1;
    out.parents[ob + o] = -1;
    out.depths[ob + o] = 0;
    out.scores[ob + o] = -INFINITY;
  }
  for (int x = 1 + threadIdx.x; x <= n; x += blockDim.x) {
    const int o = oidx[x];
    out.tokens[ob + o] = tok[x];
    out.parents[ob + o] = pout[o];
    out.depths[ob + o] = dep[x];
    out.scores[ob + o] = a.slot_score[sb + x];
  }
  const int words = (B + 63) / 64;
  const int64_t mb = int64_t(q) * B * words;
  for (int w = threadIdx.x; w < B * words; w += blockDim.x) {
    const int o = w / words, word = w % words;
    uint64_t bits = 0;
    if (o < n) {
      // parents precede children in the output, so the walk strictly decreases
      for (int j = o; j >= 0;) {
        if (j / 64 == word) bits |= 1ull << (j % 64);
        const int nx = pout[j];
        j = nx < j ? nx : -1;
      }
    }
    out.mask[mb + w] = bits;
  }
  if (threadIdx.x == 0) out.num_nodes[q] = n;
}

}  // namespace

hipError_t launch_heap_step(const HeapArgs& a, hipStream_t s) {
  if (a.batch <= 0) return hipSuccess;
  const dim3 grid(unsigned(a.batch)), block(kHeapThreads);
  switch ((a.shared_k > 0 || a.nseg <= 1) ? 1 : topk_bucket(a.k)) {
    case 1: hipLaunchKernelGGL((heap_step<1>), grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL((heap_step<2>), grid, block, 0, s, a); break;
    case 4: hipLaunchKernelGGL((heap_step<4>), grid, block, 0, s, a); break;
    case 8: hipLaunchKernelGGL((heap_step<8>), grid, block, 0, s, a); break;
    case 16: hipLaunchKernelGGL((heap_step<16>), grid, block, 0, s, a); break;
    default: hipLaunchKernelGGL((heap_step<32>), grid, block, 0, s, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_heap_emit(const HeapArgs& a, const dartree_tree& out, hipStream_t s) {
  if (a.batch <= 0) return hipSuccess;
  hipLaunchKernelGGL(heap_emit, dim3(unsigned(a.batch)), dim3(kEmitThreads), 0, s, a, out);
  return hipGetLastError();
}

}  // namespace dartree
