// C ABI of libdartree: argument validation, workspace layout and the order
// of kernel launches for one round of Algorithm 1.  No function here touches
// the device until every argument has been checked.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "internal.hpp"

using namespace dartree;

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t act_bytes(int precision) { return precision == DARTREE_BF16 ? 2 : 4; }

// Level sizes n_d = min(W, n_{d-1} k), n_0 = 1, and derived extents.
struct Shape {
  int64_t n[DARTREE_MAX_DEPTH + 1];  // n[0] = 1, n[d] for d = 1..L
  int64_t total;                     // |S| per request
  int64_t max_parent;                // max_d n_{d-1}
  int64_t max_cand;                  // max_d n_{d-1} k
};

Shape shape_of(const dartree_params& p) {
  Shape s{};
  s.n[0] = 1;
  s.total = 0;
  s.max_parent = 1;
  s.max_cand = 0;
  for (int d = 1; d <= p.depth; ++d) {
    s.max_parent = std::max(s.max_parent, s.n[d - 1]);
    s.max_cand = std::max(s.max_cand, s.n[d - 1] * p.branch);
    s.n[d] = std::min<int64_t>(p.width, s.n[d - 1] * p.branch);
    s.total += s.n[d];
  }
  return s;
}

// Workspace layout (each region 256-byte aligned), R = b * W rows:
//   hdr: u32 [4] {params key lo, key hi, last depth completed, 0} (written by
//        the selection kernel of each depth; read by the debug order check)
//   lvl_tok, lvl_par: i32 [L][b][W]     lvl_score: f32 [L][b][W]
//   lse: f32 [L][R]   cand_logp: f32 [L][R][k]   cand_ids: i32 [L][R][k]
//   state: act [2][R][h]   t: f32 [R][h]   a: act [R][h]   z: f32 [R][V]
//   k3: the row-split partials of the largest depth
//   cset: i32 [b][L][K] shared candidate sets and their chunk winners (K > 0)
//   split: partial sums of the projection tiles split along K (the head and
//          the logits of one depth run one after the other and share it)
struct Layout {
  size_t hdr, lvl_tok, lvl_par, lvl_score, lse, cand_logp, cand_ids, state0, state1, t, a, z, k3, cset, cset_scratch,
      split, split_bytes, total;
};

Layout layout_of(const dartree_params& p, const Shape& s) {
  const size_t L = p.depth, b = p.batch, W = p.width, k = p.branch, h = p.hidden, V = p.vocab;
  const size_t R = b * W;
  const size_t K = size_t(p.candidates);
  size_t k3 = 0, split = 0;
  if (K == 0)
    for (int d = 1; d <= p.depth; ++d) k3 = std::max(k3, lse_topk_scratch_bytes(int64_t(b) * s.n[d - 1], V, int(k)));
  for (int d = 1; d <= p.depth; ++d) {
    const int64_t rows = int64_t(b) * s.n[d - 1];
    split = std::max(split, proj_split_bytes(p.precision, EPI_HEAD, rows, int64_t(h), int64_t(h)));
    if (K == 0) split = std::max(split, proj_split_bytes(p.precision, EPI_LOGITS, rows, int64_t(V), int64_t(h)));
  }
  Layout l{};
  size_t o = 0;
  auto take = [&](size_t bytes) { const size_t at = o; o = align_up(o + bytes); return at; };
  l.hdr = take(16);
  l.lvl_tok = take(L * b * W * 4);
  l.lvl_par = take(L * b * W * 4);
  l.lvl_score = take(L * b * W * 4);
  l.lse = take(L * R * 4);
  l.cand_logp = take(L * R * k * 4);
  l.cand_ids = take(L * R * k * 4);
  l.state0 = take(R * h * act_bytes(p.precision));
  l.state1 = take(R * h * act_bytes(p.precision));
  l.t = take(R * h * 4);
  l.a = take(R * h * act_bytes(p.precision));
  l.z = take(R * (K > 0 ? K : V) * 4);   // logits over C_d only with a shared set
  l.k3 = take(k3);
  l.cset = take(b * L * K * 4);
  l.cset_scratch = take(K > 0 ? candidate_sets_scratch_bytes(int64_t(b) * L, V, int(K)) : 0);
  l.split = take(split);
  l.split_bytes = split;
  l.total = o;
  return l;
}

// Checks shared by the depth-wise construction and the sequential heap
// (which does not use the width).
dartree_status validate_common(const dartree_params* p) {
  if (!p) return DARTREE_ERR_INVALID_ARG;
  if (p->batch < 1 || p->vocab < 1 || p->hidden < 1 || p->depth < 1 || p->branch < 1 || p->budget < 1)
    return DARTREE_ERR_INVALID_ARG;
  if (p->branch > p->vocab) return DARTREE_ERR_INVALID_ARG;
  if (p->candidates < 0) return DARTREE_ERR_INVALID_ARG;
  if (p->candidates > 0 && (p->candidates > p->vocab || p->branch > p->candidates)) return DARTREE_ERR_INVALID_ARG;
  if (p->precision != DARTREE_FP32 && p->precision != DARTREE_BF16) return DARTREE_ERR_INVALID_ARG;
  if (p->head != DARTREE_HEAD_RNN && p->head != DARTREE_HEAD_MARKOV) return DARTREE_ERR_INVALID_ARG;
  if (!isfinite(p->temperature) || p->temperature < 0.f) return DARTREE_ERR_INVALID_ARG;
  if (!isfinite(p->depth_bonus) || p->depth_bonus > 0.f) return DARTREE_ERR_INVALID_ARG;
  if (p->vocab > DARTREE_MAX_VOCAB || p->depth > DARTREE_MAX_DEPTH) return DARTREE_ERR_UNSUPPORTED;
  if (p->candidates == 0 && p->branch > DARTREE_MAX_BRANCH) return DARTREE_ERR_UNSUPPORTED;
  if (p->candidates > 0 &&
      (p->candidates > DARTREE_MAX_CANDIDATES || !candidate_sets_supported(p->vocab, p->candidates)))
    return DARTREE_ERR_UNSUPPORTED;
  if (p->precision == DARTREE_BF16 && p->hidden % 64 != 0) return DARTREE_ERR_UNSUPPORTED;
  return DARTREE_OK;
}

dartree_status validate(const dartree_params* p) {
  dartree_status v = validate_common(p);
  if (v != DARTREE_OK) return v;
  if (p->width < 1) return DARTREE_ERR_INVALID_ARG;
  if (p->width > DARTREE_MAX_WIDTH || p->budget > DARTREE_MAX_SORT) return DARTREE_ERR_UNSUPPORTED;
  const Shape s = shape_of(*p);
  if (s.max_cand > DARTREE_MAX_SORT || s.total > DARTREE_MAX_SORT) return DARTREE_ERR_UNSUPPORTED;
  // row counts and element offsets must stay within 32-bit grid/row indexing
  if (int64_t(p->batch) * p->width > (int64_t(1) << 24)) return DARTREE_ERR_UNSUPPORTED;
  return DARTREE_OK;
}

dartree_status check_inputs(const dartree_inputs* in) {
  if (!in || !in->drafter_logits || !in->drafter_hidden || !in->prefix_state || !in->head_A || !in->head_U)
    return DARTREE_ERR_INVALID_ARG;
  if (!aligned16(in->drafter_logits) || !aligned16(in->drafter_hidden) || !aligned16(in->prefix_state) ||
      !aligned16(in->head_A) || !aligned16(in->head_U))
    return DARTREE_ERR_INVALID_ARG;
  return DARTREE_OK;
}

dartree_status check_tree(const dartree_tree* t) {
  if (!t || !t->tokens || !t->parents || !t->depths || !t->scores || !t->mask || !t->num_nodes)
    return DARTREE_ERR_INVALID_ARG;
  if (!aligned16(t->tokens) || !aligned16(t->parents) || !aligned16(t->depths) || !aligned16(t->scores) ||
      !aligned16(t->mask) || !aligned16(t->num_nodes))
    return DARTREE_ERR_INVALID_ARG;
  return DARTREE_OK;
}

dartree_status check_ws(const dartree_params& p, const void* ws, size_t ws_bytes, Layout* out) {
  const Layout l = layout_of(p, shape_of(p));
  if (!ws || (reinterpret_cast<uintptr_t>(ws) % kAlign) != 0 || ws_bytes < l.total) return DARTREE_ERR_WORKSPACE;
  *out = l;
  return DARTREE_OK;
}

template <typename T>
T* at(void* base, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(base) + off);
}
template <typename T>
const T* at(const void* base, size_t off) {
  return reinterpret_cast<const T*>(static_cast<const char*>(base) + off);
}

dartree_status hip_status(hipError_t e) { return e == hipSuccess ? DARTREE_OK : DARTREE_ERR_HIP; }

// ---------------------------------------------------------------------------
// Depth order (Algorithm 1's loop runs d = 1..L, each depth reading the level
// and states the previous one left in the workspace).
//
// Host record, always on: for each workspace the parameters it was last used
// with and the last depth enqueued on it.  expand_depth(d > 1) needs d - 1,
// prune needs L; otherwise DARTREE_ERR_ORDER before anything is enqueued.
// The record follows the host calls: replays of a captured graph do not
// update it.  At most kOrderSlots workspaces are remembered (least recently
// used dropped; a dropped one must start again at depth 1).
//
// Device record: the selection kernel of depth d writes {key, d} into the
// workspace header.  With DARTREE_DEBUG=1 in the environment (read once),
// expand_depth(d > 1) and prune also synchronise the stream and compare that
// record with the depth they need, and expand_depth checks after its launches
// that the depth's normalisers are finite (DARTREE_ERR_NONFINITE).  Debug
// checks are skipped while the stream is being captured.
// ---------------------------------------------------------------------------
uint64_t params_key(const dartree_params& p) {
  uint64_t h = 1469598103934665603ull;   // FNV-1a over the struct's bytes
  const unsigned char* b = reinterpret_cast<const unsigned char*>(&p);
  for (size_t i = 0; i < sizeof(p); ++i) h = (h ^ b[i]) * 1099511628211ull;
  return h | 1;   // never 0, so a zeroed header never matches
}

struct OrderSlot {
  const void* ws;
  uint64_t key;
  int depth;
  uint64_t used;
};
constexpr size_t kOrderSlots = 256;
std::mutex g_order_mu;
std::vector<OrderSlot> g_order;
uint64_t g_order_tick = 0;

int order_depth(const void* ws, uint64_t key) {
  std::lock_guard<std::mutex> lk(g_order_mu);
  for (OrderSlot& o : g_order)
    if (o.ws == ws) return o.key == key ? (o.used = ++g_order_tick, o.depth) : -1;
  return -1;
}

void order_set(const void* ws, uint64_t key, int depth) {
  std::lock_guard<std::mutex> lk(g_order_mu);
  for (OrderSlot& o : g_order)
    if (o.ws == ws) {
      o = OrderSlot{ws, key, depth, ++g_order_tick};
      return;
    }
  if (g_order.size() >= kOrderSlots)
    g_order.erase(std::min_element(g_order.begin(), g_order.end(),
                                   [](const OrderSlot& a, const OrderSlot& b) { return a.used < b.used; }));
  g_order.push_back(OrderSlot{ws, key, depth, ++g_order_tick});
}

bool debug_mode() {
  static const bool on = [] {
    const char* v = getenv("DARTREE_DEBUG");
    return v && v[0] && strcmp(v, "0") != 0;
  }();
  return on;
}

bool capturing(hipStream_t st) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  return hipStreamIsCapturing(st, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone;
}

// Debug: the depth the device record of `ws` holds for these parameters
// (-1: none), after the stream's work so far.
dartree_status device_depth(const void* ws, size_t hdr, uint64_t key, hipStream_t st, int* depth) {
  uint32_t rec[3] = {0, 0, 0};
  if (hipStreamSynchronize(st) != hipSuccess) return DARTREE_ERR_HIP;
  if (hipMemcpy(rec, static_cast<const char*>(ws) + hdr, sizeof(rec), hipMemcpyDeviceToHost) != hipSuccess)
    return DARTREE_ERR_HIP;
  const bool same = rec[0] == uint32_t(key) && rec[1] == uint32_t(key >> 32);
  *depth = same ? int(rec[2]) : -1;
  return DARTREE_OK;
}

LevelShape level_shape(const dartree_params& p, const Shape& s) {
  LevelShape ls{};
  ls.depth = p.depth;
  ls.width = p.width;
  ls.off[0] = 0;
  for (int d = 1; d <= p.depth; ++d) {
    ls.n[d - 1] = int32_t(s.n[d]);
    ls.off[d] = ls.off[d - 1] + int32_t(s.n[d]);
  }
  return ls;
}

// Optional event pair around one launch (see dartree_build_tree_timed).
struct Timer {
  hipEvent_t* ev = nullptr;
  hipStream_t st = nullptr;
  void mark(int index, int which) const {
    if (ev && ev[2 * index + which]) (void)hipEventRecord(ev[2 * index + which], st);
  }
};

// Depth d with a shared candidate set (after K1): the sets of every depth at
// d = 1, the logits over C_d, then selection and state update.
dartree_status expand_shared(const dartree_params& p, const dartree_inputs& in, int d, void* ws, const Layout& l,
                             const Shape& s, hipStream_t st, const Timer& tm, const float* t, const void* a, float* z,
                             void* r_out) {
  const int tb = (d - 1) * DARTREE_KERNELS_PER_DEPTH;
  const int64_t b = p.batch, V = p.vocab, h = p.hidden, L = p.depth, W = p.width, k = p.branch;
  const int K = p.candidates;
  const int64_t np = s.n[d - 1], nc = s.n[d];
  int32_t* csets = at<int32_t>(ws, l.cset);
  const float tau = p.temperature > 0.f ? p.temperature : 1.f;
  hipError_t err;
  tm.mark(tb + DARTREE_KERNEL_LSE, 0);   // marked at every depth; the sets are built at d = 1
  if (d == 1) {
    err = launch_candidate_sets(in.drafter_logits, b * L, V, K, csets, at<char>(ws, l.cset_scratch), st);
    if (err != hipSuccess) return DARTREE_ERR_HIP;
  }
  tm.mark(tb + DARTREE_KERNEL_LSE, 1);
  tm.mark(tb + DARTREE_KERNEL_LOGITS, 0);
  err = launch_shared_logits(p.precision, int(b), int(np), K, int(h), int(V), a, in.head_U,
                             in.drafter_logits + size_t(d - 1) * V, L * V, csets + (d - 1) * K, L * K, nullptr, z, st);
  tm.mark(tb + DARTREE_KERNEL_LOGITS, 1);
  if (err != hipSuccess) return DARTREE_ERR_HIP;

  LevelArgs la{};
  la.batch = int(b);
  la.n_parent = int(np);
  la.k = int(k);
  la.n_keep = int(nc);
  la.beta = p.depth_bonus;
  la.tau = tau;
  la.parent_stride = int(W);
  la.out_stride = int(W);
  la.parent_score = d == 1 ? nullptr : at<float>(ws, l.lvl_score) + (d - 2) * b * W;
  la.nseg = 1;
  la.rows_ranked = 1;
  la.lse = at<float>(ws, l.lse) + (d - 1) * b * W;
  la.cand_logp = at<float>(ws, l.cand_logp) + (d - 1) * b * W * k;
  la.cand_ids = at<int32_t>(ws, l.cand_ids) + (d - 1) * b * W * k;
  la.out_tok = at<int32_t>(ws, l.lvl_tok) + (d - 1) * b * W;
  la.out_par = at<int32_t>(ws, l.lvl_par) + (d - 1) * b * W;
  la.out_score = at<float>(ws, l.lvl_score) + (d - 1) * b * W;
  la.shared_k = K;
  la.zsh = z;
  la.cset = csets + (d - 1) * K;
  la.cset_stride = L * K;
  la.state = d < p.depth;
  la.precision = p.precision;
  la.hidden = int(h);
  la.vocab = int(V);
  la.markov = p.head == DARTREE_HEAD_MARKOV;
  la.t = t;
  la.U = in.head_U;
  la.e = float(sqrt(double(p.hidden)));
  la.r_out = r_out;
  const uint64_t key = params_key(p);
  la.stamp = at<uint32_t>(ws, l.hdr);
  la.stamp_key_lo = uint32_t(key);
  la.stamp_key_hi = uint32_t(key >> 32);
  la.stamp_depth = d;
  tm.mark(tb + DARTREE_KERNEL_SELECT, 0);
  err = launch_select_level(la, st);
  tm.mark(tb + DARTREE_KERNEL_SELECT, 1);
  return err == hipSuccess ? DARTREE_OK : DARTREE_ERR_HIP;
}

// Enqueue depth d (validated arguments).
dartree_status expand(const dartree_params& p, const dartree_inputs& in, int d, void* ws, const Layout& l,
                      const Shape& s, hipStream_t st, const Timer& tm = Timer()) {
  const int tb = (d - 1) * DARTREE_KERNELS_PER_DEPTH;
  const int64_t b = p.batch, V = p.vocab, h = p.hidden, L = p.depth, W = p.width, k = p.branch;
  const int64_t np = s.n[d - 1], nc = s.n[d];
  const int64_t R = b * np;  // parent rows of this depth
  const size_t ab = act_bytes(p.precision);
  const void* r_in = d == 1 ? in.prefix_state : at<char>(ws, (d - 1) % 2 ? l.state1 : l.state0);
  void* r_out = at<char>(ws, d % 2 ? l.state1 : l.state0);
  float* t = at<float>(ws, l.t);
  void* a = at<char>(ws, l.a);
  float* z = at<float>(ws, l.z);
  float* lse = at<float>(ws, l.lse) + (d - 1) * b * W;
  float* clp = at<float>(ws, l.cand_logp) + (d - 1) * b * W * k;
  int32_t* cid = at<int32_t>(ws, l.cand_ids) + (d - 1) * b * W * k;
  int32_t* tok = at<int32_t>(ws, l.lvl_tok) + (d - 1) * b * W;
  int32_t* par = at<int32_t>(ws, l.lvl_par) + (d - 1) * b * W;
  float* score = at<float>(ws, l.lvl_score) + (d - 1) * b * W;
  const float* parent_score = d == 1 ? nullptr : at<float>(ws, l.lvl_score) + (d - 2) * b * W;
  const float tau = p.temperature > 0.f ? p.temperature : 1.f;
  const float e = float(sqrt(double(p.hidden)));

  // K1: t = A r, a = act(tanh(t + H_d))
  ProjArgs head{};
  head.precision = p.precision;
  head.epilogue = EPI_HEAD;
  head.M = R;
  head.N = h;
  head.K = h;
  head.rows_per_group = np;
  head.x = r_in;
  head.w = in.head_A;
  head.bias_act = static_cast<const char*>(in.drafter_hidden) + size_t(d - 1) * h * ab;
  head.bias_stride = L * h;
  head.out = t;
  head.act_out = a;
  head.split = l.split_bytes ? at<float>(ws, l.split) : nullptr;
  tm.mark(tb + DARTREE_KERNEL_HEAD, 0);
  hipError_t err = launch_project(head, st);
  tm.mark(tb + DARTREE_KERNEL_HEAD, 1);
  if (err != hipSuccess) return DARTREE_ERR_HIP;

  if (p.candidates > 0) return expand_shared(p, in, d, ws, l, s, st, tm, t, a, z, r_out);

  // K2: z = L_d^base + U a
  ProjArgs lg{};
  lg.precision = p.precision;
  lg.epilogue = EPI_LOGITS;
  lg.M = R;
  lg.N = V;
  lg.K = h;
  lg.rows_per_group = np;
  lg.x = a;
  lg.w = in.head_U;
  lg.bias_f32 = in.drafter_logits + size_t(d - 1) * V;
  lg.bias_stride = L * V;
  lg.out = z;
  lg.split = l.split_bytes ? at<float>(ws, l.split) : nullptr;
  tm.mark(tb + DARTREE_KERNEL_LOGITS, 0);
  err = launch_project(lg, st);
  tm.mark(tb + DARTREE_KERNEL_LOGITS, 1);
  if (err != hipSuccess) return DARTREE_ERR_HIP;

  // K3: lse and top-k per parent row.  Segment records, if any, are merged
  // by K4, whose block takes a request's parent rows one per wave; with more
  // parent rows per request than it has waves (measured at 32 rows: 311 us of
  // selection per round against 152 + 78 more in this launch), the softmax
  // launch merges them itself, one block per row, and K4 reads finished
  // candidates.
  const bool merge_here = np > select_level_waves(int(k)) && lse_topk_segments(R, V) > 1;
  tm.mark(tb + DARTREE_KERNEL_LSE, 0);
  err = launch_lse_topk(z, R, V, int(k), tau, lse, clp, cid, at<char>(ws, l.k3), merge_here, st);
  tm.mark(tb + DARTREE_KERNEL_LSE, 1);
  if (err != hipSuccess) return DARTREE_ERR_HIP;

  // K4 (+ K5): S_d = segmented top-W, level arrays with stride W per request,
  // and the states of the kept children (unused after the last depth)
  LevelArgs la{};
  la.batch = int(b);
  la.n_parent = int(np);
  la.k = int(k);
  la.n_keep = int(nc);
  la.beta = p.depth_bonus;
  la.tau = tau;
  la.parent_stride = int(W);
  la.out_stride = int(W);
  la.parent_score = parent_score;
  la.nseg = merge_here ? 1 : lse_topk_segments(R, V);
  la.rows_ranked = 1;
  la.part = at<float>(ws, l.k3);
  la.lse = lse;
  la.cand_logp = clp;
  la.cand_ids = cid;
  la.out_tok = tok;
  la.out_par = par;
  la.out_score = score;
  la.state = d < p.depth;
  la.precision = p.precision;
  la.hidden = int(h);
  la.vocab = int(V);
  la.markov = p.head == DARTREE_HEAD_MARKOV;
  la.t = t;
  la.U = in.head_U;
  la.e = e;
  la.r_out = r_out;
  const uint64_t key = params_key(p);
  la.stamp = at<uint32_t>(ws, l.hdr);
  la.stamp_key_lo = uint32_t(key);
  la.stamp_key_hi = uint32_t(key >> 32);
  la.stamp_depth = d;
  tm.mark(tb + DARTREE_KERNEL_SELECT, 0);
  err = launch_select_level(la, st);
  tm.mark(tb + DARTREE_KERNEL_SELECT, 1);
  if (err != hipSuccess) return DARTREE_ERR_HIP;
  return DARTREE_OK;
}

// ---------------------------------------------------------------------------
// Sequential correction with a best-first heap (Sec. 3.1)
// ---------------------------------------------------------------------------
dartree_status validate_heap(const dartree_params* p) {
  dartree_status v = validate_common(p);
  if (v != DARTREE_OK) return v;
  if (p->budget > DARTREE_MAX_HEAP_BUDGET) return DARTREE_ERR_UNSUPPORTED;
  if (int64_t(p->batch) * (p->budget + 1) > (int64_t(1) << 24)) return DARTREE_ERR_UNSUPPORTED;
  return DARTREE_OK;
}

// Heap workspace (each region 256-byte aligned), S = b (B + 1) slots:
//   slot_tok, slot_par, slot_depth, slot_next, slot_nch: i32 [b][B+1]
//   slot_score: f32 [b][B+1]   cand_key: u64 [b][B+1]
//   ch_lse: f32 [B][b]   ch_lp: f32 [B][b][k]   ch_tok: i32 [B][b][k]
//   n_pop, gidx: i32 [b]
//   r_store: act [B+1][b][h]   t_store: f32 [B][b][h]   a_store: act [B][b][h] (step i's features)
//   z: f32 [b][V] (or [b][K])   k3: the row-split partials of b rows
//   cset: i32 [b][L][K] and its scratch (K > 0)
struct HeapLayout {
  size_t slot_tok, slot_par, slot_depth, slot_score, slot_next, slot_nch, cand_key, ch_lse, ch_lp, ch_tok, n_pop,
      gidx, r_store, t_store, a, z, k3, cset, cset_scratch, total;
};

HeapLayout heap_layout_of(const dartree_params& p) {
  const size_t L = p.depth, b = p.batch, B = p.budget, k = p.branch, h = p.hidden, V = p.vocab;
  const size_t K = size_t(p.candidates), ab = act_bytes(p.precision);
  const size_t S = b * (B + 1);
  HeapLayout l{};
  size_t o = 0;
  auto take = [&](size_t bytes) { const size_t at = o; o = align_up(o + bytes); return at; };
  l.slot_tok = take(S * 4);
  l.slot_par = take(S * 4);
  l.slot_depth = take(S * 4);
  l.slot_score = take(S * 4);
  l.slot_next = take(S * 4);
  l.slot_nch = take(S * 4);
  l.cand_key = take(S * 8);
  l.ch_lse = take(B * b * 4);
  l.ch_lp = take(B * b * k * 4);
  l.ch_tok = take(B * b * k * 4);
  l.n_pop = take(b * 4);
  l.gidx = take(b * 4);
  l.r_store = take((B + 1) * b * h * ab);
  l.t_store = take(B * b * h * 4);
  l.a = take(B * b * h * ab);
  l.z = take(b * (K > 0 ? K : V) * 4);
  l.k3 = take(K > 0 ? 0 : lse_topk_scratch_bytes(int64_t(b), V, int(k)));
  l.cset = take(b * L * K * 4);
  l.cset_scratch = take(K > 0 ? candidate_sets_scratch_bytes(int64_t(b) * L, V, int(K)) : 0);
  l.total = o;
  return l;
}

dartree_status check_heap_ws(const dartree_params& p, const void* ws, size_t ws_bytes, HeapLayout* out) {
  const HeapLayout l = heap_layout_of(p);
  if (!ws || (reinterpret_cast<uintptr_t>(ws) % kAlign) != 0 || ws_bytes < l.total) return DARTREE_ERR_WORKSPACE;
  *out = l;
  return DARTREE_OK;
}

// One round: B steps of (head, logits, softmax pass, heap step) on the prefix
// popped at the previous step (step 0: the root), then the emission.  Step 0
// reads depth 1's rows directly; later steps read the rows the heap step
// chose (group index q L + depth of the popped prefix).
dartree_status build_heap(const dartree_params& p, const dartree_inputs& in, void* ws, const HeapLayout& l,
                          const dartree_tree& out, hipStream_t st) {
  const int64_t b = p.batch, V = p.vocab, h = p.hidden, L = p.depth, B = p.budget, k = p.branch;
  const int K = p.candidates;
  const size_t ab = act_bytes(p.precision);
  int32_t* gidx = at<int32_t>(ws, l.gidx);
  int32_t* csets = at<int32_t>(ws, l.cset);
  float* z = at<float>(ws, l.z);
  void* a = at<char>(ws, l.a);
  HeapArgs ha{};
  ha.batch = int(b);
  ha.budget = int(B);
  ha.depth = int(L);
  ha.k = int(k);
  ha.vocab = int(V);
  ha.markov = p.head == DARTREE_HEAD_MARKOV;
  ha.shared_k = K;
  ha.beta = p.depth_bonus;
  ha.tau = p.temperature > 0.f ? p.temperature : 1.f;
  ha.e = float(sqrt(double(p.hidden)));
  ha.precision = p.precision;
  ha.hidden = int(h);
  ha.nseg = K > 0 ? 1 : lse_topk_segments(b, V);
  ha.part = at<float>(ws, l.k3);
  ha.zsh = z;
  ha.cset = csets;
  ha.slot_tok = at<int32_t>(ws, l.slot_tok);
  ha.slot_par = at<int32_t>(ws, l.slot_par);
  ha.slot_depth = at<int32_t>(ws, l.slot_depth);
  ha.slot_score = at<float>(ws, l.slot_score);
  ha.slot_next = at<int32_t>(ws, l.slot_next);
  ha.slot_nch = at<int32_t>(ws, l.slot_nch);
  ha.cand_key = at<uint64_t>(ws, l.cand_key);
  ha.ch_lse = at<float>(ws, l.ch_lse);
  ha.ch_lp = at<float>(ws, l.ch_lp);
  ha.ch_tok = at<int32_t>(ws, l.ch_tok);
  ha.n_pop = at<int32_t>(ws, l.n_pop);
  ha.group_index = gidx;
  ha.t_store = at<float>(ws, l.t_store);
  ha.U = in.head_U;
  ha.r_store = at<char>(ws, l.r_store);
  hipError_t err = hipSuccess;
  if (K > 0) {
    err = launch_candidate_sets(in.drafter_logits, b * L, V, K, csets, at<char>(ws, l.cset_scratch), st);
    if (err != hipSuccess) return DARTREE_ERR_HIP;
  }
  for (int64_t i = 0; i < B; ++i) {
    const int32_t* gi = i == 0 ? nullptr : gidx;
    void* a_i = static_cast<char*>(a) + size_t(i) * b * h * ab;   // step i's features, kept for inspection
    ProjArgs head{};
    head.precision = p.precision;
    head.epilogue = EPI_HEAD;
    head.M = b;
    head.N = h;
    head.K = h;
    head.rows_per_group = 1;
    head.x = i == 0 ? in.prefix_state : static_cast<const void*>(at<char>(ws, l.r_store) + size_t(i) * b * h * ab);
    head.w = in.head_A;
    head.bias_act = in.drafter_hidden;
    head.bias_stride = i == 0 ? L * h : h;
    head.group_index = gi;
    head.out = at<float>(ws, l.t_store) + size_t(i) * b * h;
    head.act_out = a_i;
    if ((err = launch_project(head, st)) != hipSuccess) return DARTREE_ERR_HIP;
    if (K > 0) {
      err = launch_shared_logits(p.precision, int(b), 1, K, int(h), int(V), a_i, in.head_U,
                                 in.drafter_logits, i == 0 ? L * V : V, csets, i == 0 ? L * K : K, gi, z, st);
      if (err != hipSuccess) return DARTREE_ERR_HIP;
    } else {
      ProjArgs lg{};
      lg.precision = p.precision;
      lg.epilogue = EPI_LOGITS;
      lg.M = b;
      lg.N = V;
      lg.K = h;
      lg.rows_per_group = 1;
      lg.x = a_i;
      lg.w = in.head_U;
      lg.bias_f32 = in.drafter_logits;
      lg.bias_stride = i == 0 ? L * V : V;
      lg.group_index = gi;
      lg.out = z;
      if ((err = launch_project(lg, st)) != hipSuccess) return DARTREE_ERR_HIP;
      err = launch_lse_topk(z, b, V, int(k), ha.tau, ha.ch_lse + i * b, ha.ch_lp + i * b * k, ha.ch_tok + i * b * k,
                            at<char>(ws, l.k3), false, st);
      if (err != hipSuccess) return DARTREE_ERR_HIP;
    }
    ha.step = int(i);
    if ((err = launch_heap_step(ha, st)) != hipSuccess) return DARTREE_ERR_HIP;
  }
  return hip_status(launch_heap_emit(ha, out, st));
}

}  // namespace

extern "C" {

int32_t dartree_abi_version(void) { return DARTREE_ABI_VERSION; }

const char* dartree_status_string(dartree_status status) {
  switch (status) {
    case DARTREE_OK: return "ok";
    case DARTREE_ERR_INVALID_ARG: return "invalid argument";
    case DARTREE_ERR_UNSUPPORTED: return "unsupported: beyond this library's limits";
    case DARTREE_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case DARTREE_ERR_HIP: return "HIP kernel launch failed";
    case DARTREE_ERR_ORDER: return "depths out of order: the workspace does not hold the levels this call reads";
    case DARTREE_ERR_NONFINITE: return "non-finite normaliser (debug check)";
  }
  return "unknown status";
}

dartree_status dartree_validate(const dartree_params* p) { return validate(p); }

dartree_status dartree_workspace_size(const dartree_params* p, size_t* bytes) {
  if (!bytes) return DARTREE_ERR_INVALID_ARG;
  const dartree_status v = validate(p);
  if (v != DARTREE_OK) return v;
  *bytes = layout_of(*p, shape_of(*p)).total;
  return DARTREE_OK;
}

dartree_status dartree_expand_depth(const dartree_params* p, const dartree_inputs* in, int32_t d, void* ws,
                                    size_t ws_bytes, hipStream_t stream) {
  dartree_status v = validate(p);
  if (v != DARTREE_OK) return v;
  if ((v = check_inputs(in)) != DARTREE_OK) return v;
  if (d < 1 || d > p->depth) return DARTREE_ERR_INVALID_ARG;
  Layout l;
  if ((v = check_ws(*p, ws, ws_bytes, &l)) != DARTREE_OK) return v;
  const uint64_t key = params_key(*p);
  if (d > 1 && order_depth(ws, key) != d - 1) return DARTREE_ERR_ORDER;
  const bool dbg = debug_mode() && !capturing(stream);
  if (dbg && d > 1) {
    int dev_d = -1;
    if ((v = device_depth(ws, l.hdr, key, stream, &dev_d)) != DARTREE_OK) return v;
    if (dev_d != d - 1) return DARTREE_ERR_ORDER;
  }
  if ((v = expand(*p, *in, d, ws, l, shape_of(*p), stream)) != DARTREE_OK) return v;
  order_set(ws, key, d);
  if (dbg) {   // the depth's normalisers, one per parent row
    const Shape s = shape_of(*p);
    std::vector<float> lse(size_t(p->batch) * s.n[d - 1]);
    if (hipStreamSynchronize(stream) != hipSuccess ||
        hipMemcpy(lse.data(), at<char>(ws, l.lse + size_t(d - 1) * p->batch * p->width * 4), lse.size() * 4,
                  hipMemcpyDeviceToHost) != hipSuccess)
      return DARTREE_ERR_HIP;
    for (float x : lse)
      if (!isfinite(x)) return DARTREE_ERR_NONFINITE;
  }
  return DARTREE_OK;
}

dartree_status dartree_prune(const dartree_params* p, const void* ws, size_t ws_bytes, const dartree_tree* out,
                             hipStream_t stream) {
  dartree_status v = validate(p);
  if (v != DARTREE_OK) return v;
  if ((v = check_tree(out)) != DARTREE_OK) return v;
  Layout l;
  if ((v = check_ws(*p, ws, ws_bytes, &l)) != DARTREE_OK) return v;
  const uint64_t key = params_key(*p);
  if (order_depth(ws, key) != p->depth) return DARTREE_ERR_ORDER;
  if (debug_mode() && !capturing(stream)) {
    int dev_d = -1;
    if ((v = device_depth(ws, l.hdr, key, stream, &dev_d)) != DARTREE_OK) return v;
    if (dev_d != p->depth) return DARTREE_ERR_ORDER;
  }
  const Shape s = shape_of(*p);
  return hip_status(launch_prune_emit(p->batch, level_shape(*p, s), p->budget, at<int32_t>(ws, l.lvl_tok),
                                      at<int32_t>(ws, l.lvl_par), at<float>(ws, l.lvl_score), *out, stream));
}

dartree_status dartree_build_tree_timed(const dartree_params* p, const dartree_inputs* in, void* ws, size_t ws_bytes,
                                        const dartree_tree* out, hipEvent_t* events, hipStream_t stream) {
  dartree_status v = validate(p);
  if (v != DARTREE_OK) return v;
  if ((v = check_inputs(in)) != DARTREE_OK) return v;
  if ((v = check_tree(out)) != DARTREE_OK) return v;
  Layout l;
  if ((v = check_ws(*p, ws, ws_bytes, &l)) != DARTREE_OK) return v;
  const Shape s = shape_of(*p);
  Timer tm;
  tm.ev = events;
  tm.st = stream;
  const uint64_t key = params_key(*p);
  for (int d = 1; d <= p->depth; ++d) {
    if ((v = expand(*p, *in, d, ws, l, s, stream, tm)) != DARTREE_OK) return v;
    order_set(ws, key, d);
  }
  const int ti = p->depth * DARTREE_KERNELS_PER_DEPTH;
  tm.mark(ti, 0);
  v = hip_status(launch_prune_emit(p->batch, level_shape(*p, s), p->budget, at<int32_t>(ws, l.lvl_tok),
                                   at<int32_t>(ws, l.lvl_par), at<float>(ws, l.lvl_score), *out, stream));
  tm.mark(ti, 1);
  return v;
}

dartree_status dartree_build_tree(const dartree_params* p, const dartree_inputs* in, void* ws, size_t ws_bytes,
                                  const dartree_tree* out, hipStream_t stream) {
  return dartree_build_tree_timed(p, in, ws, ws_bytes, out, nullptr, stream);
}

dartree_status dartree_export_supertree(const dartree_params* p, const void* ws, size_t ws_bytes,
                                        const dartree_supertree* dst, hipStream_t stream) {
  dartree_status v = validate(p);
  if (v != DARTREE_OK) return v;
  if (!dst) return DARTREE_ERR_INVALID_ARG;
  Layout l;
  if ((v = check_ws(*p, ws, ws_bytes, &l)) != DARTREE_OK) return v;
  if (order_depth(ws, params_key(*p)) < 1) return DARTREE_ERR_ORDER;
  const size_t L = p->depth, b = p->batch, W = p->width, k = p->branch;
  struct Item { void* to; size_t off; size_t bytes; } items[] = {
      {dst->tokens, l.lvl_tok, L * b * W * 4},   {dst->parents, l.lvl_par, L * b * W * 4},
      {dst->scores, l.lvl_score, L * b * W * 4}, {dst->lse, l.lse, L * b * W * 4},
      {dst->cand_logp, l.cand_logp, L * b * W * k * 4}, {dst->cand_ids, l.cand_ids, L * b * W * k * 4},
      {p->candidates > 0 ? dst->csets : nullptr, l.cset, b * L * size_t(p->candidates) * 4},
  };
  for (const Item& it : items)
    if (it.to && hipMemcpyAsync(it.to, at<char>(ws, it.off), it.bytes, hipMemcpyDeviceToDevice, stream) != hipSuccess)
      return DARTREE_ERR_HIP;
  return DARTREE_OK;
}

dartree_status dartree_export_states(const dartree_params* p, const void* ws, size_t ws_bytes, int32_t d, void* dst,
                                     hipStream_t stream) {
  dartree_status v = validate(p);
  if (v != DARTREE_OK) return v;
  if (!dst || d < 1 || d >= p->depth) return DARTREE_ERR_INVALID_ARG;
  Layout l;
  if ((v = check_ws(*p, ws, ws_bytes, &l)) != DARTREE_OK) return v;
  const int last = order_depth(ws, params_key(*p));
  if (last != d && last != d + 1) return DARTREE_ERR_ORDER;
  const Shape s = shape_of(*p);
  const size_t bytes = size_t(p->batch) * s.n[d] * p->hidden * act_bytes(p->precision);
  const void* src = at<char>(ws, d % 2 ? l.state1 : l.state0);
  return hip_status(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, stream));
}

dartree_status dartree_export_features(const dartree_params* p, const void* ws, size_t ws_bytes, int32_t d, void* dst,
                                       hipStream_t stream) {
  dartree_status v = validate(p);
  if (v != DARTREE_OK) return v;
  if (!dst || d < 1 || d > p->depth || p->candidates < 0) return DARTREE_ERR_INVALID_ARG;
  Layout l;
  if ((v = check_ws(*p, ws, ws_bytes, &l)) != DARTREE_OK) return v;
  if (order_depth(ws, params_key(*p)) != d) return DARTREE_ERR_ORDER;
  const Shape s = shape_of(*p);
  const size_t bytes = size_t(p->batch) * s.n[d - 1] * p->hidden * act_bytes(p->precision);
  return hip_status(hipMemcpyAsync(dst, at<char>(ws, l.a), bytes, hipMemcpyDeviceToDevice, stream));
}

dartree_status dartree_project_workspace_size(int32_t precision, int32_t rows, int32_t vocab, int32_t hidden,
                                              size_t* bytes) {
  if (!bytes) return DARTREE_ERR_INVALID_ARG;
  if (precision != DARTREE_FP32 && precision != DARTREE_BF16) return DARTREE_ERR_INVALID_ARG;
  if (rows < 1 || vocab < 1 || hidden < 1) return DARTREE_ERR_INVALID_ARG;
  *bytes = proj_split_bytes(precision, EPI_LOGITS, rows, vocab, hidden);
  return DARTREE_OK;
}

dartree_status dartree_project(int32_t precision, int32_t rows, int32_t vocab, int32_t hidden, int32_t rows_per_group,
                               const void* x, const void* U, const float* bias, int64_t bias_stride, float* z,
                               void* ws, size_t ws_bytes, hipStream_t stream) {
  if (precision != DARTREE_FP32 && precision != DARTREE_BF16) return DARTREE_ERR_INVALID_ARG;
  if (rows < 1 || vocab < 1 || hidden < 1 || rows_per_group < 1 || bias_stride < 0) return DARTREE_ERR_INVALID_ARG;
  if (!x || !U || !bias || !z || !aligned16(x) || !aligned16(U) || !aligned16(z)) return DARTREE_ERR_INVALID_ARG;
  if (precision == DARTREE_BF16 && hidden % 64 != 0) return DARTREE_ERR_UNSUPPORTED;
  const size_t need = proj_split_bytes(precision, EPI_LOGITS, rows, vocab, hidden);
  if (need > 0 && (!ws || (reinterpret_cast<uintptr_t>(ws) % kAlign) != 0 || ws_bytes < need))
    return DARTREE_ERR_WORKSPACE;
  ProjArgs a{};
  a.precision = precision;
  a.epilogue = EPI_LOGITS;
  a.M = rows;
  a.N = vocab;
  a.K = hidden;
  a.rows_per_group = rows_per_group;
  a.x = x;
  a.w = U;
  a.bias_f32 = bias;
  a.bias_stride = bias_stride;
  a.out = z;
  a.split = need > 0 ? static_cast<float*>(ws) : nullptr;
  return hip_status(launch_project(a, stream));
}

dartree_status dartree_lse_topk_workspace_size(int32_t rows, int32_t vocab, int32_t k, size_t* bytes) {
  if (!bytes || rows < 1 || vocab < 1 || k < 1 || k > vocab) return DARTREE_ERR_INVALID_ARG;
  if (k > DARTREE_MAX_BRANCH || vocab > DARTREE_MAX_VOCAB) return DARTREE_ERR_UNSUPPORTED;
  *bytes = lse_topk_scratch_bytes(rows, vocab, k);
  return DARTREE_OK;
}

dartree_status dartree_lse_topk(const float* z, int32_t rows, int32_t vocab, int32_t k, float temperature, float* lse,
                                float* cand_logp, int32_t* cand_ids, void* ws, size_t ws_bytes, hipStream_t stream) {
  size_t need = 0;
  dartree_status v = dartree_lse_topk_workspace_size(rows, vocab, k, &need);
  if (v != DARTREE_OK) return v;
  if (!isfinite(temperature) || temperature < 0.f) return DARTREE_ERR_INVALID_ARG;
  if (!z || !lse || !cand_logp || !cand_ids) return DARTREE_ERR_INVALID_ARG;
  if (need > 0 && (!ws || ws_bytes < need || !aligned16(ws))) return DARTREE_ERR_WORKSPACE;
  const float tau = temperature > 0.f ? temperature : 1.f;
  return hip_status(launch_lse_topk(z, rows, vocab, k, tau, lse, cand_logp, cand_ids, ws, true, stream));
}

dartree_status dartree_candidate_sets_workspace_size(int32_t rows, int32_t vocab, int32_t K, size_t* bytes) {
  if (!bytes || rows < 1 || vocab < 1 || K < 1 || K > vocab) return DARTREE_ERR_INVALID_ARG;
  if (vocab > DARTREE_MAX_VOCAB || K > DARTREE_MAX_CANDIDATES || !candidate_sets_supported(vocab, K))
    return DARTREE_ERR_UNSUPPORTED;
  *bytes = candidate_sets_scratch_bytes(rows, vocab, K);
  return DARTREE_OK;
}

dartree_status dartree_candidate_sets(const float* logits, int32_t rows, int32_t vocab, int32_t K, int32_t* ids,
                                      void* ws, size_t ws_bytes, hipStream_t stream) {
  size_t need = 0;
  dartree_status v = dartree_candidate_sets_workspace_size(rows, vocab, K, &need);
  if (v != DARTREE_OK) return v;
  if (!logits || !ids) return DARTREE_ERR_INVALID_ARG;
  if (!ws || ws_bytes < need || !aligned16(ws)) return DARTREE_ERR_WORKSPACE;
  return hip_status(launch_candidate_sets(logits, rows, vocab, K, ids, ws, stream));
}

dartree_status dartree_select_topw(int32_t batch, int32_t n_parent, int32_t k, int32_t n_keep, float depth_bonus,
                                   const float* parent_score, const float* cand_logp, const int32_t* cand_ids,
                                   int32_t* out_tokens, int32_t* out_parents, float* out_scores, hipStream_t stream) {
  if (batch < 1 || n_parent < 1 || k < 1 || n_keep < 1) return DARTREE_ERR_INVALID_ARG;
  if (int64_t(n_parent) * k > DARTREE_MAX_SORT) return DARTREE_ERR_UNSUPPORTED;
  if (n_keep > n_parent * k) return DARTREE_ERR_INVALID_ARG;
  if (!isfinite(depth_bonus) || depth_bonus > 0.f) return DARTREE_ERR_INVALID_ARG;
  if (!cand_logp || !cand_ids || !out_tokens || !out_parents || !out_scores) return DARTREE_ERR_INVALID_ARG;
  LevelArgs la{};
  la.batch = batch;
  la.n_parent = n_parent;
  la.k = k;
  la.n_keep = n_keep;
  la.beta = depth_bonus;
  la.tau = 1.f;
  la.parent_stride = n_parent;
  la.out_stride = n_keep;
  la.parent_score = parent_score;
  la.nseg = 1;
  la.cand_logp = const_cast<float*>(cand_logp);      // read only when nseg == 1
  la.cand_ids = const_cast<int32_t*>(cand_ids);
  la.out_tok = out_tokens;
  la.out_par = out_parents;
  la.out_score = out_scores;
  la.state = 0;
  return hip_status(launch_select_level(la, stream));
}

dartree_status dartree_prune_levels(const dartree_params* p, const int32_t* tokens, const int32_t* parents,
                                    const float* scores, const dartree_tree* out, hipStream_t stream) {
  dartree_status v = validate(p);
  if (v != DARTREE_OK) return v;
  if ((v = check_tree(out)) != DARTREE_OK) return v;
  if (!tokens || !parents || !scores) return DARTREE_ERR_INVALID_ARG;
  const Shape s = shape_of(*p);
  return hip_status(
      launch_prune_emit(p->batch, level_shape(*p, s), p->budget, tokens, parents, scores, *out, stream));
}

// ---------------------------------------------------------------------------
// The consumer of the emitted tree
// ---------------------------------------------------------------------------
dartree_status dartree_accept_walk(int32_t batch, int32_t budget, int32_t max_len, const int32_t* tokens,
                                   const int32_t* parents, const int32_t* num_nodes, const int32_t* target,
                                   int32_t* accepted, int32_t* num_accepted, int32_t* bonus, hipStream_t stream) {
  if (batch < 1 || budget < 1 || max_len < 1) return DARTREE_ERR_INVALID_ARG;
  if (budget > DARTREE_MAX_SORT) return DARTREE_ERR_UNSUPPORTED;
  if (!tokens || !parents || !num_nodes || !target || !accepted || !num_accepted || !bonus)
    return DARTREE_ERR_INVALID_ARG;
  return hip_status(launch_accept_walk(batch, budget, max_len, tokens, parents, num_nodes, target, accepted,
                                       num_accepted, bonus, stream));
}

namespace {
dartree_status check_attn(const dartree_attn_params* p) {
  if (!p) return DARTREE_ERR_INVALID_ARG;
  if (p->batch < 1 || p->budget < 1 || p->max_ctx < 0 || p->heads_q < 1 || p->heads_kv < 1 || p->head_dim < 1)
    return DARTREE_ERR_INVALID_ARG;
  if (p->heads_q % p->heads_kv != 0 || !isfinite(p->scale) || p->scale <= 0.f) return DARTREE_ERR_INVALID_ARG;
  if (p->head_dim != 128 || p->budget > DARTREE_MAX_SORT) return DARTREE_ERR_UNSUPPORTED;
  if (int64_t(p->batch) * p->budget * p->heads_q > (int64_t(1) << 30)) return DARTREE_ERR_UNSUPPORTED;
  const int64_t segs = (int64_t(p->max_ctx) + attention_segment_len() - 1) / attention_segment_len() + 1;
  if (segs > attention_max_segments()) return DARTREE_ERR_UNSUPPORTED;
  return DARTREE_OK;
}

struct AttnLayout {
  int nseg_ctx, rows_pad;
  size_t part_o, part_ml, total;
};

AttnLayout attn_layout_of(const dartree_attn_params& p) {
  AttnLayout l{};
  const int seg = attention_segment_len();
  l.nseg_ctx = (p.max_ctx + seg - 1) / seg;
  const int rows = p.budget * (p.heads_q / p.heads_kv);
  l.rows_pad = (rows + 63) / 64 * 64;
  const bool fused = attention_fused(p.batch, p.budget, p.heads_q, p.heads_kv);
  const size_t slots = fused ? 0 : size_t(l.nseg_ctx + 1) * p.batch * p.heads_kv * l.rows_pad;
  size_t o = 0;
  auto take = [&](size_t bytes) { const size_t at = o; o = align_up(o + bytes); return at; };
  l.part_o = take(slots * 128 * 4);
  l.part_ml = take(slots * 2 * 4);
  l.total = o;
  return l;
}
}  // namespace

dartree_status dartree_tree_attention_workspace_size(const dartree_attn_params* p, size_t* bytes) {
  if (!bytes) return DARTREE_ERR_INVALID_ARG;
  const dartree_status v = check_attn(p);
  if (v != DARTREE_OK) return v;
  *bytes = attn_layout_of(*p).total;
  return DARTREE_OK;
}

dartree_status dartree_tree_attention(const dartree_attn_params* p, const void* q, const void* k_ctx,
                                      const void* v_ctx, const void* k_tree, const void* v_tree,
                                      const uint64_t* mask, const int32_t* ctx_len, float* out, void* ws,
                                      size_t ws_bytes, hipStream_t stream) {
  dartree_status v = check_attn(p);
  if (v != DARTREE_OK) return v;
  if (!q || !k_tree || !v_tree || !mask || !out) return DARTREE_ERR_INVALID_ARG;
  if (p->max_ctx > 0 && (!k_ctx || !v_ctx)) return DARTREE_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k_tree) || !aligned16(v_tree) || (k_ctx && !aligned16(k_ctx)) ||
      (v_ctx && !aligned16(v_ctx)) || !aligned16(out))
    return DARTREE_ERR_INVALID_ARG;
  const AttnLayout l = attn_layout_of(*p);
  if (l.total > 0 && (!ws || (reinterpret_cast<uintptr_t>(ws) % kAlign) != 0 || ws_bytes < l.total))
    return DARTREE_ERR_WORKSPACE;
  AttnArgs a{};
  a.batch = p->batch;
  a.budget = p->budget;
  a.max_ctx = p->max_ctx;
  a.heads_q = p->heads_q;
  a.heads_kv = p->heads_kv;
  a.group = p->heads_q / p->heads_kv;
  a.nseg_ctx = l.nseg_ctx;
  a.seg_len = attention_segment_len();
  a.rows_pad = l.rows_pad;
  a.scale_log2 = p->scale * 1.4426950408889634f;
  a.q = static_cast<const uint16_t*>(q);
  a.k_ctx = static_cast<const uint16_t*>(k_ctx);
  a.v_ctx = static_cast<const uint16_t*>(v_ctx);
  a.k_tree = static_cast<const uint16_t*>(k_tree);
  a.v_tree = static_cast<const uint16_t*>(v_tree);
  a.mask = mask;
  a.ctx_len = ctx_len;
  a.part_o = l.total > 0 ? at<float>(ws, l.part_o) : nullptr;
  a.part_ml = l.total > 0 ? at<float>(ws, l.part_ml) : nullptr;
  a.out = out;
  return hip_status(launch_tree_attention(a, stream));
}

dartree_status dartree_heap_workspace_size(const dartree_params* p, size_t* bytes) {
  if (!bytes) return DARTREE_ERR_INVALID_ARG;
  const dartree_status v = validate_heap(p);
  if (v != DARTREE_OK) return v;
  *bytes = heap_layout_of(*p).total;
  return DARTREE_OK;
}

dartree_status dartree_build_tree_heap(const dartree_params* p, const dartree_inputs* in, void* ws, size_t ws_bytes,
                                       const dartree_tree* out, hipStream_t stream) {
  dartree_status v = validate_heap(p);
  if (v != DARTREE_OK) return v;
  if ((v = check_inputs(in)) != DARTREE_OK) return v;
  if ((v = check_tree(out)) != DARTREE_OK) return v;
  HeapLayout l;
  if ((v = check_heap_ws(*p, ws, ws_bytes, &l)) != DARTREE_OK) return v;
  return build_heap(*p, *in, ws, l, *out, stream);
}

dartree_status dartree_export_heap(const dartree_params* p, const void* ws, size_t ws_bytes,
                                   const dartree_heap_trace* dst, hipStream_t stream) {
  dartree_status v = validate_heap(p);
  if (v != DARTREE_OK) return v;
  if (!dst) return DARTREE_ERR_INVALID_ARG;
  HeapLayout l;
  if ((v = check_heap_ws(*p, ws, ws_bytes, &l)) != DARTREE_OK) return v;
  const size_t L = p->depth, b = p->batch, B = p->budget, k = p->branch, h = p->hidden;
  const size_t S = b * (B + 1);
  struct Item { void* to; size_t off; size_t bytes; } items[] = {
      {dst->tokens, l.slot_tok, S * 4},      {dst->parents, l.slot_par, S * 4},
      {dst->depths, l.slot_depth, S * 4},    {dst->scores, l.slot_score, S * 4},
      {dst->num_popped, l.n_pop, b * 4},     {dst->lse, l.ch_lse, B * b * 4},
      {dst->cand_logp, l.ch_lp, B * b * k * 4}, {dst->cand_ids, l.ch_tok, B * b * k * 4},
      {dst->states, l.r_store, (B + 1) * b * h * act_bytes(p->precision)},
      {dst->features, l.a, B * b * h * act_bytes(p->precision)},
      {p->candidates > 0 ? dst->csets : nullptr, l.cset, b * L * size_t(p->candidates) * 4},
  };
  for (const Item& it : items)
    if (it.to && hipMemcpyAsync(it.to, at<char>(ws, it.off), it.bytes, hipMemcpyDeviceToDevice, stream) != hipSuccess)
      return DARTREE_ERR_HIP;
  return DARTREE_OK;
}

}  // extern "C"
