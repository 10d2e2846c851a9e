// Host side of the C ABI: argument validation, workspace planning, and the
// launch sequence of one forward (everything is enqueued on the caller's
// stream, with the correction chains of large batches forked onto an
// auxiliary stream and joined back; the host never waits on the device).
//
// Launch sequence for a tree with L correction levels (a flat LorExperts
// layer is L = 1, the dense comparator L = 0):
//   bucketing              unique (token, node) rows per level, slot flags,
//                          tile tables (one kernel for <= 64 tokens, else
//                          prepare / hist / scan / place)
//   per level l >= 1       z = X[rows_l] * [B_gate; B_up]^T, dgu = z * [A_gate; A_up]^T
//   level 0 gate|up GEMM   X[rows0] * [G_a; U_a]^T, once per (token, anchor)
//   swiglu_reduce          h = w * silu(g) * u per distinct expert, sums per row
//   level 0 down GEMM      hbar0 * D_a^T, once per (token, anchor)
//   per level l >= 1       v = hbar_l * B_down^T, y_l = v * A_down^T
//   combine                out[t] = sum of the token's rows over all levels
#include <algorithm>
#include <atomic>
#include <cmath>
#include <deque>
#include <map>
#include <limits>
#include <mutex>
#include <string>
#include <vector>

#include "lx_internal.h"

namespace lx {
namespace {

thread_local std::string g_err;

lx_status fail(lx_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

// ------------------------------------------------------------ kernel timing
struct ProfRec {
  const char* name;
  hipEvent_t a, b;
};
bool g_prof = false;
std::vector<ProfRec> g_pending;
std::vector<hipEvent_t> g_pool;
std::vector<std::pair<const char*, std::pair<int64_t, double>>> g_tot;

hipEvent_t pool_get() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Set for the duration of a call that must not create any HIP object (the
// static-scratch forward): kernel timing records are skipped in it.
thread_local bool tl_no_alloc = false;

struct Timed {
  const char* name;
  hipStream_t s;
  hipEvent_t a = nullptr, b = nullptr;
  Timed(const char* n, hipStream_t st) : name(n), s(st) {
    if (g_prof && !tl_no_alloc) {
      a = pool_get();
      b = pool_get();
      if (a) (void)hipEventRecord(a, s);
    }
  }
  void done() {
    if (g_prof && !tl_no_alloc && a && b) {
      (void)hipEventRecord(b, s);
      g_pending.push_back({name, a, b});
    }
  }
};

// Launches go to `lstream` (the caller's stream, or the auxiliary stream
// while an independent correction chain is being enqueued).
#define LX_LAUNCH(NAME, CALL)                                                          \
  do {                                                                                 \
    Timed _t(NAME, lstream);                                                           \
    hipError_t _e = (CALL);                                                            \
    _t.done();                                                                         \
    if (_e != hipSuccess)                                                              \
      return fail(LX_ERR_HIP, std::string(NAME) + ": " + hipGetErrorString(_e));       \
  } while (0)

// --------------------------------------------------------------- planning
size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

// Rank of a level's fp16 factor copies (padded to a multiple of 64 where the
// copies were made that way) and the bf16 input factors the fp16 path reads.
int rank16(const lx_level& v) { return v.rank_f16 > 0 ? v.rank_f16 : v.rank; }
const void* b_gate16(const lx_level& v) { return rank16(v) > v.rank ? v.b_gate_pad : v.b_gate; }
const void* b_up16(const lx_level& v) { return rank16(v) > v.rank ? v.b_up_pad : v.b_up; }

struct LevelPlan {
  int N = 0, rank = 0, nfac = 0;
  int bm[kNumTab] = {};
  int64_t rows_max = 0, tiles_max[kNumTab] = {};
  size_t hist, offsets, row_token, slot_row, slot_flags, fac;
  size_t tiles[kNumTab], n_tiles[kNumTab];
  size_t gu, z, hbar, v, y;
  // fp16 correction products: row exponents of z, v and the level's
  // activation sums (stored value = true value * 2^exp)
  size_t z_exp = 0, v_exp = 0, hbar_exp = 0;
  size_t part, cnt;   // split-K partial tiles and counters (skinny levels)
  int64_t n_cnt;
};

struct Plan {
  int T, k, E, L, d, f, NT;
  LevelPlan lv[kMaxLvl];
  size_t flags, anc, slot_wsum, total;
  // merged: a tree (L >= 2) whose correction levels all run on the
  // large-tile kernel with ranks that are multiples of 64 computes the gate|up
  // and down corrections of every level as one product over the leaf rows
  // (K concatenated over the levels), so the intermediate levels' full-width
  // outputs are never written; path_work marks the experts whose path has a
  // factor, leaf_row maps leaf rows to intermediate-level rows
  bool merged = false;
  size_t path_work = 0;
  size_t leaf_row[kMaxLvl] = {};
  // kernel choice per level (shapes only): "fast" levels keep every
  // GEMM-feeding intermediate as a bf16 (hi, lo) pair and run on the
  // large-tile or skinny kernel; "skinny" ones (few rows per node) on the
  // skinny kernel; batch: every level with GEMM work is skinny (the
  // independent products of a phase share a launch).
  bool fast[kMaxLvl] = {}, skinny[kMaxLvl] = {};
  bool batch = false;
  // lo8: the anchor activation sums are bf16 hi + block-scaled fp8 lo and the
  // anchor down GEMM runs the lo half on the fp8 MFMA (needs the layer's fp8
  // copy of the anchor down weights and the large-tile kernel)
  bool lo8 = false;
  // f16: the anchor activation sums are fp16 rows with a power-of-two scale
  // per token and the anchor down GEMM runs once, in fp16, against the
  // layer's fp16 copy (needs the large-tile kernel and whole rows per
  // SwiGLU workgroup); preferred over lo8
  bool f16 = false;
  size_t hbar_exp = 0;
  // cf16: on top of f16, every correction product runs once in fp16 against
  // the levels' fp16 factor copies: z = B x and v = B_down hbar are fp16 with
  // one power-of-two scale per 256-row tile (a tile spans whole rows: 2 rank
  // <= 256), the correction levels' activation sums fp16 rows as the anchor's
  bool cf16 = false;
  // dmerge: a merged two-level tree on the fp16 path runs both levels'
  // down-in products as one GEMM over the leaf rows, output [v1 | v2] per
  // leaf row (level 1's v buffer, one row exponent for both)
  bool dmerge = false;
};

int level_nodes(const lx_tree_layer& t, int l) { return l == 0 ? t.n_anchors : t.levels[l - 1].n_nodes; }

Plan make_plan(const lx_tree_layer& t, int T, int k) {
  Plan p{};
  p.T = T;
  p.k = k;
  p.E = t.E;
  p.L = t.n_levels;
  p.d = t.d;
  p.f = t.f;
  p.NT = (T + kTokTile - 1) / kTokTile;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + std::max<size_t>(bytes, 16));
    return o;
  };
  {
    const int64_t two31 = (int64_t)1 << 31;
    const int64_t rows0 = (int64_t)T * std::min(k, t.n_anchors);
    p.fast[0] = t.dtype == LX_BF16 && p.d % 64 == 0 && p.f % 64 == 0 && (int64_t)T * p.d < two31 &&
                rows0 * 2 * p.f < two31;
    for (int l = 1; l <= p.L; ++l) {
      const int r = t.levels[l - 1].rank;
      const int64_t R = (int64_t)T * std::min(k, t.levels[l - 1].n_nodes);
      // rank multiple of 32: the (hi | lo) operands of K = 2r are whole 64-wide
      // K-slabs (a slab may cross from the hi to the lo half; the large-tile
      // kernel then takes its weight columns modulo r)
      p.fast[l] = p.fast[0] && r % 32 == 0 && R * 2 * p.f < two31 && R * 4 * r < two31;
    }
    // Fast levels with few rows per node (decode-sized batches) stream their
    // weights through the skinny kernel; the large tiles would spend their
    // time on MFMA work over padding rows.
    p.batch = true;
    for (int l = 0; l <= p.L; ++l) {
      const int N = level_nodes(t, l);
      const int64_t R = (int64_t)T * std::min(k, N);
      // (the skinny kernel's hi and lo halves share whole weight slabs: rank
      // a multiple of 64)
      p.skinny[l] = p.fast[l] && R / std::max(N, 1) <= 64 && (l == 0 || t.levels[l - 1].rank % 64 == 0);
      const bool work = l == 0 || t.levels[l - 1].n_factors > 0;
      if (work && !p.skinny[l]) p.batch = false;
    }
    p.lo8 = t.anchor_down_f8 && t.anchor_down_f8_scale && p.fast[0] && !p.skinny[0] && p.f % 64 == 0;
    {
      bool all_fast = true;
      for (int l = 0; l <= p.L; ++l) all_fast &= p.fast[l];
      // (the fast SwiGLU kernel: k <= 8, at most two correction levels,
      // 512+ tokens give f / 4 threads per token, one workgroup per row)
      p.f16 = t.anchor_down_f16 && t.anchor_down_f16_exp && p.fast[0] && !p.skinny[0] && all_fast && k <= 8 &&
              p.L <= 2 && T >= 512 && p.f % 256 == 0 && p.f <= 1024;
      if (p.f16) p.lo8 = false;
      p.cf16 = p.f16;
      for (int l = 1; l <= p.L && p.cf16; ++l) {
        const lx_level& v = t.levels[l - 1];
        if (v.n_factors == 0) continue;
        p.cf16 = v.a_gate_f16 && v.a_up_f16 && v.a_down_f16 && v.b_down_f16 && rank16(v) % 64 == 0 &&
                 2 * rank16(v) <= 256 && !p.skinny[l];
      }
    }
    // (batches of at most 64 tokens always run their fast levels on the
    // skinny kernel, so merged trees take the four-pass bucketing)
    p.merged = p.L >= 2 && T > kTokTile && p.f % 256 == 0 && p.d % 256 == 0;
    for (int l = 1; l <= p.L && p.merged; ++l)
      p.merged = p.fast[l] && !p.skinny[l] && t.levels[l - 1].rank % 64 == 0;
    p.dmerge = p.cf16 && p.merged && p.L == 2 && t.levels[0].n_factors > 0 && t.levels[1].n_factors > 0 &&
               rank16(t.levels[0]) + rank16(t.levels[1]) <= 256;
  }
  p.flags = take(16);  // first: lx_read_device_status reads offset 0
  p.anc = take((size_t)(p.L + 1) * p.E * 4);
  const size_t tk = (size_t)T * k;
  p.slot_wsum = take(tk * 4);
  if (p.f16) p.hbar_exp = take((size_t)T * std::min(k, t.n_anchors) * 4);
  if (p.merged) {
    p.path_work = take((size_t)p.E);
    const size_t rl = (size_t)T * std::min(k, t.E);  // leaf rows, at most
    for (int l = 1; l < p.L; ++l) p.leaf_row[l] = take(rl * 4);
  }
  for (int l = 0; l <= p.L; ++l) {
    LevelPlan& q = p.lv[l];
    q.N = level_nodes(t, l);
    q.rank = l == 0 ? 0 : t.levels[l - 1].rank;
    q.nfac = l == 0 ? q.N : t.levels[l - 1].n_factors;
    q.bm[kTabSmall] = gemm_bm(t.dtype);
    q.bm[kTabBig] = kBigBM;
    q.bm[kTabSkinny] = kSkinnyBM;
    q.rows_max = (int64_t)T * std::min(k, q.N);
    // tiles = sum over touched nodes of ceil(rows / bm) <= floor(rows / bm) +
    // touched nodes, and at most min(N, rows) nodes are touched
    for (int b = 0; b < kNumTab; ++b) q.tiles_max[b] = q.rows_max / q.bm[b] + std::min<int64_t>(q.N, q.rows_max);
    q.hist = take((size_t)q.N * p.NT * 4);
    q.offsets = take((size_t)(q.N + 1) * 4);
    q.row_token = take((size_t)q.rows_max * 4);
    q.slot_row = take(tk * 4);
    q.slot_flags = take(tk);
    for (int b = 0; b < kNumTab; ++b) {
      q.tiles[b] = take((size_t)q.tiles_max[b] * sizeof(TileEntry));
      q.n_tiles[b] = take(4);
    }
    q.fac = take((size_t)q.N * 4);
    const size_t R = (size_t)q.rows_max;
    const bool work = l == 0 || q.nfac > 0;
    // merged trees: the intermediate levels' gate|up and down outputs are
    // folded into the leaf level's (which then exist even without leaf factors)
    const bool inter = p.merged && l > 0 && l < p.L;
    const bool leafm = p.merged && l == p.L;
    q.gu = take((work && !inter) || leafm ? R * 2 * p.f * 4 : 0);
    // z and v rows: bf16 (hi, lo) pairs of the rank, or fp16 at the copies' rank
    const size_t rf = l == 0 ? 0 : (size_t)rank16(t.levels[l - 1]);
    q.z = take(l > 0 && work ? R * std::max<size_t>(2 * (size_t)q.rank * 4, 2 * rf * 2) : 0);
    q.hbar = take((work && !inter) || leafm ? R * p.f * 4 : 0);
    // merged trees: an intermediate level's down-in product runs on the leaf
    // rows (by linearity, the sum over a row's leaf rows of B_down h_leaf is
    // B_down of the row's sum), so its v has one row per leaf row
    const size_t Rv = inter ? (size_t)T * std::min(k, t.E) : R;
    const size_t vrow = p.dmerge && l == 1 ? std::max<size_t>(q.rank * 4, (rf + rank16(t.levels[1])) * 2)
                                           : std::max<size_t>((size_t)q.rank * 4, rf * 2);
    q.v = take(l > 0 && work ? Rv * vrow : 0);
    q.y = take((work && !inter) || leafm ? R * p.d * 4 : 0);
    if (p.cf16 && l > 0) {
      q.z_exp = take(work ? R * 4 : 0);
      q.v_exp = take(work ? Rv * 4 : 0);
      q.hbar_exp = take((work && !inter) || leafm ? R * 4 : 0);
    }
    // one counter per work item of the level's widest skinny product
    const int widest = std::max(std::max(2 * p.f, p.d), 2 * q.rank);
    q.n_cnt = p.skinny[l] && work && T > 0 ? q.tiles_max[kTabSkinny] * ((widest + kSkinnyBN - 1) / kSkinnyBN) : 0;
    q.part = take(q.n_cnt ? (size_t)kSplitCap * kSkinnyBM * kSkinnyBN * 4 : 0);
    q.cnt = take((size_t)q.n_cnt * 4);
  }
  p.total = off;
  return p;
}

// -------------------------------------------------------------- validation
bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

lx_status check_layer(const lx_tree_layer* t) {
  if (!t) return fail(LX_ERR_INVALID_ARGUMENT, "layer is null");
  if (t->dtype != LX_F32 && t->dtype != LX_BF16) return fail(LX_ERR_INVALID_ARGUMENT, "bad dtype");
  if (t->E < 1 || t->d < 1 || t->f < 1 || t->n_anchors < 1)
    return fail(LX_ERR_INVALID_ARGUMENT, "E, d, f and n_anchors must be positive");
  if (t->n_levels < 0 || t->n_levels > LX_MAX_LEVELS)
    return fail(LX_ERR_INVALID_ARGUMENT, "n_levels out of range");
  if (t->E > LX_MAX_NODES || t->n_anchors > LX_MAX_NODES)
    return fail(LX_ERR_UNSUPPORTED, "more nodes than LX_MAX_NODES");
  if (t->d % 8 || t->f % 8) return fail(LX_ERR_UNSUPPORTED, "d and f must be multiples of 8");
  if ((int64_t)t->f * t->d > ((int64_t)1 << 31)) return fail(LX_ERR_UNSUPPORTED, "f*d too large");
  const int last = t->n_levels == 0 ? t->n_anchors : t->levels[t->n_levels - 1].n_nodes;
  if (last != t->E) return fail(LX_ERR_INVALID_ARGUMENT, "the last level must have E nodes");
  const void* aw[3] = {t->anchor_gate, t->anchor_up, t->anchor_down};
  for (const void* q : aw)
    if (!q || !aligned(q, 16)) return fail(LX_ERR_INVALID_ARGUMENT, "anchor weights null or not 16-byte aligned");
  if (t->anchor_down_f8 || t->anchor_down_f8_scale) {
    if (!t->anchor_down_f8 || !t->anchor_down_f8_scale || !aligned(t->anchor_down_f8, 16) ||
        !aligned(t->anchor_down_f8_scale, 4))
      return fail(LX_ERR_INVALID_ARGUMENT, "fp8 down copy and its scales: both or neither, 16/4-byte aligned");
    if (t->dtype != LX_BF16 || t->f % 64)
      return fail(LX_ERR_UNSUPPORTED, "an fp8 down copy needs a bf16 layer with f a multiple of 64");
  }
  if (t->anchor_down_f16 || t->anchor_down_f16_exp) {
    if (!t->anchor_down_f16 || !t->anchor_down_f16_exp || !aligned(t->anchor_down_f16, 16) ||
        !aligned(t->anchor_down_f16_exp, 4))
      return fail(LX_ERR_INVALID_ARGUMENT, "fp16 down copy and its exponents: both or neither, 16/4-byte aligned");
    if (t->dtype != LX_BF16) return fail(LX_ERR_UNSUPPORTED, "an fp16 down copy needs a bf16 layer");
  }
  for (int l = 0; l < t->n_levels; ++l) {
    const lx_level& v = t->levels[l];
    if (v.n_nodes < 1 || v.n_nodes > LX_MAX_NODES) return fail(LX_ERR_INVALID_ARGUMENT, "level node count out of range");
    if (v.n_factors < 0) return fail(LX_ERR_INVALID_ARGUMENT, "negative n_factors");
    if (!v.parent || !v.factor_of || !aligned(v.parent, 4) || !aligned(v.factor_of, 4))
      return fail(LX_ERR_INVALID_ARGUMENT, "level parent/factor_of null or misaligned");
    if (v.n_factors > 0) {
      if (v.rank < 1) return fail(LX_ERR_INVALID_ARGUMENT, "rank must be positive");
      if (t->dtype == LX_BF16 && v.rank % 8) return fail(LX_ERR_UNSUPPORTED, "bf16 ranks must be multiples of 8");
      const void* fw[6] = {v.a_gate, v.b_gate, v.a_up, v.b_up, v.a_down, v.b_down};
      for (const void* q : fw)
        if (!q || !aligned(q, 16)) return fail(LX_ERR_INVALID_ARGUMENT, "factor arrays null or not 16-byte aligned");
    }
    const void* cw[4] = {v.a_gate_f16, v.a_up_f16, v.a_down_f16, v.b_down_f16};
    const int32_t* ce[4] = {v.a_gate_f16_exp, v.a_up_f16_exp, v.a_down_f16_exp, v.b_down_f16_exp};
    int nset = 0;
    for (int i = 0; i < 4; ++i) {
      nset += (cw[i] != nullptr) + (ce[i] != nullptr);
      if ((cw[i] && !aligned(cw[i], 16)) || (ce[i] && !aligned(ce[i], 4)))
        return fail(LX_ERR_INVALID_ARGUMENT, "fp16 factor copies not 16-byte aligned or exponents not 4-byte aligned");
    }
    if (nset != 0 && nset != 8)
      return fail(LX_ERR_INVALID_ARGUMENT, "fp16 factor copies and their exponents: all eight or none");
    if (nset && t->dtype != LX_BF16) return fail(LX_ERR_UNSUPPORTED, "fp16 factor copies need a bf16 layer");
    if (v.rank_f16 != 0) {
      if (v.rank_f16 < v.rank || v.rank_f16 % 64 || v.rank_f16 > 128)
        return fail(LX_ERR_INVALID_ARGUMENT, "rank_f16 must be 0 or a multiple of 64 in [rank, 128]");
      if (!nset) return fail(LX_ERR_INVALID_ARGUMENT, "rank_f16 is set without fp16 factor copies");
    }
    if (rank16(v) > v.rank) {
      if (!v.b_gate_pad || !v.b_up_pad || !aligned(v.b_gate_pad, 16) || !aligned(v.b_up_pad, 16))
        return fail(LX_ERR_INVALID_ARGUMENT, "rank_f16 > rank needs b_gate_pad and b_up_pad, 16-byte aligned");
    }
  }
  return LX_OK;
}

lx_status check_call(const lx_tree_layer* t, int T, int k) {
  lx_status s = check_layer(t);
  if (s != LX_OK) return s;
  if (T < 0) return fail(LX_ERR_INVALID_ARGUMENT, "T must be >= 0");
  if (k < 1 || k > LX_MAX_K) return fail(LX_ERR_INVALID_ARGUMENT, "k must be in [1, LX_MAX_K]");
  if ((int64_t)T * k >= ((int64_t)1 << 31)) return fail(LX_ERR_UNSUPPORTED, "T*k too large");
  return LX_OK;
}

lx_tree_layer flat_to_tree(const lx_flat_layer& F) {
  lx_tree_layer t{};
  t.E = F.E;
  t.d = F.d;
  t.f = F.f;
  t.dtype = F.dtype;
  t.n_anchors = F.C;
  t.anchor_gate = F.dom_gate;
  t.anchor_up = F.dom_up;
  t.anchor_down = F.dom_down;
  t.anchor_down_f8 = F.dom_down_f8;
  t.anchor_down_f8_scale = F.dom_down_f8_scale;
  t.anchor_down_f16 = F.dom_down_f16;
  t.anchor_down_f16_exp = F.dom_down_f16_exp;
  t.n_levels = 1;
  lx_level& v = t.levels[0];
  v.n_nodes = F.E;
  v.rank = F.r;
  v.n_factors = F.M;
  v.parent = F.cluster_of;
  v.factor_of = F.factor_of;
  v.a_gate = F.a_gate;
  v.b_gate = F.b_gate;
  v.a_up = F.a_up;
  v.b_up = F.b_up;
  v.a_down = F.a_down;
  v.b_down = F.b_down;
  v.a_gate_f16 = F.a_gate_f16;
  v.a_gate_f16_exp = F.a_gate_f16_exp;
  v.a_up_f16 = F.a_up_f16;
  v.a_up_f16_exp = F.a_up_f16_exp;
  v.a_down_f16 = F.a_down_f16;
  v.a_down_f16_exp = F.a_down_f16_exp;
  v.b_down_f16 = F.b_down_f16;
  v.b_down_f16_exp = F.b_down_f16_exp;
  v.rank_f16 = F.r_f16;
  v.b_gate_pad = F.b_gate_pad;
  v.b_up_pad = F.b_up_pad;
  return t;
}

lx_tree_layer dense_to_tree(const lx_dense_layer& D) {
  lx_tree_layer t{};
  t.E = D.E;
  t.d = D.d;
  t.f = D.f;
  t.dtype = D.dtype;
  t.n_anchors = D.E;
  t.anchor_gate = D.w_gate;
  t.anchor_up = D.w_up;
  t.anchor_down = D.w_down;
  t.anchor_down_f8 = D.w_down_f8;
  t.anchor_down_f8_scale = D.w_down_f8_scale;
  t.anchor_down_f16 = D.w_down_f16;
  t.anchor_down_f16_exp = D.w_down_f16_exp;
  t.n_levels = 0;
  return t;
}

const char* kLowIn[kMaxLvl] = {"", "lowrank_gate_up_in_l1", "lowrank_gate_up_in_l2", "lowrank_gate_up_in_l3",
                               "lowrank_gate_up_in_l4"};
const char* kLowOut[kMaxLvl] = {"", "lowrank_gate_up_out_l1", "lowrank_gate_up_out_l2",
                                "lowrank_gate_up_out_l3", "lowrank_gate_up_out_l4"};
const char* kDownIn[kMaxLvl] = {"", "lowrank_down_in_l1", "lowrank_down_in_l2", "lowrank_down_in_l3",
                                "lowrank_down_in_l4"};
const char* kDownOut[kMaxLvl] = {"", "lowrank_down_out_l1", "lowrank_down_out_l2", "lowrank_down_out_l3",
                                 "lowrank_down_out_l4"};

// ------------------------------------------------------- auxiliary stream
// The correction-level GEMM chains do not depend on the anchor GEMMs, so
// they are enqueued on a second stream of the same device (default
// priority) between an event fork and join on the caller's stream; the
// hardware then fills compute units left idle by one chain with the other
// (the tail of the persistent anchor GEMM; decode-sized batches, where both
// chains stream weights). The mutex serialises the fork/join event use of
// concurrent callers on one device.
struct Aux {
  std::mutex mu;
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  bool ok = false;
};

// lx_set_aux_stream: whether prefill-sized forwards may use the auxiliary
// stream at all (process-wide; off by default: the persistent GEMMs of the
// two chains contend for the compute units rather than overlap).
std::atomic<int> g_aux_enabled{0};

Aux* aux_for_current_device() {
  static std::mutex mu;
  static Aux aux[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lk(mu);
  Aux& a = aux[dev];
  if (!a.ok && !a.s) {
    if (hipStreamCreateWithFlags(&a.s, hipStreamNonBlocking) != hipSuccess ||
        hipEventCreateWithFlags(&a.fork, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&a.join, hipEventDisableTiming) != hipSuccess)
      return nullptr;
    a.ok = true;
  }
  return a.ok ? &a : nullptr;
}

// Fork/join of the auxiliary stream around one independent chain. The
// destructor joins an open fork, so an early error return still leaves the
// caller's stream ordered after everything that was enqueued.
struct ForkJoin {
  Aux* aux;
  hipStream_t main;
  bool open = false;
  ForkJoin(Aux* a, hipStream_t m) : aux(a), main(m) {}
  hipError_t fork() {
    if (!aux) return hipSuccess;
    hipError_t e = hipEventRecord(aux->fork, main);
    if (e == hipSuccess) e = hipStreamWaitEvent(aux->s, aux->fork, 0);
    open = e == hipSuccess;
    return e;
  }
  hipError_t join() {
    if (!aux || !open) return hipSuccess;
    open = false;
    hipError_t e = hipEventRecord(aux->join, aux->s);
    if (e == hipSuccess) e = hipStreamWaitEvent(main, aux->join, 0);
    return e;
  }
  ~ForkJoin() { (void)join(); }
};

// Stable C string for a launch name built at run time (batched launches).
const char* intern_name(const std::string& n) {
  static std::mutex mu;
  static std::deque<std::string> names;
  std::lock_guard<std::mutex> lk(mu);
  for (const std::string& s : names)
    if (s == n) return s.c_str();
  names.push_back(n);
  return names.back().c_str();
}

enum Stop { RUN_ALL, RUN_BUCKET };

// The whole forward (or just the bucketing) of a validated tree.
// route: the router's logits, when its top-k is fused into the bucketing
// (ids and w are then outputs, written by the first bucketing kernel).
lx_status run(const lx_tree_layer& t, int T, int k, const void* x, const int32_t* ids, const float* w,
              void* out, lx_dtype out_dtype, void* ws, size_t ws_bytes, hipStream_t stream, Stop stop,
              Plan* plan_out = nullptr, const RouteIn* route = nullptr) {
  lx_status st = check_call(&t, T, k);
  if (st != LX_OK) return st;
  if (stop == RUN_ALL && out_dtype != LX_F32 && out_dtype != LX_BF16)
    return fail(LX_ERR_INVALID_ARGUMENT, "bad out_dtype");
  if (T > 0) {
    if (!ids || !aligned(ids, 4)) return fail(LX_ERR_INVALID_ARGUMENT, "topk_ids null or misaligned");
    if (stop == RUN_ALL) {
      if (!x || !aligned(x, 16)) return fail(LX_ERR_INVALID_ARGUMENT, "x null or not 16-byte aligned");
      if (!w || !aligned(w, 4)) return fail(LX_ERR_INVALID_ARGUMENT, "topk_weights null or misaligned");
      if (!out || !aligned(out, 16)) return fail(LX_ERR_INVALID_ARGUMENT, "out null or not 16-byte aligned");
    }
  }
  const Plan P = make_plan(t, T, k);
  if (plan_out) *plan_out = P;
  if (!ws || !aligned(ws, 16)) return fail(LX_ERR_INVALID_ARGUMENT, "workspace null or not 16-byte aligned");
  if (ws_bytes < P.total) return fail(LX_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than required");
  char* W = (char*)ws;
  const int L = P.L, E = P.E, d = P.d, f = P.f;
  hipStream_t lstream = stream;

  PrepareArgs pa{};
  pa.E = E;
  pa.L = L;
  pa.anc = (int32_t*)(W + P.anc);
  pa.flags = (uint32_t*)(W + P.flags);
  pa.path_work = P.merged ? (uint8_t*)(W + P.path_work) : nullptr;
  for (int l = 0; l <= L; ++l) {
    pa.n_nodes[l] = P.lv[l].N;
    if (l > 0) {
      pa.n_factors[l] = t.levels[l - 1].n_factors;
      pa.parent[l] = t.levels[l - 1].parent;
      pa.factor_of[l] = t.levels[l - 1].factor_of;
      pa.fac[l] = (int32_t*)(W + P.lv[l].fac);
    }
  }
  if (T == 0) {  // nothing to route: the status word is still reset
    LX_LAUNCH("bucket_prepare", launch_prepare(pa, lstream));
    return LX_OK;
  }

  const lx_dtype dt = t.dtype;
  const bool* const fast = P.fast;
  const bool* const skinny = P.skinny;

  BucketArgs ba{};
  ba.T = T;
  ba.k = k;
  ba.E = E;
  ba.L = L;
  ba.n_tok_tiles = P.NT;
  ba.ids = ids;
  ba.w = w;
  ba.slot_wsum = (float*)(W + P.slot_wsum);
  ba.anc = pa.anc;
  ba.flags = pa.flags;
  if (route) ba.route = *route;
  for (int l = 0; l <= L; ++l) {
    const LevelPlan& q = P.lv[l];
    BucketLevel& b = ba.lv[l];
    b.n_nodes = q.N;
    for (int i = 0; i < kNumTab; ++i) b.tile_bm[i] = q.bm[i];
    // skinny levels use only the skinny table; others the register-staged
    // (also 128-row large-tile) and 256-row tables
    b.tab_mask = skinny[l] ? 1u << kTabSkinny : (1u << kTabSmall) | (1u << kTabBig);
    b.work_all = l == 0;
    b.work_node = P.merged && l == L ? pa.path_work : nullptr;
    b.fac = l > 0 ? (const int32_t*)(W + q.fac) : nullptr;
    b.hist = (int32_t*)(W + q.hist);
    b.offsets = (int32_t*)(W + q.offsets);
    b.row_token = (int32_t*)(W + q.row_token);
    b.slot_row = (int32_t*)(W + q.slot_row);
    b.slot_flags = (uint8_t*)(W + q.slot_flags);
    for (int i = 0; i < kNumTab; ++i) {
      b.tiles[i] = (TileEntry*)(W + q.tiles[i]);
      b.n_tiles[i] = (int32_t*)(W + q.n_tiles[i]);
    }
    b.split_cnt = (uint32_t*)(W + q.cnt);
    b.n_split_cnt = (int32_t)q.n_cnt;
  }
  if (bucket_small_ok(ba) && !P.merged) {
    if (route) {
      // batches of at most 64 tokens: the single-workgroup bucketing would
      // run every token's top-k on one compute unit, slower than the
      // router's own kernel with one wavefront per token
      LX_LAUNCH("router_topk", launch_topk(route->logits, route->part, route->S, T, E, k,
                                           const_cast<int32_t*>(ids), const_cast<float*>(w), lstream));
      ba.route = RouteIn{};
    }
    LX_LAUNCH("bucket_small", launch_bucket_small(pa, ba, lstream));
  } else {
    LX_LAUNCH("bucket_prepare", launch_prepare(pa, lstream));
    if (route)
      LX_LAUNCH("router_topk+bucket_hist", launch_bucket_hist_route(ba, lstream));
    else
      LX_LAUNCH("bucket_hist", launch_bucket_hist(ba, lstream));
    LX_LAUNCH("bucket_scan", launch_bucket_scan(ba, lstream));
    LX_LAUNCH("bucket_place", launch_bucket_place(ba, lstream));
  }
  if (stop == RUN_BUCKET) return LX_OK;
  if (P.merged) {
    LeafMapArgs lm{};
    lm.T = T;
    lm.k = k;
    lm.L = L;
    for (int l = 0; l <= L; ++l) {
      lm.slot_row[l] = ba.lv[l].slot_row;
      lm.slot_flags[l] = ba.lv[l].slot_flags;
      if (l >= 1 && l < L) lm.leaf_row_map[l] = (int32_t*)(W + P.leaf_row[l]);
    }
    LX_LAUNCH("leaf_maps", launch_leaf_maps(lm, lstream));
  }

  // Decode-sized batches (every level with GEMM work on the skinny kernel):
  // the independent products of one phase share a launch.
  const bool batch_mode = P.batch;
  struct Pend {
    GemmArgs g;
    int ofmt;
    int tiles;
    const char* name;
  };
  Pend pend[kSkinnyMaxProblems];
  int npend = 0;
  auto flush = [&]() -> lx_status {
    if (npend == 0) return LX_OK;
    GemmArgs g[kSkinnyMaxProblems];
    int ofmt[kSkinnyMaxProblems];
    int tiles[kSkinnyMaxProblems];
    std::string name;
    const bool named = g_prof && !tl_no_alloc;  // the name only labels timing records
    for (int i = 0; i < npend; ++i) {
      g[i] = pend[i].g;
      ofmt[i] = pend[i].ofmt;
      tiles[i] = pend[i].tiles;
      if (named) name += (i ? "+" : "") + std::string(pend[i].name);
    }
    const int n = npend;
    npend = 0;
    LX_LAUNCH(named ? intern_name(name) : "skinny_batch", launch_gemm_skinny_batch(g, ofmt, tiles, n, lstream));
    return LX_OK;
  };
  auto big = [&](const char* name, GemmArgs g, int l, int bm, int bn, int ofmt,
                 int64_t a_rows_total) -> lx_status {
    const LevelPlan& q = P.lv[l];
    if (!g.B[1]) g.B[1] = g.B[0];
    if (skinny[l]) {
      if (!gemm_big_ok(g, kSkinnyBN, a_rows_total) || (g.Kb > 0 ? g.Kb : g.K) % 64)
        return fail(LX_ERR_UNSUPPORTED, std::string(name) + ": shape not supported by the skinny GEMM");
      g.tiles = ba.lv[l].tiles[kTabSkinny];
      g.n_tiles = ba.lv[l].n_tiles[kTabSkinny];
      if (q.n_cnt >= (int64_t)q.tiles_max[kTabSkinny] * ((g.ncols[0] + g.ncols[1] + kSkinnyBN - 1) / kSkinnyBN)) {
        g.part = (float*)(W + q.part);
        g.cnt = (uint32_t*)(W + q.cnt);
        g.split_cap = kSplitCap;
      }
      if (batch_mode) {
        if (npend == kSkinnyMaxProblems) {
          const lx_status st = flush();
          if (st != LX_OK) return st;
        }
        pend[npend++] = Pend{g, ofmt, (int)q.tiles_max[kTabSkinny], name};
        return LX_OK;
      }
      LX_LAUNCH(name, launch_gemm_skinny(g, ofmt, (int)q.tiles_max[kTabSkinny], lstream));
      return LX_OK;
    }
    if (!gemm_big_ok(g, bn, a_rows_total))
      return fail(LX_ERR_UNSUPPORTED, std::string(name) + ": shape not supported by the large-tile GEMM");
    const int tab = bm == kBigBM ? kTabBig : kTabSmall;
    if (q.bm[tab] != bm) return fail(LX_ERR_UNSUPPORTED, std::string(name) + ": no tile table for this height");
    g.tiles = ba.lv[l].tiles[tab];
    g.n_tiles = ba.lv[l].n_tiles[tab];
    LX_LAUNCH(name, launch_gemm_big(g, bm, bn, ofmt, (int)q.tiles_max[tab], lstream));
    return LX_OK;
  };
  // fp16 operands (A rows and weight matrices with power-of-two scales) on
  // the large-tile kernel, level l's 256-row tiles
  auto f16big = [&](const char* name, GemmArgs g, int l, int bn, int ofmt, int64_t a_rows_total) -> lx_status {
    if (!g.B[1]) g.B[1] = g.B[0];
    if (!gemm_f16_ok(g, bn, ofmt, a_rows_total))
      return fail(LX_ERR_UNSUPPORTED, std::string(name) + ": shape not supported by the fp16 GEMM");
    g.tiles = ba.lv[l].tiles[kTabBig];
    g.n_tiles = ba.lv[l].n_tiles[kTabBig];
    LX_LAUNCH(name, launch_gemm_f16(g, bn, ofmt, (int)P.lv[l].tiles_max[kTabBig], lstream));
    return LX_OK;
  };
  auto small = [&](const char* name, GemmArgs g, int l, AMode am) -> lx_status {
    g.tiles = ba.lv[l].tiles[kTabSmall];
    g.n_tiles = ba.lv[l].n_tiles[kTabSmall];
    LX_LAUNCH(name, launch_gemm(g, dt, am, (int)P.lv[l].tiles_max[kTabSmall], lstream));
    return LX_OK;
  };
#define LX_TRY(X)                  \
  do {                             \
    const lx_status s_ = (X);      \
    if (s_ != LX_OK) return s_;    \
  } while (0)

#define LX_HIP(X)                                                        \
  do {                                                                   \
    const hipError_t e_ = (X);                                           \
    if (e_ != hipSuccess) return fail(LX_ERR_HIP, hipGetErrorString(e_)); \
  } while (0)

  // The correction chains go to the auxiliary stream, concurrently with the
  // anchor GEMMs on the caller's stream, when the anchor level is large
  // enough to run on the persistent kernel (for decode-sized batches the
  // cross-stream event latency outweighs the overlap; those batch their
  // launches instead). Per-kernel timing runs serialised so that each
  // kernel's duration is its own.
  bool any_fac = false;
  for (int l = 1; l <= L; ++l) any_fac |= t.levels[l - 1].n_factors > 0;
  Aux* const aux = any_fac && !skinny[0] && !g_prof && !tl_no_alloc && g_aux_enabled.load(std::memory_order_relaxed)
                       ? aux_for_current_device()
                       : nullptr;
  std::unique_lock<std::mutex> aux_lock;
  if (aux) aux_lock = std::unique_lock<std::mutex>(aux->mu);
  ForkJoin fj_up(aux, stream), fj_down(aux, stream);
  hipStream_t const side = aux ? aux->s : stream;
  LX_HIP(fj_up.fork());

  // correction gate|up per level, part 1: z = B x (once per (token, node))
  lstream = side;
  for (int l = 1; l <= L; ++l) {
    const LevelPlan& q = P.lv[l];
    const lx_level& v = t.levels[l - 1];
    if (v.n_factors == 0) continue;
    const int r = v.rank;
    GemmArgs g{};
    g.A = x;
    g.lda = d;
    g.a_rows = ba.lv[l].row_token;
    g.B[0] = v.b_gate;
    g.B[1] = v.b_up;
    g.b_stride[0] = g.b_stride[1] = (int64_t)r * d;
    g.ncols[0] = g.ncols[1] = r;
    g.K = d;
    g.C = (float*)(W + q.z);
    if (fast[l] && P.cf16) {
      // [gate | up], fp16, one scale per tile, at the copies' rank (padded
      // factor rows give zero columns)
      const int rf = rank16(v);
      g.B[0] = b_gate16(v);
      g.B[1] = b_up16(v);
      g.b_stride[0] = g.b_stride[1] = (int64_t)rf * d;
      g.ncols[0] = g.ncols[1] = rf;
      g.ldc = 2 * (int64_t)rf;
      g.c_row_exp = (int32_t*)(W + q.z_exp);
      LX_TRY(big(kLowIn[l], g, l, kBigBM, 2 * rf <= 128 ? 128 : 256, OUT_F16T, T));
    } else if (fast[l]) {
      g.ldc = 4 * (int64_t)r;  // [gate hi | gate lo | up hi | up lo], bf16
      LX_TRY(big(kLowIn[l], g, l, kBigBM, 2 * r <= 128 ? 128 : 256, OUT_HILO, T));
    } else {
      g.ldc = 2 * (int64_t)r;
      g.c_coloff[1] = r;
      LX_TRY(small(kLowIn[l], g, l, A_BF16));
    }
  }
  // anchor gate|up, once per (token, anchor)
  lstream = stream;
  {
    const LevelPlan& q = P.lv[0];
    GemmArgs g{};
    g.A = x;
    g.lda = d;
    g.a_rows = ba.lv[0].row_token;
    g.B[0] = t.anchor_gate;
    g.B[1] = t.anchor_up;
    g.b_stride[0] = g.b_stride[1] = (int64_t)f * d;
    g.ncols[0] = g.ncols[1] = f;
    g.K = d;
    g.C = (float*)(W + q.gu);
    g.ldc = 2 * (int64_t)f;
    g.c_coloff[1] = f;
    if (fast[0])
      LX_TRY(big("anchor_gate_up", g, 0, kBigBM, 256, OUT_X16, T));
    else
      LX_TRY(small("anchor_gate_up", g, 0, A_BF16));
  }
  LX_TRY(flush());
  // correction gate|up per level, part 2: dgu = A z (merged trees: one
  // product over the leaf rows, dgu_L = sum over levels of A_l z_l)
  lstream = side;
  auto seg_args = [&](bool down) {
    SegArgs sa{};
    sa.anc = pa.anc;
    sa.f16 = P.cf16 ? 1 : 0;
    for (int l = 1; l <= L; ++l) {
      const lx_level& v = t.levels[l - 1];
      if (v.n_factors == 0) continue;
      const LevelPlan& q = P.lv[l];
      // fp16: the copies' rank (padded columns of A and rows of B are zero)
      const int r = P.cf16 ? rank16(v) : v.rank;
      SegDesc& sd = sa.s[sa.nseg++];
      sd.rank = r;
      sd.anc_off = l == L ? -1 : l * E;
      sd.fac = l == L ? nullptr : (const int32_t*)(W + q.fac);
      if (!down) {
        sd.A = W + q.z;
        sd.lda = (P.cf16 ? 2 : 4) * (int64_t)r;  // [gate | up] fp16 or [gate hi | gate lo | up hi | up lo]
        sd.akoff1 = (P.cf16 ? 1 : 2) * r;
        sd.map = l == L ? nullptr : (const int32_t*)(W + P.leaf_row[l]);
        sd.zero_row = 0;
        sd.B[0] = P.cf16 ? v.a_gate_f16 : v.a_gate;
        sd.B[1] = P.cf16 ? v.a_up_f16 : v.a_up;
        sd.b_stride[0] = sd.b_stride[1] = (int64_t)f * r;
        sd.a_exp = P.cf16 ? (const int32_t*)(W + q.z_exp) : nullptr;
        sd.b_exp[0] = v.a_gate_f16_exp;
        sd.b_exp[1] = v.a_up_f16_exp;
      } else {
        sd.A = W + q.v;  // one row per leaf row at every level
        sd.lda = (P.cf16 ? 1 : 2) * (int64_t)r;  // fp16 or [hi | lo]
        sd.akoff1 = 0;
        sd.map = nullptr;
        sd.zero_row = 0;
        sd.B[0] = sd.B[1] = P.cf16 ? v.a_down_f16 : v.a_down;
        sd.b_stride[0] = sd.b_stride[1] = (int64_t)d * r;
        sd.a_exp = P.cf16 ? (const int32_t*)(W + q.v_exp) : nullptr;
        sd.b_exp[0] = sd.b_exp[1] = v.a_down_f16_exp;
        if (P.dmerge) {  // [v1 | v2] rows of level 1's buffer, one exponent per row
          const LevelPlan& q1 = P.lv[1];
          sd.A = W + q1.v;
          sd.lda = rank16(t.levels[0]) + rank16(t.levels[1]);
          sd.a_col0 = l == 1 ? 0 : rank16(t.levels[0]);
          sd.a_exp = (const int32_t*)(W + q1.v_exp);
        }
      }
    }
    return sa;
  };
  auto seg = [&](const char* name, bool down) -> lx_status {
    const LevelPlan& q = P.lv[L];
    const SegArgs sa = seg_args(down);
    GemmArgs g{};
    g.tiles = ba.lv[L].tiles[kTabBig];
    g.n_tiles = ba.lv[L].n_tiles[kTabBig];
    g.ncols[0] = down ? d : f;
    g.ncols[1] = down ? 0 : f;
    g.C = (float*)(W + (down ? q.y : q.gu));
    g.ldc = down ? d : 2 * (int64_t)f;
    if (!gemm_seg_ok(g, sa, q.rows_max))
      return fail(LX_ERR_UNSUPPORTED, std::string(name) + ": shape not supported by the merged GEMM");
    LX_LAUNCH(name, launch_gemm_seg(g, sa, (int)q.tiles_max[kTabBig], lstream));
    return LX_OK;
  };
  if (P.merged) LX_TRY(seg("lowrank_gate_up_out_merged", false));
  for (int l = 1; l <= L && !P.merged; ++l) {
    const LevelPlan& q = P.lv[l];
    const lx_level& v = t.levels[l - 1];
    if (v.n_factors == 0) continue;
    const int r = v.rank;
    GemmArgs h{};
    h.B[0] = v.a_gate;
    h.B[1] = v.a_up;
    h.b_stride[0] = h.b_stride[1] = (int64_t)f * r;
    h.ncols[0] = h.ncols[1] = f;
    h.A = W + q.z;
    h.C = (float*)(W + q.gu);
    h.ldc = 2 * (int64_t)f;
    h.c_coloff[1] = f;
    if (fast[l] && P.cf16) {
      const int rf = rank16(v);
      h.B[0] = v.a_gate_f16;
      h.B[1] = v.a_up_f16;
      h.b_stride[0] = h.b_stride[1] = (int64_t)f * rf;
      h.lda = 2 * (int64_t)rf;  // [gate | up] fp16
      h.a_koff[1] = rf;
      h.K = h.Kb = rf;
      h.a_row_exp = (const int32_t*)(W + q.z_exp);
      h.b_exp = v.a_gate_f16_exp;
      h.b_exp1 = v.a_up_f16_exp;
      LX_TRY(f16big(kLowOut[l], h, l, 256, OUT_X16, q.rows_max));
    } else if (fast[l]) {
      h.lda = 4 * (int64_t)r;
      h.a_koff[1] = 2 * r;
      h.K = 2 * r;
      h.Kb = r;
      // gate and up read different z columns: tiles must not straddle them
      LX_TRY(big(kLowOut[l], h, l, kBigBM, f % 256 == 0 ? 256 : f % 128 == 0 ? 128 : 64, OUT_X16, q.rows_max));
    } else {
      h.lda = 2 * (int64_t)r;
      h.a_koff[1] = r;
      h.K = r;
      LX_TRY(small(kLowOut[l], h, l, A_F32_HILO));
    }
  }
  LX_TRY(flush());
  lstream = stream;

  TokenArgs ta{};
  ta.T = T;
  ta.k = k;
  ta.E = E;
  ta.L = L;
  ta.d = d;
  ta.f = f;
  ta.slot_wsum = ba.slot_wsum;
  ta.gu0 = (const float*)(W + P.lv[0].gu);
  for (int l = 0; l <= L; ++l) {
    const LevelPlan& q = P.lv[l];
    ta.slot_row[l] = ba.lv[l].slot_row;
    ta.slot_flags[l] = ba.lv[l].slot_flags;
    ta.dgu[l] = (const float*)(W + q.gu);
    ta.hbar[l] = (float*)(W + q.hbar);
    const bool hf16 = l == 0 ? P.f16 : P.cf16;
    ta.hbar_mode[l] = hf16 ? HBAR_F16 : l == 0 && P.lo8 ? HBAR_LO8 : fast[l] ? HBAR_HILO : HBAR_F32;
    ta.hbar_exp[l] = !hf16 ? nullptr : l == 0 ? (int32_t*)(W + P.hbar_exp) : (int32_t*)(W + q.hbar_exp);
    ta.x16[l] = fast[l] ? 1 : 0;
    ta.y[l] = (const float*)(W + q.y);
  }
  ta.out = out;
  ta.out_dtype = out_dtype;
  ta.merged = P.merged ? 1 : 0;
  LX_HIP(fj_up.join());
  LX_LAUNCH("swiglu_reduce", launch_swiglu_reduce(ta, lstream));
  LX_HIP(fj_down.fork());

  // anchor down, once per (token, anchor), on the weighted activation sums.
  // With the merged down-in of a two-level tree on the same stream, both fp16
  // products share one persistent launch (below).
  const bool pair_down = P.f16 && P.dmerge && side == stream;
  GemmArgs g_anchor_down{};
  {
    const LevelPlan& q = P.lv[0];
    GemmArgs g{};
    g.A = W + q.hbar;
    g.B[0] = t.anchor_down;
    g.b_stride[0] = (int64_t)d * f;
    g.ncols[0] = d;
    g.C = (float*)(W + q.y);
    g.ldc = d;
    if (P.f16) {
      // row = fp16 [f] scaled by 2^hbar_exp[row]
      g.lda = f;
      g.K = f;
      g.Kb = f;
      g.B[0] = g.B[1] = t.anchor_down_f16;
      g.a_row_exp = (const int32_t*)(W + P.hbar_exp);
      g.b_exp = t.anchor_down_f16_exp;
      g.tiles = ba.lv[0].tiles[kTabBig];
      g.n_tiles = ba.lv[0].n_tiles[kTabBig];
      if (!gemm_f16_ok(g, 256, OUT_X16, q.rows_max))
        return fail(LX_ERR_UNSUPPORTED, "anchor_down: shape not supported by the fp16 GEMM");
      if (pair_down)
        g_anchor_down = g;
      else
        LX_LAUNCH("anchor_down", launch_gemm_f16(g, 256, OUT_X16, (int)q.tiles_max[kTabBig], lstream));
    } else if (P.lo8) {
      // row = [bf16 hi (f) | fp8 lo (f bytes) | scale words (f / 64)] in 4f bytes
      g.lda = 2 * (int64_t)f;
      g.K = 2 * f;
      g.Kb = f;
      g.b8 = (const uint8_t*)t.anchor_down_f8;
      g.bsc = t.anchor_down_f8_scale;
      g.a_lo8_off = 2 * f;
      g.a_sc_off = 3 * f;
      g.B[1] = g.B[0];
      g.tiles = ba.lv[0].tiles[kTabBig];
      g.n_tiles = ba.lv[0].n_tiles[kTabBig];
      if (!gemm_lo8_ok(g, q.rows_max))
        return fail(LX_ERR_UNSUPPORTED, "anchor_down: shape not supported by the fp8-lo GEMM");
      LX_LAUNCH("anchor_down", launch_gemm_lo8(g, OUT_X16, (int)q.tiles_max[kTabBig], lstream));
    } else if (fast[0]) {
      g.lda = 2 * (int64_t)f;
      g.K = 2 * f;
      g.Kb = f;
      LX_TRY(big("anchor_down", g, 0, kBigBM, 256, OUT_X16, q.rows_max));
    } else {
      g.lda = f;
      g.K = f;
      LX_TRY(small("anchor_down", g, 0, A_F32_HILO));
    }
  }
  // correction down per level, part 1: v = B_down hbar (merged trees: over
  // the leaf rows at every level, each with its ancestor's weights)
  lstream = side;
  if (P.dmerge) {
    // both levels at once: part 0 the leaf's level-1 ancestor's B_down, part 1
    // the leaf's own
    const lx_level& v1 = t.levels[0];
    const lx_level& v2 = t.levels[1];
    const LevelPlan& qL = P.lv[L];
    GemmArgs g{};
    g.A = W + qL.hbar;
    g.lda = f;
    g.K = g.Kb = f;
    g.B[0] = v1.b_down_f16;
    g.B[1] = v2.b_down_f16;
    g.b_stride[0] = (int64_t)rank16(v1) * f;
    g.b_stride[1] = (int64_t)rank16(v2) * f;
    g.ncols[0] = rank16(v1);
    g.ncols[1] = rank16(v2);
    g.widx_anc = pa.anc + (size_t)1 * E;
    g.widx_fac = (const int32_t*)(W + P.lv[1].fac);
    g.widx_own1 = 1;
    g.a_row_exp = (const int32_t*)(W + qL.hbar_exp);
    g.b_exp = v1.b_down_f16_exp;
    g.b_exp1 = v2.b_down_f16_exp;
    g.C = (float*)(W + P.lv[1].v);
    g.ldc = rank16(v1) + rank16(v2);
    g.c_row_exp = (int32_t*)(W + P.lv[1].v_exp);
    if (pair_down) {
      g.tiles = ba.lv[L].tiles[kTabBig];
      g.n_tiles = ba.lv[L].n_tiles[kTabBig];
      if (!gemm_f16_ok(g, 256, OUT_F16T, qL.rows_max))
        return fail(LX_ERR_UNSUPPORTED, "lowrank_down_in_merged: shape not supported by the fp16 GEMM");
      LX_LAUNCH("anchor_down+lowrank_down_in_merged",
                launch_gemm_f16_pair(g_anchor_down, (int)P.lv[0].tiles_max[kTabBig], g, OUT_F16T,
                                     (int)qL.tiles_max[kTabBig], lstream));
    } else {
      LX_TRY(f16big("lowrank_down_in_merged", g, L, 256, OUT_F16T, qL.rows_max));
    }
  }
  for (int l = 1; l <= L && !P.dmerge; ++l) {
    const LevelPlan& q = P.lv[l];
    const lx_level& v = t.levels[l - 1];
    if (v.n_factors == 0) continue;
    const int r = v.rank;
    GemmArgs g{};
    g.A = W + q.hbar;
    g.B[0] = v.b_down;
    g.b_stride[0] = (int64_t)r * f;
    g.ncols[0] = r;
    g.C = (float*)(W + q.v);
    if (P.cf16) {
      // fp16 activation sums (row scales) against the fp16 copy; v fp16 with
      // one scale per tile (merged trees: over the leaf rows, as below)
      const int lt = P.merged ? L : l;
      const LevelPlan& qa = P.lv[lt];
      g.A = W + qa.hbar;
      if (P.merged && l < L) {
        g.widx_anc = pa.anc + (size_t)l * E;
        g.widx_fac = (const int32_t*)(W + q.fac);
      }
      const int rf = rank16(v);
      g.B[0] = v.b_down_f16;
      g.b_stride[0] = (int64_t)rf * f;
      g.ncols[0] = rf;
      g.lda = f;
      g.K = g.Kb = f;
      g.ldc = rf;
      g.a_row_exp = (const int32_t*)(W + qa.hbar_exp);
      g.b_exp = v.b_down_f16_exp;
      g.c_row_exp = (int32_t*)(W + q.v_exp);
      LX_TRY(f16big(kDownIn[l], g, lt, rf <= 64 ? 64 : 128, OUT_F16T, qa.rows_max));
      continue;
    }
    if (P.merged) {
      const LevelPlan& qL = P.lv[L];
      g.A = W + qL.hbar;
      if (l < L) {
        g.widx_anc = pa.anc + (size_t)l * E;
        g.widx_fac = (const int32_t*)(W + q.fac);
      }
      g.lda = 2 * (int64_t)f;
      g.K = 2 * f;
      g.Kb = f;
      g.ldc = 2 * (int64_t)r;
      LX_TRY(big(kDownIn[l], g, L, kBigBM, r <= 64 ? 64 : 128, OUT_HILO, qL.rows_max));
      continue;
    }
    if (fast[l]) {
      g.lda = 2 * (int64_t)f;
      g.K = 2 * f;
      g.Kb = f;
      g.ldc = 2 * (int64_t)r;  // [hi | lo], bf16
      LX_TRY(big(kDownIn[l], g, l, kBigBM, r <= 64 ? 64 : 128, OUT_HILO, q.rows_max));
    } else {
      g.lda = f;
      g.K = f;
      g.ldc = r;
      LX_TRY(small(kDownIn[l], g, l, A_F32_HILO));
    }
  }
  LX_TRY(flush());
  // correction down per level, part 2: y = A_down v (merged trees: one
  // product over the leaf rows; a level-l row's term rides on the leaf row of
  // its first slot)
  if (P.merged) LX_TRY(seg("lowrank_down_out_merged", true));
  for (int l = 1; l <= L && !P.merged; ++l) {
    const LevelPlan& q = P.lv[l];
    const lx_level& v = t.levels[l - 1];
    if (v.n_factors == 0) continue;
    const int r = v.rank;
    GemmArgs h{};
    h.A = W + q.v;
    h.B[0] = v.a_down;
    h.b_stride[0] = (int64_t)d * r;
    h.ncols[0] = d;
    h.C = (float*)(W + q.y);
    h.ldc = d;
    if (fast[l] && P.cf16) {
      const int rf = rank16(v);
      h.B[0] = v.a_down_f16;
      h.b_stride[0] = (int64_t)d * rf;
      h.lda = rf;
      h.K = h.Kb = rf;
      h.a_row_exp = (const int32_t*)(W + q.v_exp);
      h.b_exp = v.a_down_f16_exp;
      LX_TRY(f16big(kDownOut[l], h, l, 256, OUT_X16, q.rows_max));
    } else if (fast[l]) {
      h.lda = 2 * (int64_t)r;
      h.K = 2 * r;
      h.Kb = r;
      LX_TRY(big(kDownOut[l], h, l, kBigBM, 256, OUT_X16, q.rows_max));
    } else {
      h.lda = r;
      h.K = r;
      LX_TRY(small(kDownOut[l], h, l, A_F32_HILO));
    }
  }
  LX_TRY(flush());
#undef LX_TRY
  lstream = stream;
  LX_HIP(fj_down.join());
  LX_LAUNCH("combine", launch_combine(ta, lstream));
#undef LX_HIP
  return LX_OK;
}

lx_status check_flat(const lx_flat_layer* F) {
  if (!F) return fail(LX_ERR_INVALID_ARGUMENT, "layer is null");
  if (F->C < 1 || F->M < 0) return fail(LX_ERR_INVALID_ARGUMENT, "C must be positive and M non-negative");
  return LX_OK;
}

lx_status check_dense(const lx_dense_layer* D) {
  if (!D) return fail(LX_ERR_INVALID_ARGUMENT, "layer is null");
  return LX_OK;
}

}  // namespace
}  // namespace lx

using namespace lx;

// Device scratch of lx_moe_forward_tree_static: one copy per GPU, allocated
// when the code object is loaded there and held until the process ends. Host
// code never uses this name as an address (on the host it is only a
// stand-in): the device address comes from hipGetSymbolAddress, once per
// device, and only that address is passed to kernels.
static __device__ __align__(256) unsigned char scratch[LX_STATIC_SCRATCH_BYTES];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[64] = {};

// Device address of this device's `scratch` (looked up on the first call on
// the device, with that device current).
lx_status scratch_for_current_device(void** ptr) {
  int dev = 0;
  const hipError_t e0 = hipGetDevice(&dev);
  if (e0 != hipSuccess) return fail(LX_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e0));
  if (dev < 0 || dev >= 64) return fail(LX_ERR_UNSUPPORTED, "device index beyond 63");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(LX_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return LX_OK;
}
}  // namespace

extern "C" {

const char* lx_status_string(lx_status s) {
  switch (s) {
    case LX_OK: return "LX_OK";
    case LX_ERR_INVALID_ARGUMENT: return "LX_ERR_INVALID_ARGUMENT";
    case LX_ERR_UNSUPPORTED: return "LX_ERR_UNSUPPORTED";
    case LX_ERR_WORKSPACE_TOO_SMALL: return "LX_ERR_WORKSPACE_TOO_SMALL";
    case LX_ERR_HIP: return "LX_ERR_HIP";
  }
  return "LX_ERR_UNKNOWN";
}

const char* lx_last_error(void) { return g_err.c_str(); }

int32_t lx_version(void) { return 100; }

int32_t lx_set_aux_stream(int32_t enable) { return g_aux_enabled.exchange(enable ? 1 : 0); }

size_t lx_moe_tree_workspace_bytes(const lx_tree_layer* layer, int32_t T, int32_t k) {
  if (check_call(layer, T, k) != LX_OK) return 0;
  return make_plan(*layer, T, k).total;
}

size_t lx_moe_workspace_bytes(const lx_flat_layer* layer, int32_t T, int32_t k) {
  if (check_flat(layer) != LX_OK) return 0;
  const lx_tree_layer t = flat_to_tree(*layer);
  return lx_moe_tree_workspace_bytes(&t, T, k);
}

size_t lx_dense_moe_workspace_bytes(const lx_dense_layer* layer, int32_t T, int32_t k) {
  if (check_dense(layer) != LX_OK) return 0;
  const lx_tree_layer t = dense_to_tree(*layer);
  return lx_moe_tree_workspace_bytes(&t, T, k);
}

lx_status lx_moe_forward_tree(const lx_tree_layer* layer, int32_t T, int32_t k, const void* x,
                              const int32_t* topk_ids, const float* topk_weights, void* out,
                              lx_dtype out_dtype, void* workspace, size_t workspace_bytes, void* stream) {
  g_err.clear();
  if (!layer) return fail(LX_ERR_INVALID_ARGUMENT, "layer is null");
  return run(*layer, T, k, x, topk_ids, topk_weights, out, out_dtype, workspace, workspace_bytes,
             (hipStream_t)stream, RUN_ALL);
}

lx_status lx_moe_forward(const lx_flat_layer* layer, int32_t T, int32_t k, const void* x,
                         const int32_t* topk_ids, const float* topk_weights, void* out, lx_dtype out_dtype,
                         void* workspace, size_t workspace_bytes, void* stream) {
  g_err.clear();
  lx_status s = check_flat(layer);
  if (s != LX_OK) return s;
  const lx_tree_layer t = flat_to_tree(*layer);
  return run(t, T, k, x, topk_ids, topk_weights, out, out_dtype, workspace, workspace_bytes,
             (hipStream_t)stream, RUN_ALL);
}

lx_status lx_dense_moe_forward(const lx_dense_layer* layer, int32_t T, int32_t k, const void* x,
                               const int32_t* topk_ids, const float* topk_weights, void* out,
                               lx_dtype out_dtype, void* workspace, size_t workspace_bytes, void* stream) {
  g_err.clear();
  lx_status s = check_dense(layer);
  if (s != LX_OK) return s;
  const lx_tree_layer t = dense_to_tree(*layer);
  return run(t, T, k, x, topk_ids, topk_weights, out, out_dtype, workspace, workspace_bytes,
             (hipStream_t)stream, RUN_ALL);
}

lx_status lx_moe_forward_tree_static(const lx_tree_layer* layer, int32_t T, int32_t k, const void* x,
                                     const int32_t* topk_ids, const float* topk_weights, void* out,
                                     lx_dtype out_dtype, void* stream) {
  g_err.clear();
  if (!layer) return fail(LX_ERR_INVALID_ARGUMENT, "layer is null");
  lx_status st = check_call(layer, T, k);
  if (st != LX_OK) return st;
  const size_t need = make_plan(*layer, T, k).total;
  if (need > (size_t)LX_STATIC_SCRATCH_BYTES)
    return fail(LX_ERR_WORKSPACE_TOO_SMALL, "this batch needs " + std::to_string(need) +
                                                " bytes of scratch; the static scratch holds " +
                                                std::to_string((size_t)LX_STATIC_SCRATCH_BYTES) +
                                                " (use lx_moe_forward_tree with a workspace)");
  void* ws = nullptr;
  st = scratch_for_current_device(&ws);
  if (st != LX_OK) return st;
  tl_no_alloc = true;
  st = run(*layer, T, k, x, topk_ids, topk_weights, out, out_dtype, ws, (size_t)LX_STATIC_SCRATCH_BYTES,
           (hipStream_t)stream, RUN_ALL);
  tl_no_alloc = false;
  return st;
}

lx_status lx_bucket(const lx_tree_layer* layer, int32_t T, int32_t k, const int32_t* topk_ids, int32_t level,
                    int32_t* row_token, int32_t* node_offsets, int32_t* slot_row, void* workspace,
                    size_t workspace_bytes, void* stream) {
  g_err.clear();
  if (!layer) return fail(LX_ERR_INVALID_ARGUMENT, "layer is null");
  if (level < 0 || level > layer->n_levels) return fail(LX_ERR_INVALID_ARGUMENT, "level out of range");
  Plan P{};
  hipStream_t s = (hipStream_t)stream;
  lx_status st = run(*layer, T, k, nullptr, topk_ids, nullptr, nullptr, LX_F32, workspace, workspace_bytes, s,
                     RUN_BUCKET, &P);
  if (st != LX_OK) return st;
  const LevelPlan& q = P.lv[level];
  const char* W = (const char*)workspace;
  hipError_t e = hipSuccess;
  if (T == 0) {
    // no bucketing ran: the level has no rows
    if (node_offsets) e = hipMemsetAsync(node_offsets, 0, (size_t)(q.N + 1) * 4, s);
    if (e != hipSuccess) return fail(LX_ERR_HIP, hipGetErrorString(e));
    return LX_OK;
  }
  if (row_token && q.rows_max > 0)
    e = hipMemcpyAsync(row_token, W + q.row_token, (size_t)q.rows_max * 4, hipMemcpyDeviceToDevice, s);
  if (e == hipSuccess && node_offsets)
    e = hipMemcpyAsync(node_offsets, W + q.offsets, (size_t)(q.N + 1) * 4, hipMemcpyDeviceToDevice, s);
  if (e == hipSuccess && slot_row)
    e = hipMemcpyAsync(slot_row, W + q.slot_row, (size_t)T * k * 4, hipMemcpyDeviceToDevice, s);
  if (e != hipSuccess) return fail(LX_ERR_HIP, hipGetErrorString(e));
  return LX_OK;
}

lx_status lx_convert_f16(const void* w, int32_t n, int32_t rows, int32_t cols, void* w_f16, int32_t* exps,
                         void* stream) {
  g_err.clear();
  if (n < 1 || rows < 1 || cols < 1) return fail(LX_ERR_INVALID_ARGUMENT, "n, rows and cols must be positive");
  if (!w || !w_f16 || !exps || !aligned(w, 2) || !aligned(w_f16, 16) || !aligned(exps, 4))
    return fail(LX_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  const hipError_t e = launch_convert_f16(w, n, (int64_t)rows * cols, w_f16, exps, (hipStream_t)stream);
  if (e != hipSuccess) return fail(LX_ERR_HIP, std::string("lx_convert_f16: ") + hipGetErrorString(e));
  return LX_OK;
}

lx_status lx_convert_f16_padded(const void* w, int32_t n, int32_t rows, int32_t cols, int32_t rows_out,
                                int32_t cols_out, void* w_f16, int32_t* exps, void* stream) {
  g_err.clear();
  if (n < 1 || rows < 1 || cols < 1 || rows_out < rows || cols_out < cols)
    return fail(LX_ERR_INVALID_ARGUMENT, "n, rows, cols positive; rows_out >= rows, cols_out >= cols");
  if ((int64_t)rows_out * cols_out >= ((int64_t)1 << 31)) return fail(LX_ERR_UNSUPPORTED, "matrix too large");
  if (!w || !w_f16 || !exps || !aligned(w, 2) || !aligned(w_f16, 16) || !aligned(exps, 4))
    return fail(LX_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  const hipError_t e = launch_copy_pad(w, n, rows, cols, rows_out, cols_out, w_f16, exps, (hipStream_t)stream);
  if (e != hipSuccess) return fail(LX_ERR_HIP, std::string("lx_convert_f16_padded: ") + hipGetErrorString(e));
  return LX_OK;
}

lx_status lx_pad_bf16(const void* w, int32_t n, int32_t rows, int32_t cols, int32_t rows_out, int32_t cols_out,
                      void* w_out, void* stream) {
  g_err.clear();
  if (n < 1 || rows < 1 || cols < 1 || rows_out < rows || cols_out < cols)
    return fail(LX_ERR_INVALID_ARGUMENT, "n, rows, cols positive; rows_out >= rows, cols_out >= cols");
  if ((int64_t)rows_out * cols_out >= ((int64_t)1 << 31)) return fail(LX_ERR_UNSUPPORTED, "matrix too large");
  if (!w || !w_out || !aligned(w, 2) || !aligned(w_out, 16))
    return fail(LX_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  const hipError_t e = launch_copy_pad(w, n, rows, cols, rows_out, cols_out, w_out, nullptr, (hipStream_t)stream);
  if (e != hipSuccess) return fail(LX_ERR_HIP, std::string("lx_pad_bf16: ") + hipGetErrorString(e));
  return LX_OK;
}

lx_status lx_quantize_f8(const void* w, int32_t n, int32_t rows, int32_t cols, void* w_f8, uint32_t* scales,
                         void* stream) {
  g_err.clear();
  if (n < 0 || rows < 0 || cols < 0) return fail(LX_ERR_INVALID_ARGUMENT, "negative size");
  if (cols % 64) return fail(LX_ERR_UNSUPPORTED, "cols must be a multiple of 64");
  const int64_t n_rows = (int64_t)n * rows;
  if (n_rows == 0 || cols == 0) return LX_OK;
  if (!w || !w_f8 || !scales || !aligned(w, 16) || !aligned(w_f8, 16) || !aligned(scales, 4))
    return fail(LX_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  const hipError_t e = launch_quantize_f8(w, n_rows, cols, (uint8_t*)w_f8, scales, (hipStream_t)stream);
  if (e != hipSuccess) return fail(LX_ERR_HIP, hipGetErrorString(e));
  return LX_OK;
}

namespace {
// Router plan: logits [T][E] fp32, then (split) the partial tiles.
struct RoutePlan {
  int items, s, S;  // work items, requested and made splits
  size_t logits, part, total;
};
RoutePlan route_plan(int T, int d, int E) {
  RoutePlan r{};
  r.items = (T + kSkinnyBM - 1) / kSkinnyBM * ((E + kSkinnyBN - 1) / kSkinnyBN);
  const int nkw = d / 64;
  r.s = std::min(kSplitCap / std::max(r.items, 1), nkw / kSplitMinSlabs);
  r.S = skinny_splits(nkw, r.s);
  r.logits = 0;
  r.part = align_up((size_t)T * E * 4);
  r.total = r.part + (r.S > 1 ? align_up((size_t)r.items * r.S * kSkinnyBM * kSkinnyBN * 4) : 0);
  return r;
}

lx_status check_route(lx_dtype dtype, int32_t T, int32_t d, int32_t E, int32_t k) {
  if (T < 0 || d < 0 || E < 0) return fail(LX_ERR_INVALID_ARGUMENT, "negative size");
  if (dtype != LX_BF16) return fail(LX_ERR_UNSUPPORTED, "the router takes bf16 activations and weights");
  if (d == 0 || d % 64) return fail(LX_ERR_UNSUPPORTED, "d must be a positive multiple of 64");
  if (E < 1 || E > kRouteMaxE || E % 4) return fail(LX_ERR_UNSUPPORTED, "E must be a multiple of 4 in 4 .. 512");
  if (k < 1 || k > E || k > LX_MAX_K) return fail(LX_ERR_INVALID_ARGUMENT, "k must be in 1 .. min(E, LX_MAX_K)");
  if ((int64_t)T * d >= ((int64_t)1 << 31)) return fail(LX_ERR_UNSUPPORTED, "T * d must be below 2^31");
  return LX_OK;
}
}  // namespace

size_t lx_route_workspace_bytes(int32_t T, int32_t d, int32_t E) {
  if (check_route(LX_BF16, T, d, E, 1) != LX_OK) return 0;
  return route_plan(T, d, E).total;
}

lx_status lx_route_topk(const void* x, const void* w_r, lx_dtype dtype, int32_t T, int32_t d, int32_t E,
                        int32_t k, int32_t* topk_ids, float* topk_weights, void* workspace,
                        size_t workspace_bytes, void* stream) {
  g_err.clear();
  const lx_status st = check_route(dtype, T, d, E, k);
  if (st != LX_OK) return st;
  if (T == 0) return LX_OK;
  if (!x || !w_r || !topk_ids || !topk_weights || !workspace || !aligned(x, 16) || !aligned(w_r, 16) ||
      !aligned(topk_ids, 4) || !aligned(topk_weights, 4) || !aligned(workspace, 256))
    return fail(LX_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  const RoutePlan P = route_plan(T, d, E);
  if (workspace_bytes < P.total) return fail(LX_ERR_WORKSPACE_TOO_SMALL, "workspace too small");
  hipStream_t s = (hipStream_t)stream;
  uint8_t* const W = (uint8_t*)workspace;
  // logits = x W_r^T on the skinny kernel over implicit 32-row tiles
  GemmArgs g{};
  g.A = x;
  g.lda = d;
  g.B[0] = g.B[1] = w_r;
  g.ncols[0] = E;
  g.K = d;
  g.C = (float*)(W + P.logits);
  g.ldc = E;
  g.dense_rows = T;
  if (P.S > 1) {
    g.part = (float*)(W + P.part);
    g.split_force = P.s;
    g.defer = 1;
  }
  if (!gemm_big_ok(g, kSkinnyBN, T)) return fail(LX_ERR_UNSUPPORTED, "router shape not supported");
  hipStream_t lstream = s;
  LX_LAUNCH("router_logits", launch_gemm_skinny(g, OUT_F32, (T + kSkinnyBM - 1) / kSkinnyBM, lstream));
  LX_LAUNCH("router_topk", launch_topk((const float*)(W + P.logits), (const float*)(W + P.part), P.S, T, E, k,
                                       topk_ids, topk_weights, lstream));
  return LX_OK;
}

size_t lx_route_moe_tree_workspace_bytes(const lx_tree_layer* layer, int32_t T, int32_t k) {
  if (check_call(layer, T, k) != LX_OK) return 0;
  if (check_route(layer->dtype, T, layer->d, layer->E, k) != LX_OK) return 0;
  return align_up(make_plan(*layer, T, k).total) + route_plan(T, layer->d, layer->E).total;
}

lx_status lx_route_moe_forward_tree(const lx_tree_layer* layer, int32_t T, int32_t k, const void* x, const void* w_r,
                                    int32_t* topk_ids, float* topk_weights, void* out, lx_dtype out_dtype,
                                    void* workspace, size_t workspace_bytes, void* stream) {
  g_err.clear();
  if (!layer) return fail(LX_ERR_INVALID_ARGUMENT, "layer is null");
  lx_status st = check_call(layer, T, k);
  if (st != LX_OK) return st;
  st = check_route(layer->dtype, T, layer->d, layer->E, k);
  if (st != LX_OK) return st;
  if (T == 0) return run(*layer, 0, k, x, topk_ids, topk_weights, out, out_dtype, workspace, workspace_bytes,
                         (hipStream_t)stream, RUN_ALL);
  if (!x || !w_r || !topk_ids || !topk_weights || !workspace || !aligned(x, 16) || !aligned(w_r, 16) ||
      !aligned(topk_ids, 4) || !aligned(topk_weights, 4) || !aligned(workspace, 256))
    return fail(LX_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  const size_t fwd = align_up(make_plan(*layer, T, k).total);
  const RoutePlan R = route_plan(T, layer->d, layer->E);
  if (workspace_bytes < fwd + R.total) return fail(LX_ERR_WORKSPACE_TOO_SMALL, "workspace too small");
  uint8_t* const W = (uint8_t*)workspace + fwd;
  // logits = x W_r^T on the skinny kernel over implicit 32-row tiles, as in
  // lx_route_topk; their top-k runs inside the first bucketing kernel
  GemmArgs g{};
  g.A = x;
  g.lda = layer->d;
  g.B[0] = g.B[1] = w_r;
  g.ncols[0] = layer->E;
  g.K = layer->d;
  g.C = (float*)(W + R.logits);
  g.ldc = layer->E;
  g.dense_rows = T;
  RouteIn ri{};
  ri.logits = g.C;
  ri.S = R.S;
  if (R.S > 1) {
    g.part = (float*)(W + R.part);
    g.split_force = R.s;
    g.defer = 1;
    ri.part = g.part;
  }
  if (!gemm_big_ok(g, kSkinnyBN, T)) return fail(LX_ERR_UNSUPPORTED, "router shape not supported");
  hipStream_t lstream = (hipStream_t)stream;
  LX_LAUNCH("router_logits", launch_gemm_skinny(g, OUT_F32, (T + kSkinnyBM - 1) / kSkinnyBM, lstream));
  return run(*layer, T, k, x, topk_ids, topk_weights, out, out_dtype, workspace, fwd, lstream, RUN_ALL, nullptr,
             &ri);
}

lx_status lx_coact_distance(const int32_t* topk_ids, int32_t N, int32_t k, int32_t E, uint32_t* fire,
                            uint32_t* pair, double* dist, void* stream) {
  g_err.clear();
  if (N < 0 || k < 1 || k > LX_MAX_K) return fail(LX_ERR_INVALID_ARGUMENT, "need N >= 0 and 1 <= k <= LX_MAX_K");
  if (E < 1 || E > kClusterMaxE) return fail(LX_ERR_UNSUPPORTED, "E must be in 1 .. 1024");
  if ((N > 0 && (!topk_ids || !aligned(topk_ids, 4))) || !fire || !pair || !dist || !aligned(fire, 4) ||
      !aligned(pair, 4) || !aligned(dist, 8))
    return fail(LX_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  hipStream_t lstream = (hipStream_t)stream;
  LX_LAUNCH("coact_distance", launch_coact(topk_ids, N, k, E, fire, pair, dist, lstream));
  return LX_OK;
}

lx_status lx_kmedoids(const double* dist, const uint32_t* fire, int32_t E, int32_t C, const int32_t* protected_ids,
                      int32_t n_protected, int32_t max_iter, int32_t* cluster_of, int32_t* factor_of,
                      int32_t* dominant, int32_t* iterations, void* stream) {
  g_err.clear();
  if (E < 1 || E > kClusterMaxE) return fail(LX_ERR_UNSUPPORTED, "E must be in 1 .. 1024");
  if (n_protected < 0 || n_protected > E || (n_protected > 0 && !protected_ids) || max_iter < 0)
    return fail(LX_ERR_INVALID_ARGUMENT, "bad protection list or max_iter");
  if (C - n_protected < 1 || C - n_protected > E - n_protected)
    return fail(LX_ERR_INVALID_ARGUMENT, "need 1 <= C - n_protected <= E - n_protected");
  ProtMask pm{};
  for (int i = 0; i < n_protected; ++i) {
    const int p = protected_ids[i];
    if (p < 0 || p >= E) return fail(LX_ERR_INVALID_ARGUMENT, "protected expert id out of range");
    if ((pm.bits[p >> 5] >> (p & 31)) & 1u) return fail(LX_ERR_INVALID_ARGUMENT, "repeated protected expert id");
    pm.bits[p >> 5] |= 1u << (p & 31);
  }
  if (!dist || !fire || !cluster_of || !factor_of || !dominant || !iterations || !aligned(dist, 8) ||
      !aligned(fire, 4) || !aligned(cluster_of, 4) || !aligned(factor_of, 4) || !aligned(dominant, 4) ||
      !aligned(iterations, 4))
    return fail(LX_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  hipStream_t lstream = (hipStream_t)stream;
  LX_LAUNCH("kmedoids", launch_kmedoids(dist, fire, E, C, pm, n_protected, max_iter, cluster_of, factor_of, dominant,
                                        iterations, lstream));
  return LX_OK;
}

size_t lx_align_workspace_bytes(int32_t f, int32_t d) {
  if (f < 1 || d < 1) return 0;
  return (size_t)2 * f * (3 * (size_t)d + 1) * sizeof(double);
}

lx_status lx_align_cost(const void* dom_gate, const void* dom_up, const void* dom_down, const void* mem_gate,
                        const void* mem_up, const void* mem_down, lx_dtype dtype, int32_t f, int32_t d, double* cost,
                        void* workspace, size_t workspace_bytes, void* stream) {
  g_err.clear();
  if (dtype != LX_BF16 && dtype != LX_F32) return fail(LX_ERR_INVALID_ARGUMENT, "bad dtype");
  if (f < 1 || d < 1) return fail(LX_ERR_INVALID_ARGUMENT, "f and d must be positive");
  if ((int64_t)f * 3 * d >= ((int64_t)1 << 31)) return fail(LX_ERR_UNSUPPORTED, "f * 3d must be below 2^31");
  const size_t es = dtype == LX_BF16 ? 2 : 4;
  const void* w[6] = {dom_gate, dom_up, dom_down, mem_gate, mem_up, mem_down};
  for (const void* q : w)
    if (!q || !aligned(q, es)) return fail(LX_ERR_INVALID_ARGUMENT, "null or misaligned weight pointer");
  if (!cost || !aligned(cost, 8) || !workspace || !aligned(workspace, 256))
    return fail(LX_ERR_INVALID_ARGUMENT, "null or misaligned cost or workspace");
  if (workspace_bytes < lx_align_workspace_bytes(f, d)) return fail(LX_ERR_WORKSPACE_TOO_SMALL, "workspace too small");
  hipStream_t lstream = (hipStream_t)stream;
  LX_LAUNCH("align_cost", launch_align_cost(dom_gate, dom_up, dom_down, mem_gate, mem_up, mem_down,
                                            dtype == LX_BF16, f, d, cost, (double*)workspace, lstream));
  return LX_OK;
}

lx_status lx_assign(const double* cost, int32_t n, int32_t* perm, double* total) {
  g_err.clear();
  if (n < 0 || (n > 0 && (!cost || !perm))) return fail(LX_ERR_INVALID_ARGUMENT, "bad arguments");
  // Shortest augmenting paths with dual potentials (the augmentation phase of
  // Jonker-Volgenant): rows are added one at a time; each is matched along a
  // shortest alternating path in reduced costs, found Dijkstra-style over the
  // columns, after which the potentials keep every reduced cost >= 0.
  const double inf = std::numeric_limits<double>::infinity();
  std::vector<double> u(n + 1, 0.0), v(n + 1, 0.0), minv(n + 1);
  std::vector<int> match(n + 1, 0), way(n + 1, 0);  // match[j]: row of column j (1-based, 0 = free)
  std::vector<char> used(n + 1);
  for (int i = 1; i <= n; ++i) {
    match[0] = i;
    int j0 = 0;
    std::fill(minv.begin(), minv.end(), inf);
    std::fill(used.begin(), used.end(), 0);
    do {
      used[j0] = 1;
      const int i0 = match[j0];
      double delta = inf;
      int j1 = 0;
      const double* const crow = cost + (size_t)(i0 - 1) * n;
      for (int j = 1; j <= n; ++j) {
        if (used[j]) continue;
        const double cur = crow[j - 1] - u[i0] - v[j];
        if (cur < minv[j]) {
          minv[j] = cur;
          way[j] = j0;
        }
        if (minv[j] < delta) {
          delta = minv[j];
          j1 = j;
        }
      }
      if (j1 == 0) return fail(LX_ERR_INVALID_ARGUMENT, "cost matrix has non-finite entries");
      for (int j = 0; j <= n; ++j) {
        if (used[j]) {
          u[match[j]] += delta;
          v[j] -= delta;
        } else {
          minv[j] -= delta;
        }
      }
      j0 = j1;
    } while (match[j0] != 0);
    do {  // flip the path
      const int j1 = way[j0];
      match[j0] = match[j1];
      j0 = j1;
    } while (j0 != 0);
  }
  double t = 0.0;
  for (int j = 1; j <= n; ++j) perm[match[j] - 1] = j - 1;
  for (int i = 0; i < n; ++i) t += cost[(size_t)i * n + perm[i]];
  if (total) *total = t;
  return LX_OK;
}

size_t lx_lowrank_workspace_bytes(int32_t rows, int32_t cols, int32_t r, int32_t p) {
  const int l = r + p;
  if (rows < 1 || cols < 1 || r < 1 || p < 0 || l > 128 || l > rows || l > cols) return 0;
  return lowrank_ws_doubles(rows, cols, l) * sizeof(double);
}

lx_status lx_lowrank_factors(const void* w_dom, const void* w_mem, lx_dtype dtype, int32_t rows, int32_t cols,
                             const int32_t* perm, int32_t perm_axis, int32_t r, int32_t p, int32_t q,
                             const double* omega, float* A, float* B, double* sigma, void* workspace,
                             size_t workspace_bytes, void* stream) {
  g_err.clear();
  if (dtype != LX_BF16 && dtype != LX_F32) return fail(LX_ERR_INVALID_ARGUMENT, "bad dtype");
  if (rows < 1 || cols < 1 || r < 1 || p < 0 || q < 0 || q > 16 || (perm_axis != 0 && perm_axis != 1))
    return fail(LX_ERR_INVALID_ARGUMENT, "bad sizes, q or perm_axis");
  const int l = r + p;
  if (l > 128 || l > rows || l > cols) return fail(LX_ERR_UNSUPPORTED, "r + p must be at most 128, rows and cols");
  if ((int64_t)rows * cols >= ((int64_t)1 << 31)) return fail(LX_ERR_UNSUPPORTED, "rows * cols must be below 2^31");
  const size_t es = dtype == LX_BF16 ? 2 : 4;
  if (!w_dom || !w_mem || !aligned(w_dom, es) || !aligned(w_mem, es) || !omega || !aligned(omega, 8) || !A ||
      !aligned(A, 4) || !B || !aligned(B, 4) || !sigma || !aligned(sigma, 8) || (perm && !aligned(perm, 4)) ||
      !workspace || !aligned(workspace, 256))
    return fail(LX_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  if (workspace_bytes < lx_lowrank_workspace_bytes(rows, cols, r, p))
    return fail(LX_ERR_WORKSPACE_TOO_SMALL, "workspace too small");
  hipStream_t lstream = (hipStream_t)stream;
  LX_LAUNCH("lowrank_factors", launch_lowrank(w_dom, w_mem, dtype == LX_BF16, rows, cols, perm, perm_axis, r, l, q,
                                              omega, A, B, sigma, (double*)workspace, lstream));
  return LX_OK;
}

size_t lx_weighted_workspace_bytes(int32_t rows, int32_t cols, int32_t n, int32_t damped, int32_t r, int32_t p) {
  const int l = r + p;
  const int64_t np = (int64_t)n + (damped ? cols : 0);
  if (rows < 1 || cols < 1 || n < 0 || r < 1 || p < 0 || l > 128 || l > rows || l > cols || np < l) return 0;
  if ((int64_t)rows * cols >= ((int64_t)1 << 31) || np * cols >= ((int64_t)1 << 31)) return 0;
  return weighted_ws_doubles(rows, cols, (int)np, l) * sizeof(double);
}

lx_status lx_weighted_factors(const void* w_dom, const void* w_mem, lx_dtype dtype, int32_t rows, int32_t cols,
                              const int32_t* perm, int32_t perm_axis, const void* x, lx_dtype x_dtype, int32_t n,
                              double damp, int32_t r, int32_t p, int32_t q, const double* omega, float* A, float* B,
                              double* sigma, void* workspace, size_t workspace_bytes, void* stream) {
  g_err.clear();
  if ((dtype != LX_BF16 && dtype != LX_F32) || (x_dtype != LX_BF16 && x_dtype != LX_F32))
    return fail(LX_ERR_INVALID_ARGUMENT, "bad dtype");
  if (rows < 1 || cols < 1 || n < 0 || r < 1 || p < 0 || q < 0 || q > 16 || (perm_axis != 0 && perm_axis != 1) ||
      !(damp >= 0.0) || !std::isfinite(damp))
    return fail(LX_ERR_INVALID_ARGUMENT, "bad sizes, damp, q or perm_axis");
  const int l = r + p;
  const int64_t np = (int64_t)n + (damp > 0.0 ? cols : 0);
  if (l > 128 || l > rows || l > cols || np < l)
    return fail(LX_ERR_UNSUPPORTED, "r + p must be at most 128, rows, cols and the activation rows");
  if ((int64_t)rows * cols >= ((int64_t)1 << 31) || np * cols >= ((int64_t)1 << 31))
    return fail(LX_ERR_UNSUPPORTED, "rows * cols and activation rows * cols must be below 2^31");
  const size_t es = dtype == LX_BF16 ? 2 : 4, xs = x_dtype == LX_BF16 ? 2 : 4;
  if (!w_dom || !w_mem || !aligned(w_dom, es) || !aligned(w_mem, es) || (n > 0 && (!x || !aligned(x, xs))) ||
      !omega || !aligned(omega, 8) || !A || !aligned(A, 4) || !B || !aligned(B, 4) || !sigma || !aligned(sigma, 8) ||
      (perm && !aligned(perm, 4)) || !workspace || !aligned(workspace, 256))
    return fail(LX_ERR_INVALID_ARGUMENT, "null or misaligned pointer");
  if (workspace_bytes < lx_weighted_workspace_bytes(rows, cols, n, damp > 0.0 ? 1 : 0, r, p))
    return fail(LX_ERR_WORKSPACE_TOO_SMALL, "workspace too small");
  hipStream_t lstream = (hipStream_t)stream;
  LX_LAUNCH("weighted_factors", launch_weighted(w_dom, w_mem, dtype == LX_BF16, rows, cols, perm, perm_axis, x,
                                                x_dtype == LX_BF16, n, damp, r, l, q, omega, A, B, sigma,
                                                (double*)workspace, lstream));
  return LX_OK;
}

lx_status lx_read_device_status(const void* workspace, void* stream, uint32_t* flags) {
  g_err.clear();
  if (!workspace || !flags) return fail(LX_ERR_INVALID_ARGUMENT, "null argument");
  hipStream_t s = (hipStream_t)stream;
  uint32_t v = 0;
  hipError_t e = hipMemcpyAsync(&v, workspace, sizeof(v), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return fail(LX_ERR_HIP, hipGetErrorString(e));
  *flags = v;
  return LX_OK;
}

lx_status lx_profile_enable(int32_t on) {
  g_prof = on != 0;
  return LX_OK;
}

lx_status lx_profile_collect(void) {
  for (const ProfRec& r : g_pending) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess) return fail(LX_ERR_HIP, hipGetErrorString(e));
    auto it = std::find_if(g_tot.begin(), g_tot.end(),
                           [&](const std::pair<const char*, std::pair<int64_t, double>>& p) {
                             return std::string(p.first) == r.name;
                           });
    if (it == g_tot.end()) {
      g_tot.push_back({r.name, {1, (double)ms}});
    } else {
      it->second.first += 1;
      it->second.second += ms;
    }
    g_pool.push_back(r.a);
    g_pool.push_back(r.b);
  }
  g_pending.clear();
  return LX_OK;
}

int32_t lx_profile_count(void) { return (int32_t)g_tot.size(); }

lx_status lx_profile_entry(int32_t i, const char** name, int64_t* launches, double* total_ms) {
  if (i < 0 || i >= (int32_t)g_tot.size()) return fail(LX_ERR_INVALID_ARGUMENT, "profile index out of range");
  if (name) *name = g_tot[i].first;
  if (launches) *launches = g_tot[i].second.first;
  if (total_ms) *total_ms = g_tot[i].second.second;
  return LX_OK;
}

lx_status lx_profile_reset(void) {
  lx_profile_collect();
  g_tot.clear();
  return LX_OK;
}

}  // extern "C"
