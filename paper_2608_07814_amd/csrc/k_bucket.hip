// Routing bucketing (first step of the forward).
//
// The amortized forward (Sec. 5.1) computes each shared term once per token:
// the anchor's gate/up once per (token, anchor), each node's correction once
// per (token, node). Bucketing lists those unique (token, node) pairs for
// every tree level, sorted by (node, token), and maps every routing slot to
// its row. The result is a pure function of the inputs (no atomics decide an
// order), so it is bit-identical run to run.
//
// Three passes over 64-token tiles (one wavefront each):
//   hist  : per (level, tile) a 64-bit LDS mask per node marks the tile's
//           tokens that reach the node; popcounts give hist[node][tile];
//   scan  : per level, an exclusive scan of hist in (node, tile) order gives
//           each (node, tile) its first row; node offsets and the GEMM tile
//           table follow;
//   place : the masks are rebuilt; a token's row inside its (node, tile)
//           segment is the popcount of the mask bits below its lane.
#include "lx_internal.h"
#include "lx_topk.h"

namespace lx {
namespace {

// single-workgroup path: nodes (and experts) per level, and tree nodes in all
// correction levels together
constexpr int kSmallMaxNodes = 1024, kSmallMaxTree = 1024;
constexpr int kPlaceThr = 256;  // placement: threads per 64-token tile
constexpr int kScanThr = 1024;  // scan: threads of the one workgroup per level

// Inclusive prefix sum over the 64 lanes of a wavefront; every lane must be
// active. Row shifts (DPP) scan each row of 16 lanes, then each row adds the
// totals of the rows before it, read from lanes 15, 31 and 47.
__device__ __forceinline__ int wave_incl_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);  // row_shr:8
  const int r0 = __builtin_amdgcn_readlane(x, 15), r1 = __builtin_amdgcn_readlane(x, 31),
            r2 = __builtin_amdgcn_readlane(x, 47);
  const int row = (threadIdx.x & 63) >> 4;
  return x + (row >= 1 ? r0 : 0) + (row >= 2 ? r1 : 0) + (row >= 3 ? r2 : 0);
}

// Tile counts of a node: tile heights are powers of two (static_asserts at
// their definitions), so the division is a shift.
__device__ __forceinline__ int n_tiles_of(int cnt, int bm) { return (cnt + bm - 1) >> __builtin_ctz(bm); }

// Workgroup barrier for LDS communication only: waits for this wave's LDS
// operations, not for its global stores (which nothing in the workgroup
// reads back), unlike __syncthreads().
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xF | (0x7 << 4) | (0x3 << 14));  // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Ancestors of every expert at every level and validated factor indices.
// Single workgroup: it also zeroes the status word before anything else runs.
// Ancestors of every expert at every level and validated factor indices,
// by one workgroup; returns this thread's tree-error bits.
__device__ inline uint32_t prepare_tables(const PrepareArgs& a) {
  uint32_t bad = 0;
  const int E = a.E, L = a.L;
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    int n = e;
    bool ok = true;
    a.anc[(int64_t)L * E + e] = e;
    for (int l = L; l >= 1; --l) {
      const int p = a.parent[l][n];
      if (p < 0 || p >= a.n_nodes[l - 1]) {
        ok = false;
        break;
      }
      n = p;
      a.anc[(int64_t)(l - 1) * E + e] = n;
    }
    if (!ok) {
      bad |= LX_DEVFLAG_BAD_TREE;
      for (int l = 0; l <= L; ++l) a.anc[(int64_t)l * E + e] = -1;
    }
  }
  for (int l = 1; l <= L; ++l) {
    for (int n = threadIdx.x; n < a.n_nodes[l]; n += blockDim.x) {
      int m = a.factor_of[l][n];
      if (m < -1 || m >= a.n_factors[l]) {
        bad |= LX_DEVFLAG_BAD_TREE;
        m = -1;
      }
      a.fac[l][n] = m;
    }
  }
  return bad;
}

// Single workgroup: it also zeroes the status word before anything else runs.
__global__ __launch_bounds__(1024) void k_prepare(PrepareArgs a) {
  __shared__ uint32_t s_bad;
  if (threadIdx.x == 0) s_bad = 0;
  __syncthreads();
  const uint32_t bad = prepare_tables(a);
  if (bad) atomicOr(&s_bad, bad);
  __syncthreads();  // (also orders the tables written above for the loop below)
  if (a.path_work) {
    // an expert's path does correction work if any of its nodes carries a
    // factor (broken paths: none)
    for (int e = threadIdx.x; e < a.E; e += blockDim.x) {
      uint8_t pw = 0;
      for (int l = 1; l <= a.L; ++l) {
        const int n = a.anc[(int64_t)l * a.E + e];
        if (n >= 0 && a.fac[l][n] >= 0) pw = 1;
      }
      a.path_work[e] = pw;
    }
  }
  if (threadIdx.x == 0) *a.flags = s_bad;
}

__device__ __forceinline__ bool node_works(const BucketLevel& lv, int n) {
  return lv.work_all || (lv.work_node ? lv.work_node[n] != 0 : lv.fac[n] >= 0);
}

__device__ inline int node_of(const BucketArgs& a, int l, int e) {
  if (e < 0 || e >= a.E) return -1;
  return a.anc[(int64_t)l * a.E + e];
}

__device__ inline void build_masks(const BucketArgs& a, int l, int tt,
                                   unsigned long long* s_mask, int n_nodes) {
  const int lane = threadIdx.x;
  for (int n = lane; n < n_nodes; n += 64) s_mask[n] = 0ull;
  __syncthreads();
  const int t = tt * kTokTile + lane;
  if (t < a.T) {
    for (int j = 0; j < a.k; ++j) {
      const int n = node_of(a, l, a.ids[(int64_t)t * a.k + j]);
      if (n >= 0) atomicOr(&s_mask[n], 1ull << lane);
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(64) void k_bucket_hist(BucketArgs a) {
  extern __shared__ unsigned long long s_mask[];
  const int l = blockIdx.y, tt = blockIdx.x, lane = threadIdx.x;
  const int N = a.lv[l].n_nodes;
  build_masks(a, l, tt, s_mask, N);
  int32_t* hist = a.lv[l].hist;
  for (int n = lane; n < N; n += 64)
    hist[(int64_t)n * a.n_tok_tiles + tt] = __popcll(s_mask[n]);
  if (l == 0) {
    const int t = tt * kTokTile + lane;
    bool bad = false;
    if (t < a.T)
      for (int j = 0; j < a.k; ++j) {
        const int e = a.ids[(int64_t)t * a.k + j];
        bad |= (e < -1 || e >= a.E);
      }
    if (bad) atomicOr(a.flags, (uint32_t)LX_DEVFLAG_BAD_ID);
  }
}

// Router top-k fused with the histogram pass: one workgroup per 64-token
// tile; each wavefront picks the experts of 16 of the tile's tokens (ids and
// weights to memory, for the later passes and the forward, and ids to LDS),
// then every level's masks are built from LDS in turn.
constexpr int kRouteHistThr = 1024, kRouteTok = kTokTile / (kRouteHistThr / 64);
__global__ __launch_bounds__(kRouteHistThr) void k_bucket_hist_route(BucketArgs a) {
  extern __shared__ unsigned long long s_mask[];
  __shared__ int s_ids[kTokTile * LX_MAX_K];
  const int tt = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int k = a.k;
  const int t0 = tt * kTokTile;
  const int nt = a.T - t0 < kTokTile ? a.T - t0 : kTokTile;
  int32_t* const ids_out = const_cast<int32_t*>(a.ids);
  {
    // wavefront w: tokens w, w + 16, w + 32, w + 48 of the tile together
    int tok[kRouteTok], id[kRouteTok];
    float wt[kRouteTok];
#pragma unroll
    for (int u = 0; u < kRouteTok; ++u) {
      const int r = wave + u * (kRouteHistThr / 64);
      tok[u] = r < nt ? t0 + r : -1;
    }
    topk_tokens<kRouteTok>(a.route.logits, a.route.part, a.route.S, a.E, k, tok, id, wt);
#pragma unroll
    for (int u = 0; u < kRouteTok; ++u)
      if (tok[u] >= 0 && lane < k) {
        ids_out[(int64_t)tok[u] * k + lane] = id[u];
        const_cast<float*>(a.w)[(int64_t)tok[u] * k + lane] = wt[u];
        s_ids[(tok[u] - t0) * k + lane] = id[u];
      }
  }
  for (int l = 0; l <= a.L; ++l) {
    const int N = a.lv[l].n_nodes;
    for (int n = tid; n < N; n += kRouteHistThr) s_mask[n] = 0ull;
    __syncthreads();  // (the first round also orders the ids written above)
    for (int s = tid; s < nt * k; s += kRouteHistThr) {
      const int n = node_of(a, l, s_ids[s]);
      if (n >= 0) atomicOr(&s_mask[n], 1ull << (s / k));
    }
    __syncthreads();
    int32_t* hist = a.lv[l].hist;
    for (int n = tid; n < N; n += kRouteHistThr) hist[(int64_t)n * a.n_tok_tiles + tt] = __popcll(s_mask[n]);
    __syncthreads();  // before the next level clears the masks
  }
}

// Exclusive scan of one value per thread across the workgroup (LDS only:
// callers' pending global stores are not waited for).
__device__ inline int block_exscan(int v, int* s_wave, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  const int incl = wave_incl_scan(v);
  if (lane == 63) s_wave[wave] = incl;
  lds_barrier();
  if (threadIdx.x < 64) {
    const int w = threadIdx.x < nwaves ? s_wave[threadIdx.x] : 0;
    const int wi = wave_incl_scan(w);
    if (threadIdx.x < nwaves) s_wave[threadIdx.x] = wi - w;
    if (threadIdx.x == nwaves - 1) s_wave[63] = wi;
  }
  lds_barrier();
  const int res = s_wave[wave] + incl - v;
  total = s_wave[63];
  lds_barrier();
  return res;
}

// GEMM tile tables over the nodes that do work, in node order, one per tile
// height. off / fac: the level's node offsets and validated factor indices
// (global or LDS), complete and visible to the whole workgroup. Each thread
// reads its nodes' offsets, work flags and weight indices once (at most
// LX_MAX_NODES / 1024 nodes per thread), before the first table's stores.
__device__ inline void build_tile_tables(const BucketLevel& lv, const int32_t* off, const int32_t* fac,
                                         int* s_wave) {
  constexpr int kMaxChunk = (LX_MAX_NODES + 1023) / 1024;
  const int N = lv.n_nodes;
  const int nth = blockDim.x, tid = threadIdx.x;
  const int nchunk = (N + nth - 1) / nth;
  const int nb = tid * nchunk;
  int o_[kMaxChunk], cnt_[kMaxChunk], widx_[kMaxChunk];  // cnt_ 0: no tiles
#pragma unroll
  for (int u = 0; u < kMaxChunk; ++u) {
    const int n = nb + u;
    o_[u] = cnt_[u] = widx_[u] = 0;
    if (u < nchunk && n < N) {
      const bool work = lv.work_all || (lv.work_node ? lv.work_node[n] != 0 : fac[n] >= 0);
      o_[u] = off[n];
      cnt_[u] = work ? off[n + 1] - o_[u] : 0;
      widx_[u] = lv.work_all ? n : fac[n];
    }
  }
  for (int tab = 0; tab < kNumTab; ++tab) {
    if (!((lv.tab_mask >> tab) & 1u)) continue;  // uniform across the workgroup
    const int bm = lv.tile_bm[tab];
    TileEntry* tiles = lv.tiles[tab];
    int my_tiles = 0;
#pragma unroll
    for (int u = 0; u < kMaxChunk; ++u) my_tiles += n_tiles_of(cnt_[u], bm);
    int ntiles = 0;
    int tpos = block_exscan(my_tiles, s_wave, ntiles);
#pragma unroll
    for (int u = 0; u < kMaxChunk; ++u) {
      const int cnt = cnt_[u];
      for (int r = 0; r < cnt; r += bm) {
        TileEntry te;
        te.widx = widx_[u];
        te.row0 = o_[u] + r;
        te.nrows = cnt - r < bm ? cnt - r : bm;
        te.node = nb + u;
        tiles[tpos++] = te;
      }
    }
    if (tid == 0) *lv.n_tiles[tab] = ntiles;
  }
}

// CH: entries per thread kept in registers (8, 16 or 32, the smallest that
// holds the largest level's chunk).
template <int CH>
__global__ __launch_bounds__(kScanThr) void k_bucket_scan(BucketArgs a) {
  __shared__ int s_wave[64];
  extern __shared__ int s_off[];  // [N + 1] node offsets
  const int l = blockIdx.x;
  const BucketLevel& lv = a.lv[l];
  const int N = lv.n_nodes, NT = a.n_tok_tiles;
  const int64_t total = (int64_t)N * NT;
  constexpr int nth = kScanThr;
  const int tid = threadIdx.x;
  for (int i = tid; i < lv.n_split_cnt; i += nth) lv.split_cnt[i] = 0u;

  // exclusive scan of hist in (node, tile) order, in place; entry (n, 0)
  // is node n's offset (kept in LDS for the tile tables)
  // Each thread owns a chunk of consecutive entries (a multiple of 4, so it
  // is read and written as 16-byte vectors): up to CH entries stay in
  // registers between the two passes, all loaded at once; longer chunks are
  // read CH at a time in both passes. A block of CH entries handles only its
  // m valid ones.
  const int64_t chunk = ((total + nth - 1) / nth + 3) & ~(int64_t)3;
  const int64_t b = (int64_t)tid * chunk;
  const int64_t e = b + chunk < total ? b + chunk : total;
  auto valid = [&](int64_t c0) { return (int)(e - c0 < CH ? e - c0 : CH); };
  int v[CH];
#pragma unroll
  for (int u = 0; u < CH; ++u) v[u] = 0;
  auto load = [&](int64_t c0) {
    const int m = valid(c0);
#pragma unroll
    for (int u = 0; u < CH; u += 4) {
      if (u + 4 <= m) {
        const int4 q = *(const int4*)(lv.hist + c0 + u);
        v[u] = q.x;
        v[u + 1] = q.y;
        v[u + 2] = q.z;
        v[u + 3] = q.w;
      } else if (u < m) {
#pragma unroll
        for (int w = 0; w < 4; ++w) v[u + w] = u + w < m ? lv.hist[c0 + u + w] : 0;
      }
    }
  };
  int local = 0;
  for (int64_t c0 = b; c0 < e; c0 += CH) {
    load(c0);
    const int m = valid(c0);
#pragma unroll
    for (int u = 0; u < CH; ++u) local += u < m ? v[u] : 0;
  }
  int grand = 0;
  int run = block_exscan(local, s_wave, grand);
  // next node start at or after b (its entries begin at nnode * NT)
  int nnode = 0;  // at most N (LX_MAX_NODES)
  if (b < e) {
    if (b < ((int64_t)1 << 31)) {
      const uint32_t q = (uint32_t)b / (uint32_t)NT;
      nnode = (int)q + ((int64_t)q * NT != b ? 1 : 0);
    } else {
      nnode = (int)((b + NT - 1) / NT);
    }
  }
  for (int64_t c0 = b; c0 < e; c0 += CH) {
    if (e - b > CH) load(c0);  // chunk larger than the register cache: reload
    const int m = valid(c0);
    // position of the next node start within this block (CH: none)
    const int64_t nx = (int64_t)nnode * NT - c0;
    int nxt = nx < CH ? (int)nx : CH;
    if (NT >= CH) {
      // at most one node start in the block: its offset is selected, no
      // branches per entry (entries past m are not stored)
      int bval = 0;
#pragma unroll
      for (int u = 0; u < CH; ++u) {
        const int cnt = u < m ? v[u] : 0;
        v[u] = run;
        bval = u == nxt ? run : bval;
        run += cnt;
      }
      if (nxt < m) {
        s_off[nnode] = bval;
        ++nnode;
      }
    } else {
#pragma unroll
      for (int u = 0; u < CH; ++u) {
        if (u < m) {
          const int cnt = v[u];
          v[u] = run;
          if (u == nxt) {
            s_off[nnode] = run;
            ++nnode;
            nxt += NT;
          }
          run += cnt;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < CH; u += 4) {
      if (u + 4 <= m) {
        *(int4*)(lv.hist + c0 + u) = make_int4(v[u], v[u + 1], v[u + 2], v[u + 3]);
      } else if (u < m) {
#pragma unroll
        for (int w = 0; w < 4; ++w)
          if (u + w < m) lv.hist[c0 + u + w] = v[u + w];
      }
    }
  }
  if (tid == 0) s_off[N] = grand;
  lds_barrier();
  for (int n = tid; n <= N; n += nth) lv.offsets[n] = s_off[n];
  build_tile_tables(lv, s_off, lv.fac, s_wave);
}

// One thread per routing slot of the tile's 64 tokens.
__global__ __launch_bounds__(kPlaceThr) void k_bucket_place(BucketArgs a) {
  extern __shared__ unsigned long long s_mask[];
  __shared__ int s_node[kTokTile * LX_MAX_K];
  const int l = blockIdx.y, tt = blockIdx.x, tid = threadIdx.x;
  const BucketLevel& lv = a.lv[l];
  const int N = lv.n_nodes, k = a.k;
  const int t0 = tt * kTokTile;
  const int nt = a.T - t0 < kTokTile ? a.T - t0 : kTokTile;
  const int TK = nt * k;
  for (int n = tid; n < N; n += blockDim.x) s_mask[n] = 0ull;
  lds_barrier();
  for (int s = tid; s < TK; s += blockDim.x) {
    const int n = node_of(a, l, a.ids[(int64_t)t0 * k + s]);
    s_node[s] = n;
    if (n >= 0) atomicOr(&s_mask[n], 1ull << (s / k));
  }
  lds_barrier();
  for (int s = tid; s < TK; s += blockDim.x) {
    const int t = s / k, j = s - t * k;
    const int64_t gs = (int64_t)t0 * k + s;
    const int n = s_node[s];
    if (n < 0) {
      lv.slot_row[gs] = -1;
      lv.slot_flags[gs] = 0;
      if (l == a.L && a.w) a.slot_wsum[gs] = 0.f;
      continue;
    }
    const int row = lv.hist[(int64_t)n * a.n_tok_tiles + tt] + __popcll(s_mask[n] & ((1ull << t) - 1ull));
    lv.slot_row[gs] = row;
    bool first = true;
    for (int j2 = 0; j2 < j; ++j2) first &= (s_node[t * k + j2] != n);
    if (first) lv.row_token[row] = t0 + t;
    const bool work = node_works(lv, n);
    lv.slot_flags[gs] = (uint8_t)((first ? 1 : 0) | (work ? 2 : 0));
    // expert level: summed weight of each distinct expert, on its first slot
    if (l == a.L && a.w) {
      float ws = 0.f;
      if (first)
        for (int j2 = j; j2 < k; ++j2)
          if (s_node[t * k + j2] == n) ws += a.w[(int64_t)(t0 + t) * k + j2];
      a.slot_wsum[gs] = ws;
    }
  }
}

// One thread per routing slot; the first slot of each leaf row writes that
// row's map entries.
__global__ __launch_bounds__(256) void k_leaf_maps(LeafMapArgs a) {
  const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= (int64_t)a.T * a.k) return;
  if (!(a.slot_flags[a.L][s] & 1)) return;  // not the first slot of a leaf row (or dropped)
  const int rL = a.slot_row[a.L][s];
  for (int l = 1; l < a.L; ++l) a.leaf_row_map[l][rL] = a.slot_row[l][s];
}

// Whole bucketing of a batch of at most 64 tokens in one workgroup. All
// global inputs are read into LDS once; then per level three phases, each
// ended by one barrier:
//   A  every thread: the node of each routing slot (walking the parent
//      arrays to the root, so a broken path invalidates the expert at every
//      level, as in k_prepare), one 64-bit token mask per node (the batch is
//      one token tile), validated factor indices;
//   B  wavefront 0 alone (no barriers): node offsets and the tile tables by
//      wavefront-wide scans;
//   C  every thread: slot placement, one thread per routing slot.
// Same results as the four-pass path with one token tile.
// Levels are processed in pairs (l0, l0 + 1): index q of the per-level
// arrays is the level's place in its pair. Nodes and ids are below
// kSmallMaxNodes, so 16 bits hold them (ids outside [0, E) are kept as -1).
struct SmallLds {
  unsigned long long mask[2][kSmallMaxNodes];
  int32_t off[2][kSmallMaxNodes + 1];
  int32_t fac[2][kSmallMaxNodes];
  int32_t par[kSmallMaxTree];   // parent arrays of levels 1..L, concatenated
  int32_t fo[kSmallMaxTree];    // factor_of arrays of levels 1..L, concatenated
  int16_t node[2][kTokTile * LX_MAX_K];
  int16_t ids[kTokTile * LX_MAX_K];
  float w[kTokTile * LX_MAX_K];
  int32_t base[kMaxLvl];        // offset of level l's arrays in par / fo
  uint32_t bad;
};
static_assert(sizeof(SmallLds) <= 64 * 1024, "single-workgroup bucketing: default LDS limit");

// Node of expert e at level l, or -1 (invalid id or broken path to the root).
__device__ inline int small_node(const SmallLds& S, const PrepareArgs& pa, int L, int E, int e, int l) {
  if (e < 0 || e >= E) return -1;
  int n = e, at = l == L ? e : -1;
  for (int q = L; q >= 1; --q) {
    const int p = S.par[S.base[q] + n];
    if (p < 0 || p >= pa.n_nodes[q - 1]) return -1;
    n = p;
    if (q - 1 == l) at = n;
  }
  return at;
}


__device__ inline int wave_exscan(int v, int& total) {
  const int incl = wave_incl_scan(v);
  total = __builtin_amdgcn_readlane(incl, 63);
  return incl - v;
}

// NL = the number of correction levels, a compile-time constant so that every
// per-level loop unrolls and the level descriptors are read at fixed offsets
// (their loads are issued together instead of one dependent load per use).
template <int NL>
__global__ __launch_bounds__(1024) void k_bucket_small(PrepareArgs pa, BucketArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char s_raw[];
  SmallLds& S = *(SmallLds*)s_raw;
  const int tid = threadIdx.x, nth = blockDim.x;
  const int T = a.T, k = a.k, TK = T * k, E = a.E;
  constexpr int L = NL;
  if (tid == 0) {
    S.bad = 0;
    int o = 0;
#pragma unroll
    for (int l = 1; l <= L; ++l) {
      S.base[l] = o;
      o += pa.n_nodes[l];
    }
  }
  lds_barrier();
  uint32_t bad = 0;
  for (int s = tid; s < TK; s += nth) {
    const int e = a.ids[s];
    S.ids[s] = (int16_t)(e >= 0 && e < E ? e : -1);
    S.w[s] = a.w ? a.w[s] : 0.f;
    if (e < -1 || e >= E) bad |= LX_DEVFLAG_BAD_ID;
  }
#pragma unroll
  for (int l = 1; l <= L; ++l)
    for (int n = tid; n < pa.n_nodes[l]; n += nth) {
      S.par[S.base[l] + n] = pa.parent[l][n];
      S.fo[S.base[l] + n] = pa.factor_of[l][n];
    }
  for (int n = tid; n < a.lv[0].n_nodes; n += nth) S.mask[0][n] = 0ull;
  if (L >= 1)
    for (int n = tid; n < a.lv[L >= 1 ? 1 : 0].n_nodes; n += nth) S.mask[1][n] = 0ull;
#pragma unroll
  for (int l = 0; l <= L; ++l)
    for (int i = tid; i < a.lv[l].n_split_cnt; i += nth) a.lv[l].split_cnt[i] = 0u;
  lds_barrier();

  // A: slot nodes, the level's token masks and validated factor indices
  auto phase_a = [&](const int l, const int q) {
    const int N = a.lv[l].n_nodes;
    unsigned long long* const mask = S.mask[q];
    for (int s = tid; s < TK; s += nth) {
      const int n = small_node(S, pa, L, E, S.ids[s], l);
      S.node[q][s] = (int16_t)n;
      if (n >= 0) atomicOr(&mask[n], 1ull << (s / k));
    }
    for (int n = tid; n < N; n += nth) {
      int m = -1;
      if (l > 0) {
        m = S.fo[S.base[l] + n];
        if (m < -1 || m >= pa.n_factors[l]) {
          bad |= LX_DEVFLAG_BAD_TREE;
          m = -1;
        }
      }
      S.fac[q][n] = m;
    }
    if (l == 0)  // tree check of every expert, routed or not
      for (int e = tid; e < E; e += nth)
        if (L > 0 && small_node(S, pa, L, E, e, 0) < 0) bad |= LX_DEVFLAG_BAD_TREE;
  };
  // B (one wavefront): node offsets by a wavefront scan, then the tile tables
  auto phase_b = [&](const int l, const int q) {
    const BucketLevel& lv = a.lv[l];
    const int N = lv.n_nodes;
    const unsigned long long* const mask = S.mask[q];
    int* const off = S.off[q];
    const int* const fac = S.fac[q];
    const int lane = tid & 63;
    const int per = (N + 63) / 64;
    const int nb = lane * per, ne = nb + per < N ? nb + per : N;
    int local = 0;
    for (int n = nb; n < ne; ++n) local += __popcll(mask[n]);
    int total = 0;
    int run = wave_exscan(local, total);
    for (int n = nb; n < ne; ++n) {
      off[n] = run;
      lv.hist[n] = run;
      lv.offsets[n] = run;
      run += __popcll(mask[n]);
    }
    if (lane == 0) {
      off[N] = total;
      lv.offsets[N] = total;
    }
    // off[ne] is read below but written by the next lane: keep the
    // compiler from hoisting reads above the writes (a wavefront's LDS
    // accesses execute in program order)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_wave_barrier();
    asm volatile("" ::: "memory");
    for (int tab = 0; tab < kNumTab; ++tab) {
      if (!((lv.tab_mask >> tab) & 1u)) continue;
      const int bm = lv.tile_bm[tab];
      int mine = 0;
      for (int n = nb; n < ne; ++n) {
        const int cnt = off[n + 1] - off[n];
        if ((lv.work_all || fac[n] >= 0) && cnt > 0) mine += n_tiles_of(cnt, bm);
      }
      int ntiles = 0;
      int tpos = wave_exscan(mine, ntiles);
      for (int n = nb; n < ne; ++n) {
        const int o = off[n], cnt = off[n + 1] - o;
        if (!(lv.work_all || fac[n] >= 0) || cnt == 0) continue;
        const int widx = lv.work_all ? n : fac[n];
        for (int r = 0; r < cnt; r += bm) {
          TileEntry te;
          te.widx = widx;
          te.row0 = o + r;
          te.nrows = cnt - r < bm ? cnt - r : bm;
          te.node = n;
          lv.tiles[tab][tpos++] = te;
        }
      }
      if (lane == 0) *lv.n_tiles[tab] = ntiles;
    }
  };
  // C: each slot's row, first-slot flags, row tokens, summed weights
  auto phase_c = [&](const int l, const int q) {
    const BucketLevel& lv = a.lv[l];
    const unsigned long long* const mask = S.mask[q];
    for (int s = tid; s < TK; s += nth) {
      const int t = s / k, j = s - t * k;
      const int n = S.node[q][s];
      if (n < 0) {
        lv.slot_row[s] = -1;
        lv.slot_flags[s] = 0;
        if (l == L && a.w) a.slot_wsum[s] = 0.f;
        continue;
      }
      const int row = S.off[q][n] + __popcll(mask[n] & ((1ull << t) - 1ull));
      lv.slot_row[s] = row;
      bool first = true;
      for (int j2 = 0; j2 < j; ++j2) first &= (S.node[q][t * k + j2] != n);
      if (first) lv.row_token[row] = t;
      const bool work = lv.work_all || S.fac[q][n] >= 0;
      lv.slot_flags[s] = (uint8_t)((first ? 1 : 0) | (work ? 2 : 0));
      // expert level: summed weight of each distinct expert, on its first slot
      if (l == L && a.w) {
        float ws = 0.f;
        if (first)
          for (int j2 = j; j2 < k; ++j2)
            if (S.node[q][t * k + j2] == n) ws += S.w[t * k + j2];
        a.slot_wsum[s] = ws;
      }
    }
  };

  // levels in pairs: both levels' A, then B on wavefronts 0 and 1, then both C
#pragma unroll
  for (int l0 = 0; l0 <= L; l0 += 2) {
    const bool two = l0 + 1 <= L;
    phase_a(l0, 0);
    if (two) phase_a(l0 + 1, 1);
    lds_barrier();
    if (tid < 64)
      phase_b(l0, 0);
    else if (two && tid < 128)
      phase_b(l0 + 1, 1);
    lds_barrier();
    phase_c(l0, 0);
    if (two) phase_c(l0 + 1, 1);
    if (l0 + 2 <= L) {  // the next pair's masks (both read by the C phase above)
      lds_barrier();
      for (int n = tid; n < a.lv[l0 + 2].n_nodes; n += nth) S.mask[0][n] = 0ull;
      if (l0 + 3 <= L)
        for (int n = tid; n < a.lv[l0 + 3 <= L ? l0 + 3 : l0 + 2].n_nodes; n += nth) S.mask[1][n] = 0ull;
      lds_barrier();
    }
  }
  if (bad) atomicOr(&S.bad, bad);
  lds_barrier();
  if (tid == 0) *a.flags = S.bad;
}

}  // namespace

static size_t mask_lds_bytes(const BucketArgs& a) {
  int mx = 1;
  for (int l = 0; l <= a.L; ++l) mx = a.lv[l].n_nodes > mx ? a.lv[l].n_nodes : mx;
  return (size_t)mx * sizeof(unsigned long long);
}

hipError_t launch_prepare(const PrepareArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_prepare, dim3(1), dim3(1024), 0, s, a);
  return hipGetLastError();
}

bool bucket_small_ok(const BucketArgs& a) {
  if (a.T < 1 || a.T > kTokTile || a.k > LX_MAX_K || a.E > kSmallMaxNodes) return false;
  int tree = 0;
  for (int l = 0; l <= a.L; ++l) {
    if (a.lv[l].n_nodes > kSmallMaxNodes) return false;
    if (l > 0) tree += a.lv[l].n_nodes;
  }
  return tree <= kSmallMaxTree;
}

hipError_t launch_bucket_small(const PrepareArgs& pa, const BucketArgs& a, hipStream_t s) {
  switch (a.L) {
    case 0: hipLaunchKernelGGL(k_bucket_small<0>, dim3(1), dim3(1024), sizeof(SmallLds), s, pa, a); break;
    case 1: hipLaunchKernelGGL(k_bucket_small<1>, dim3(1), dim3(1024), sizeof(SmallLds), s, pa, a); break;
    case 2: hipLaunchKernelGGL(k_bucket_small<2>, dim3(1), dim3(1024), sizeof(SmallLds), s, pa, a); break;
    case 3: hipLaunchKernelGGL(k_bucket_small<3>, dim3(1), dim3(1024), sizeof(SmallLds), s, pa, a); break;
    default: hipLaunchKernelGGL(k_bucket_small<4>, dim3(1), dim3(1024), sizeof(SmallLds), s, pa, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_leaf_maps(const LeafMapArgs& a, hipStream_t s) {
  const int64_t n = (int64_t)a.T * a.k;
  const int grid = (int)((n + 255) / 256);
  hipLaunchKernelGGL(k_leaf_maps, dim3(grid > 0 ? grid : 1), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_bucket_hist_route(const BucketArgs& a, hipStream_t s) {
  if (a.n_tok_tiles == 0) return hipSuccess;
  hipLaunchKernelGGL(k_bucket_hist_route, dim3(a.n_tok_tiles), dim3(kRouteHistThr), mask_lds_bytes(a), s, a);
  return hipGetLastError();
}

hipError_t launch_bucket_hist(const BucketArgs& a, hipStream_t s) {
  if (a.n_tok_tiles == 0) return hipSuccess;
  hipLaunchKernelGGL(k_bucket_hist, dim3(a.n_tok_tiles, a.L + 1), dim3(64), mask_lds_bytes(a), s, a);
  return hipGetLastError();
}

hipError_t launch_bucket_scan(const BucketArgs& a, hipStream_t s) {
  int mx = 1;
  int64_t chunk = 0;  // the kernel's per-thread chunk at the largest level
  for (int l = 0; l <= a.L; ++l) {
    mx = a.lv[l].n_nodes > mx ? a.lv[l].n_nodes : mx;
    const int64_t total = (int64_t)a.lv[l].n_nodes * a.n_tok_tiles;
    const int64_t c = ((total + kScanThr - 1) / kScanThr + 3) & ~(int64_t)3;
    chunk = c > chunk ? c : chunk;
  }
  const size_t lds = (size_t)(mx + 1) * sizeof(int);
  if (chunk <= 8)
    hipLaunchKernelGGL(k_bucket_scan<8>, dim3(a.L + 1), dim3(kScanThr), lds, s, a);
  else if (chunk <= 16)
    hipLaunchKernelGGL(k_bucket_scan<16>, dim3(a.L + 1), dim3(kScanThr), lds, s, a);
  else
    hipLaunchKernelGGL(k_bucket_scan<32>, dim3(a.L + 1), dim3(kScanThr), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_bucket_place(const BucketArgs& a, hipStream_t s) {
  if (a.n_tok_tiles == 0) return hipSuccess;
  hipLaunchKernelGGL(k_bucket_place, dim3(a.n_tok_tiles, a.L + 1), dim3(kPlaceThr), mask_lds_bytes(a), s, a);
  return hipGetLastError();
}

}  // namespace lx
