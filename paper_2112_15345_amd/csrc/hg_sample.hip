// Per-hop neighbour sampling on gfx950 (DistDGLv2, arXiv 2112.15345, Sec. 3.2
// and Sec. 4.2.2): the counting pass over (frontier vertex, edge type) pairs
// and the fanout sampler.
//
// Each pair keeps min(deg, K) of its in-edges: all of them when deg <= K (or
// K == -1), else the K with the smallest (key, edge ID), where the key of edge
// `eid` is word (eid & 3) of Philox4x32-10 at counter (eid >> 2, hop, etype)
// under the sampling seed.  Kept edges are written grouped by pair, ascending
// edge ID within a pair.
//
// Work is split by pair shape: a wavefront takes 64 consecutive pairs and
// writes the kept edges of those that keep every one of at most
// kThreadTakeAll in-edges or select among at most kLaneSelect (one lane ranks
// such a pair's keys); other pairs run one per wavefront; pairs that select
// among more than kHubChunk edges ("hubs") are cut into chunks of kHubChunk
// edges, handed to wavefronts in runs of consecutive chunks, which append
// their candidates to a per-hub list; a second launch then selects each hub's
// K edges from its list.  Every edge key is computed once.  Pairs of more
// than kHubChunk edges that keep all of them (none excluded) are hubs too:
// their chunks are copied straight to the output, and the second launch skips
// them.  Every kept edge marks its source reached (a byte, or a bit on hops
// that keep few edges next to the graph's vertices) for the compaction.
#include <hip/hip_ext.h>

#include <algorithm>

#include "hg_device.hpp"
#include "hg_internal.hpp"

namespace hg {

namespace {

__device__ __forceinline__ int64_t grid_stride_start() {
  return int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
}
__device__ __forceinline__ int64_t grid_stride_step() {
  return int64_t(gridDim.x) * blockDim.x;
}

unsigned grid_for(int64_t n, int threads, int64_t cap = 1 << 20) {
  int64_t b = (n + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return unsigned(b);
}

// Node type of item x of a concatenation of the hop's frontiers.
__device__ __forceinline__ int type_of(const int64_t *nF, int32_t n_types,
                                       int64_t x, int64_t *first) {
  int64_t acc = 0;
  int t = 0;
  for (; t < n_types - 1; ++t) {
    if (x < acc + nF[t]) break;
    acc += nF[t];
  }
  *first = acc;
  return t;
}

// ---- exclusion lookups (edge-seeded mini-batches) ---------------------------

// Excluded in-edges of the pair (etype e, destination local ID i).
__device__ __forceinline__ int32_t excl_count(const ExclView &X, int e, int64_t i) {
  if (!X.pair_keys || i >= X.n_seed[e]) return 0;
  const uint64_t key = (uint64_t(uint32_t(e)) << 32) | uint64_t(i);
  for (uint32_t h = hash_slot(key, X.pair_mask);; h = (h + 1) & X.pair_mask) {
    const uint64_t k = X.pair_keys[h];
    if (k == key) return X.pair_cnt[h];
    if (k == kHashEmpty) return 0;
  }
}

// Whether edge `eid` of etype e is excluded (the table has empty slots, so a
// probe run always ends).
__device__ __forceinline__ bool is_excluded(const ExclView &X, int e, uint64_t eid) {
  const uint64_t key = (uint64_t(uint32_t(e)) << 32) | uint64_t(uint32_t(eid));
  for (uint32_t h = hash_slot(key, X.edge_mask);; h = (h + 1) & X.edge_mask) {
    const uint64_t k = X.edge_keys[h];
    if (k == key) return true;
    if (k == kHashEmpty) return false;
  }
}

// ---- frontier map maintenance --------------------------------------------

__global__ void k_insert_frontier(HopView hv, const TypeStatic *ts,
                                  int32_t n_types, int64_t total, int64_t *small) {
  int32_t *err = reinterpret_cast<int32_t *>(small + kSlotErr);
  for (int64_t x = grid_stride_start(); x < total; x += grid_stride_step()) {
    int64_t first;
    const int t = type_of(hv.nF, n_types, x, &first);
    const int64_t i = x - first;
    if (i >= hv.nF[t]) continue;
    const int64_t v = hv.frontier[t][i];
    if (v < 0 || v >= ts[t].num_nodes) {
      atomicOr(err, kErrSeedRange);
      continue;
    }
    // the first seed to set the frontier bit owns the vertex; a later one
    // is a repeat
    const uint32_t bit = 1u << (v & 31);
    if (atomicOr(ts[t].fbits + (v >> 5), bit) & bit)
      atomicOr(err, kErrSeedRepeat);
    else
      ts[t].map[v] = int32_t(i);
  }
}

// ---- counting pass ---------------------------------------------------------

// Per pair: kept edges s, hub chunks, "one wavefront" flag, hub flag.
// What the counting pass keeps of a pair until its outputs are written, next
// to its kept count: its hub chunk count (a pair has fewer than 2^32 in-edges,
// so fewer than 2^21 chunks) and whether it takes the wavefront or the hub role.
constexpr uint32_t kPairWave = 1u << 30, kPairHub = 1u << 31, kPairChunks = kPairWave - 1;

// Per edge type, what the counting pass reads for every pair; staged in
// (dynamic) LDS, 52 bytes per edge type, when the graph has at most
// kCountMaxEtypes edge types (a bundle's virtual graph counts each copy).
constexpr int kCountMaxEtypes = 1200;
struct CountTable {
  int64_t *pbase;  // [n + 1]
  const int64_t **indptr;
  const int64_t **front;
  int64_t *n_dst;
  const uint32_t **nz_mask;
  int32_t *fanout, *nz_words, *nz_slot;
  __host__ __device__ static constexpr size_t bytes(int n) {
    return size_t(8) * (n + 1) + size_t(8) * 4 * n + size_t(4) * 3 * n;
  }
  __device__ void carve(char *p, int n) {
    pbase = reinterpret_cast<int64_t *>(p);
    indptr = reinterpret_cast<const int64_t **>(pbase + n + 1);
    front = reinterpret_cast<const int64_t **>(indptr + n);
    n_dst = reinterpret_cast<int64_t *>(front + n);
    nz_mask = reinterpret_cast<const uint32_t **>(n_dst + n);
    fanout = reinterpret_cast<int32_t *>(nz_mask + n);
    nz_words = fanout + n;
    nz_slot = nz_words + n;
  }
};
static_assert(CountTable::bytes(kCountMaxEtypes) <= 64 * 1024, "the table fits 64 KiB of LDS");

template <bool kStaged>
struct CountView {
  const CountTable *t;
  const HopView *hv;
  const EtypeStatic *es;
  __device__ int64_t pbase(int e) const { return kStaged ? t->pbase[e] : hv->pair_base[e]; }
  __device__ const int64_t *indptr(int e) const { return kStaged ? t->indptr[e] : es[e].indptr; }
  __device__ const int64_t *front(int e) const {
    return kStaged ? t->front[e] : hv->frontier[es[e].dst_type];
  }
  __device__ int64_t n_dst(int e) const { return kStaged ? t->n_dst[e] : es[e].n_dst_nodes; }
  __device__ int32_t fanout(int e) const { return kStaged ? t->fanout[e] : hv->fanout[e]; }
  __device__ const uint32_t *nz_mask(int e) const { return kStaged ? t->nz_mask[e] : es[e].nz_mask; }
  __device__ int32_t nz_words(int e) const { return kStaged ? t->nz_words[e] : es[e].nz_words; }
  __device__ int32_t nz_slot(int e) const { return kStaged ? t->nz_slot[e] : es[e].nz_slot; }
};

// Thread i of a tile owns kPairItems consecutive pairs.  The pair's edge type
// comes from the (staged) table; the frontier vertices of all items are
// loaded together, then their indptr entries, so a thread waits on two
// rounds of memory accesses.
template <bool kStaged, int kPairItems>
__global__ __launch_bounds__(kTileThreads) void k_count_scan(
    HopView hv, const EtypeStatic *es, int32_t n_etypes, int32_t n_types,
    int64_t n_items, PairArrays pa, Lookback lb, uint32_t epoch,
    uint64_t ticket_base, ExclView X, int64_t *small) {
  __shared__ int64_t lds[16];
  extern __shared__ __align__(16) char count_lds[];
  CountTable table;
  if (kStaged) {
    table.carve(count_lds, n_etypes);
    for (int e = threadIdx.x; e <= n_etypes; e += kTileThreads) {
      table.pbase[e] = hv.pair_base[e];
      if (e < n_etypes) {
        const EtypeStatic &E = es[e];
        table.indptr[e] = E.indptr;
        table.front[e] = hv.frontier[E.dst_type];
        table.n_dst[e] = E.n_dst_nodes;
        table.fanout[e] = hv.fanout[e];
        table.nz_mask[e] = E.nz_mask;
        table.nz_words[e] = E.nz_words;
        table.nz_slot[e] = E.nz_slot;
      }
    }
  }
  const int64_t tile = take_ticket(small, ticket_base, lds);  // also a barrier
  const CountView<kStaged> V{&table, &hv, es};
  const int64_t P = V.pbase(n_etypes);
  const int64_t base = (tile * kTileThreads + threadIdx.x) * kPairItems;
  int32_t *err = reinterpret_cast<int32_t *>(small + kSlotErr);
  if (tile == 0 && threadIdx.x == 0 && P + 1 > n_items) atomicOr(err, kErrBound);

  // edge type of every item; bit k of `valid` says item k is a pair (not past
  // the pairs), bit k of `reads` that it reads its indptr entries
  int etype[kPairItems];
  uint32_t valid = 0, reads = 0;
  {
    int e = 0;
    if (base < P) {
      int lo = 0, hi = n_etypes;  // pbase(lo) <= base < pbase(hi)
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (V.pbase(mid) <= base)
          lo = mid;
        else
          hi = mid;
      }
      e = lo;
    }
#pragma unroll
    for (int k = 0; k < kPairItems; ++k) {
      const int64_t p = base + k;
      if (p < P) {
        while (V.pbase(e + 1) <= p) ++e;
        valid |= 1u << k;
      }
      etype[k] = e;
    }
  }
  // the frontier vertex of every item (all loads issued together)
  int64_t v[kPairItems];
#pragma unroll
  for (int k = 0; k < kPairItems; ++k)
    v[k] = (valid >> k) & 1 ? load_global(V.front(etype[k]) + (base + k - V.pbase(etype[k]))) : 0;
#pragma unroll
  for (int k = 0; k < kPairItems; ++k) {
    if ((valid >> k) & 1) {
      if (v[k] >= 0 && v[k] < V.n_dst(etype[k]))
        reads |= 1u << k;
      else
        atomicOr(err, kErrSeedRange);
    }
  }
  // with a non-empty mask, a pair whose destination has no in-edge of its
  // type reads no indptr (one mask word, shared by the vertex's edge types)
#pragma unroll
  for (int k = 0; k < kPairItems; ++k) {
    const uint32_t *m = (reads >> k) & 1 ? V.nz_mask(etype[k]) : nullptr;
    if (m) {
      const int32_t slot = V.nz_slot(etype[k]);
      const uint32_t w = load_global(m + v[k] * V.nz_words(etype[k]) + (slot >> 5));
      if (((w >> (slot & 31)) & 1u) == 0) reads &= ~(1u << k);
    }
  }
  int64_t lo[kPairItems], hi[kPairItems];
#pragma unroll
  for (int k = 0; k < kPairItems; ++k) {
    const int64_t *ip = V.indptr(etype[k]) + v[k];
    lo[k] = (reads >> k) & 1 ? load_global(ip) : 0;
    hi[k] = (reads >> k) & 1 ? load_global(ip + 1) : 0;
  }

  // per item: kept count cs and the packed chunk count and role flags cf;
  // the keys the sampler will evaluate (every in-edge of a pair that selects
  // among its in-edges) summed per thread
  int64_t cs[kPairItems];
  uint32_t cf[kPairItems];
  int64_t keys = 0;
#pragma unroll
  for (int k = 0; k < kPairItems; ++k) {
    const int64_t p = base + k;
    cs[k] = 0;
    cf[k] = 0;
    if (!((valid >> k) & 1)) continue;  // past the pairs (an out-of-range vertex counts as deg 0)
    const int64_t deg = hi[k] - lo[k];
    const int64_t K = V.fanout(etype[k]);
    // in-edges that take part: all but the excluded ones
    const int32_t nx = excl_count(X, etype[k], p - V.pbase(etype[k]));
    const int64_t avail = deg - nx;
    const int64_t s = (K < 0 || avail <= K) ? avail : K;
    cs[k] = s;
    if (s < avail) keys += deg;  // a selection keys every in-edge
    if (deg > kHubChunk && (s < avail || nx == 0)) {
      cf[k] = uint32_t((deg + kHubChunk - 1) / kHubChunk) | kPairHub;
    } else if (nx == 0 && s < deg && deg <= kLaneSelect) {
      // one lane of the pair-group role ranks its keys
    } else if (s > 0 && !(nx == 0 && s == deg && deg <= kThreadTakeAll)) {
      cf[k] = kPairWave;  // pairs with excluded edges always take this role
    }
    if (deg > 0) {  // nothing reads these for an empty pair
      pa.plo[p] = lo[k];
      pa.pdeg[p] = deg;
    }
  }

  // the keys: wavefront sums in LDS, added up by thread 0 after the block
  // scan's barriers (one atomic per tile)
  __shared__ int64_t s_keys[kTileThreads / kWave];
  keys = wave_sum_i64(keys);
  if (lane_id() == 0) s_keys[threadIdx.x / kWave] = keys;

  // block scan of the per-thread sums, then the tile's prefix by look-back
  int64_t sum[4] = {0, 0, 0, 0};
#pragma unroll
  for (int k = 0; k < kPairItems; ++k) {
    sum[0] += cs[k];
    sum[1] += cf[k] & kPairChunks;
    sum[2] += (cf[k] & kPairWave) ? 1 : 0;
    sum[3] += (cf[k] & kPairHub) ? 1 : 0;
  }
  int64_t pre[4], agg[4];
  block_excl_scan4_256(sum, pre, agg, lds);
  if (threadIdx.x == 0) {
    int64_t keys = 0;
#pragma unroll
    for (int w = 0; w < kTileThreads / kWave; ++w) keys += s_keys[w];
    if (keys)
      atomicAdd(reinterpret_cast<unsigned long long *>(small + kSlotKeys),
                (unsigned long long)keys);
  }
  int64_t ex[4];
  tile_lookback<4>(lb, tile, 0, epoch, agg, ex, small);
#pragma unroll
  for (int a = 0; a < 4; ++a) pre[a] += ex[a];

  int64_t *ebase = small + kSlotNew + n_types;
#pragma unroll
  for (int k = 0; k < kPairItems; ++k) {
    const int64_t p = base + k;
    const bool wave = (cf[k] & kPairWave) != 0, hub = (cf[k] & kPairHub) != 0;
    if (p < n_items) {
      pa.off[p] = pre[0];
      pa.pet[p] = etype[k];
      if (wave) pa.wlist[pre[2]] = p;
      if (hub) {
        pa.hub_cnt[pre[3]] = 0;
        pa.hub_pair[pre[3]] = p;
        pa.hub_choff[pre[3]] = pre[1];
      }
      // edge start of every etype whose first pair (or end, for the last) is p
      if (p <= P) {
        const int e = p < P ? etype[k] : n_etypes;
        for (int e2 = e; e2 >= 0 && V.pbase(e2) == p; --e2) ebase[e2] = pre[0];
      }
    }
    pre[0] += cs[k];
    pre[1] += cf[k] & kPairChunks;
    pre[2] += wave ? 1 : 0;
    pre[3] += hub ? 1 : 0;
  }
  // the last tile holds the totals
  if (tile == int64_t(gridDim.x) - 1 && threadIdx.x == kTileThreads - 1) {
    small[kSlotPairs] = P;
    small[kSlotEdges] = pre[0];
    small[kSlotChunks] = pre[1];
    small[kSlotWaves] = pre[2];
    small[kSlotHubs] = pre[3];
  }
}

// ---- the sampler -----------------------------------------------------------

struct EmitCtx {
  const int64_t *indices;
  uint8_t *src_reached;
  uint32_t *src_rbits;  // non-NULL: the hop marks reached bits instead of bytes
  int64_t *src_gid;
  int64_t *eid;
  int32_t *dst_local;
  int32_t dst;
};

__device__ __forceinline__ EmitCtx make_ctx(const EtypeStatic &E, int64_t *src_gid,
                                            int64_t *eid, int32_t *dst_local,
                                            int64_t dst, bool bits) {
  return EmitCtx{E.indices, E.src_reached, bits ? E.src_rbits : nullptr, src_gid, eid,
                 dst_local, int32_t(dst)};
}

// Marks source g reached: in bit mode an atomic OR whose result is not used,
// skipped when the bit is already seen; otherwise a plain byte store.  A
// popular source (a hub of the forward edge type, seen through its reverse)
// is reached by many lanes of many wavefronts, and atomics on one word queue
// one behind the other in its L2 channel; reading first lets all but the
// first few pass by (a stale read only costs a redundant atomic).  Plain byte
// stores do not wait on each other, and reading first would cost them a load.
__device__ __forceinline__ void mark_reached(uint8_t *bytes, uint32_t *bits, int64_t g) {
  if (bits) {
    const uint32_t m = 1u << (g & 31);
    if ((bits[g >> 5] & m) == 0) atomicOr(bits + (g >> 5), m);
  } else {
    bytes[g] = 1;
  }
}

// Writes kept edge `e` at output slot `pos`; its source is reached.
__device__ __forceinline__ void emit_edge(const EmitCtx &c, int64_t pos,
                                          int64_t e) {
  const int64_t g = c.indices[e];
  c.src_gid[pos] = g;
  c.eid[pos] = e;
  c.dst_local[pos] = c.dst;
  mark_reached(c.src_reached, c.src_rbits, g);
}

// Keys of the four edges 4g .. 4g+3 (g < 2^30: edge IDs are below 2^32).
__device__ __forceinline__ U32x4 edge_keys(const PhiloxLine &L, uint64_t g,
                                           uint32_t shift) {
  U32x4 r = philox_keys(L, uint32_t(g));
  r.x >>= shift;
  r.y >>= shift;
  r.z >>= shift;
  r.w >>= shift;
  return r;
}

__device__ __forceinline__ uint32_t word_of(const U32x4 &r, int w) {
  return w == 0 ? r.x : (w == 1 ? r.y : (w == 2 ? r.z : r.w));
}

// Keys are uniform, so about deg * tau / 2^bits of them fall below tau; tau is
// set for K + 4 sqrt(K) + 16 expected candidates.  A pure function of
// (K, deg, bits), so every chunk of a hub uses the same value.
__device__ __forceinline__ uint64_t cand_threshold(int64_t K, int64_t deg,
                                                   uint64_t key_space) {
  uint64_t tau = uint64_t(ceil((double(K) + 4.0 * sqrt(double(K)) + 16.0) /
                               double(deg) * double(key_space)));
  if (tau < 1) tau = 1;
  if (tau > key_space) tau = key_space;
  return tau;
}

// The rule on one pair when the candidates could not decide it (too few or
// too many): bisect the composite (key << 32 | j), j = eid - lo, for the K-th
// smallest value T within [a, b], then keep every edge with composite <= T,
// in edge order.  One wavefront; exact.
__device__ void select_by_bisection(const EmitCtx &c, int64_t lo, int64_t deg,
                                    int64_t K, int64_t o, uint64_t a,
                                    uint64_t b, const PhiloxLine &L, uint32_t shift,
                                    const ExclView &X, int xe, bool excl) {
  const int lane = lane_id();
  const uint64_t g_first = uint64_t(lo) >> 2;
  const uint64_t g_last = uint64_t(lo + deg - 1) >> 2;
  const uint64_t hi = uint64_t(lo + deg);
  while (a < b) {
    const uint64_t mid = a + ((b - a) >> 1);
    int64_t le = 0;
    for (uint64_t gb = g_first; gb <= g_last; gb += kWave) {
      const uint64_t g = gb + lane;
      if (g > g_last) continue;
      const U32x4 r = edge_keys(L, g, shift);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint64_t ed = 4 * g + w;
        if (ed >= uint64_t(lo) && ed < hi &&
            ((uint64_t(word_of(r, w)) << 32) | (ed - uint64_t(lo))) <= mid &&
            !(excl && is_excluded(X, xe, ed)))
          ++le;
      }
    }
    le = wave_sum_i64(le);
    if (le >= K)
      b = mid;
    else
      a = mid + 1;
  }
  const uint64_t T = a;
  int64_t emitted = 0;
  for (uint64_t gb = g_first; gb <= g_last; gb += kWave) {
    const uint64_t g = gb + lane;
    int mask = 0;
    if (g <= g_last) {
      const U32x4 r = edge_keys(L, g, shift);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint64_t ed = 4 * g + w;
        if (ed >= uint64_t(lo) && ed < hi &&
            ((uint64_t(word_of(r, w)) << 32) | (ed - uint64_t(lo))) <= T &&
            !(excl && is_excluded(X, xe, ed)))
          mask |= 1 << w;
      }
    }
    int tot;
    int64_t pos = o + emitted + wave_prefix_small(__popc(mask), &tot);
#pragma unroll
    for (int w = 0; w < 4; ++w)
      if (mask & (1 << w)) emit_edge(c, pos++, int64_t(4 * g + w));
    emitted += tot;
  }
}

// Bisection bounds that the candidate count already implies.
__device__ __forceinline__ void bisection_bounds(int64_t n_cand, int64_t K,
                                                 uint64_t tau, uint64_t key_space,
                                                 int64_t deg, uint64_t *a,
                                                 uint64_t *b) {
  *a = 0;
  *b = ((key_space - 1) << 32) | uint64_t(deg - 1);
  if (tau < key_space) {
    if (n_cand >= K)
      *b = min(*b, (tau << 32) - 1);  // the K smallest all have key < tau
    else
      *a = tau << 32;  // fewer than K keys below tau
  }
}

constexpr int kSampleWaves = 4;
constexpr int kSampleThreads = kSampleWaves * kWave;

struct SampleArgs {
  HopView hv;
  const EtypeStatic *es;
  int32_t n_etypes, n_types;
  int64_t n_pairs, n_wave, n_chunks, n_hubs;
  int64_t blocks_a, blocks_b, blocks_c;
  int64_t chunks_per_wave;
  PairArrays pa;
  uint64_t *cand;
  const int64_t *small;
  // edge type e of this launch is copy e / key_R of the graph's edge type
  // e % key_R (a mini-batch of a bundle); its key uses that type index and the
  // copy's sampling seed sigmas[e / key_R]
  const uint64_t *sigmas;
  int32_t key_R;
  int32_t hop, key_bits;
  bool bits;  // the hop marks reached bits (bit mode) instead of bytes
  bool xcd;   // blocks ordered per XCD (xcd_block)
  int64_t *src_gid, *eid;
  int32_t *dst_local;
  int64_t *indptr_all;
  // block 0 stores the hop's source-list pointers into the hop's table (read
  // only by later launches)
  int64_t **src_out_slot;
  int64_t *src_out_new[kInlineSrcOut];
  int32_t n_src_out;
  ExclView X;
};

// Philox key words and counter edge type of (virtual) edge type e.
struct KeyCtx {
  uint32_t k0, k1;
  int32_t ke;
};
__device__ __forceinline__ KeyCtx key_ctx(const SampleArgs &A, int e) {
  const int b = e / A.key_R;
  const uint64_t s = A.sigmas[b];
  return KeyCtx{uint32_t(s), uint32_t(s >> 32), e - b * A.key_R};
}

// Role A: a wavefront per 64 consecutive pairs.  Each lane writes its pair's
// block-CSC entry; a lane whose pair selects K of at most kLaneSelect in-edges
// (nothing excluded) ranks their keys in registers.  Then the wavefront writes
// the kept edges of the small take-all pairs and of those small selections,
// one output slot per lane and kGroupSlots slots per lane at a time (their
// source loads are issued together, before any store), so that neighbouring
// lanes write neighbouring slots.  The first block of this role also writes
// each etype's closing CSC entry.
struct GroupLds {
  int64_t start[kWave];        // first output slot of the pair
  int64_t lo[kWave];           // first in-edge slot
  const int64_t *src[kWave];   // the pair's in-edge sources (indices + lo)
  uint8_t *reached[kWave];     // reached flags of its source type
  uint32_t *rbits[kWave];      // or its reached bits (bit mode)
  // a small selection's kept in-edges, ascending: nibble k is the in-edge
  // (offset from lo) of its output slot k; 0 for a take-all pair, whose slot k
  // is in-edge k (a selection that keeps only in-edge 0 is 0 as well, and
  // means the same)
  uint64_t pick[kWave];
  int32_t tpre[kWave + 1];     // prefix of take-all slots over the group
  int32_t dst[kWave];
};

// The K smallest (key, j) of the deg <= kLaneSelect in-edges lo .. lo+deg-1 of
// one pair, for one lane: their offsets j, ascending, packed 4 bits each.
__device__ uint64_t lane_select(const SampleArgs &A, int e, int64_t lo, int deg, int K) {
  static_assert(kLaneSelect == 16, "the unrolled loops cover 16 in-edges");
  const int b = e / A.key_R;
  const uint64_t sig = A.sigmas[b];
  const uint32_t k0 = uint32_t(sig), k1 = uint32_t(sig >> 32), ke = uint32_t(e - b * A.key_R);
  const uint32_t shift = uint32_t(32 - A.key_bits);
  // key groups g0 .. g0+4 hold the in-edges, from word lo & 3
  const uint64_t g0 = uint64_t(lo) >> 2;
  uint32_t w[20];
#pragma unroll
  for (int q = 0; q < 5; ++q) {
    U32x4 r{0, 0, 0, 0};
    if (4 * (g0 + q) < uint64_t(lo + deg))
      r = philox4x32_10(U32x4{uint32_t(g0 + q), uint32_t((g0 + q) >> 32), uint32_t(A.hop), ke},
                        k0, k1);
    w[4 * q] = r.x;
    w[4 * q + 1] = r.y;
    w[4 * q + 2] = r.z;
    w[4 * q + 3] = r.w;
  }
  uint32_t key[16];
  switch (int(lo & 3)) {  // constant register indices in every branch
    case 0:
#pragma unroll
      for (int j = 0; j < 16; ++j) key[j] = w[j] >> shift;
      break;
    case 1:
#pragma unroll
      for (int j = 0; j < 16; ++j) key[j] = w[j + 1] >> shift;
      break;
    case 2:
#pragma unroll
      for (int j = 0; j < 16; ++j) key[j] = w[j + 2] >> shift;
      break;
    default:
#pragma unroll
      for (int j = 0; j < 16; ++j) key[j] = w[j + 3] >> shift;
      break;
  }
  // in-edge j is kept when fewer than K in-edges have a smaller (key, j)
  uint64_t pick = 0;
  int n = 0;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    int rank = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i)
      rank += (i < deg && (key[i] < key[j] || (key[i] == key[j] && i < j))) ? 1 : 0;
    if (j < deg && rank < K) {
      pick |= uint64_t(j) << (4 * n);
      ++n;
    }
  }
  return pick;
}
constexpr int kGroupSlots = 4;

__device__ void role_pair_groups(const SampleArgs &A, GroupLds &L, int64_t group,
                                 bool first_block) {
  const int lane = lane_id();
  const int64_t *ebase = A.small + kSlotNew + A.n_types;
  const int64_t *pb = A.hv.pair_base;
  if (first_block)
    for (int e = threadIdx.x; e < A.n_etypes; e += kSampleThreads)
      A.indptr_all[pb[e + 1] + e] = ebase[e + 1] - ebase[e];
  const int64_t p = group * kWave + lane;
  int take = 0;
  if (p < A.n_pairs) {
    const int e = A.pa.pet[p];
    const int64_t i = p - pb[e];
    const int64_t o = A.pa.off[p];
    A.indptr_all[pb[e] + e + i] = o - ebase[e];
    const int64_t s = A.pa.off[p + 1] - o;
    const int64_t deg = s > 0 ? A.pa.pdeg[p] : 0;
    uint64_t pick = 0;
    if (s > 0 && s == deg && s <= kThreadTakeAll) {
      take = int(s);  // every in-edge
    } else if (s > 0 && s < deg && deg <= kLaneSelect && excl_count(A.X, e, i) == 0) {
      take = int(s);  // K of at most kLaneSelect in-edges
      pick = lane_select(A, e, A.pa.plo[p], int(deg), int(s));
    }
    if (take) {
      const int64_t lo = A.pa.plo[p];
      L.start[lane] = o;
      L.lo[lane] = lo;
      L.src[lane] = A.es[e].indices + lo;
      L.reached[lane] = A.es[e].src_reached;
      L.rbits[lane] = A.bits ? A.es[e].src_rbits : nullptr;
      L.pick[lane] = pick;
      L.dst[lane] = int32_t(i);
    }
  }
  int total;
  // exclusive prefix of the take-all slot counts over the lanes
  const int64_t inc = wave_incl_scan_i64(take);
  L.tpre[lane] = int32_t(inc - take);
  total = __shfl(int(inc), kWave - 1, kWave);
  if (lane == kWave - 1) L.tpre[kWave] = total;
  wave_sync();
  for (int t0 = 0; t0 < total; t0 += kWave * kGroupSlots) {
    // the lanes q[u] whose take-all ranges hold slots t0 + u * 64 + lane
    int q[kGroupSlots], k[kGroupSlots];
#pragma unroll
    for (int u = 0; u < kGroupSlots; ++u) {
      const int t = t0 + u * kWave + lane;
      q[u] = -1;
      k[u] = 0;
      if (t < total) {
        int a = 0, b = kWave;
        while (b - a > 1) {
          const int m = (a + b) >> 1;
          if (L.tpre[m] <= t)
            a = m;
          else
            b = m;
        }
        q[u] = a;
        k[u] = t - L.tpre[a];
        // a small selection's slot k holds its k-th kept in-edge
        if (L.pick[a]) k[u] = int((L.pick[a] >> (4 * k[u])) & 15);
      }
    }
    int64_t g[kGroupSlots];
#pragma unroll
    for (int u = 0; u < kGroupSlots; ++u) g[u] = q[u] >= 0 ? L.src[q[u]][k[u]] : 0;
#pragma unroll
    for (int u = 0; u < kGroupSlots; ++u) {
      if (q[u] < 0) continue;
      const int64_t pos = L.start[q[u]] + (t0 + u * kWave + lane - L.tpre[q[u]]);
      A.src_gid[pos] = g[u];
      A.eid[pos] = L.lo[q[u]] + k[u];
      A.dst_local[pos] = L.dst[q[u]];
      mark_reached(L.reached[q[u]], L.rbits[q[u]], g[u]);
    }
  }
}

// Role B: a wavefront per kWavePairs pairs (large take-all, or selection
// among at most kHubChunk edges with the candidate list in LDS), one after
// the other; what every pair needs is loaded for all of them first, so the
// wavefront waits on those loads once.
constexpr int kWavePairs = 2;

struct WavePair {
  EmitCtx c;
  KeyCtx kc;
  int64_t lo, deg, o, s;
  int32_t nx;
  int e;
};

__device__ __forceinline__ WavePair wave_pair(const SampleArgs &A, int64_t p) {
  WavePair P;
  P.e = A.pa.pet[p];
  const int64_t i = p - A.hv.pair_base[P.e];
  P.c = make_ctx(A.es[P.e], A.src_gid, A.eid, A.dst_local, i, A.bits);
  P.kc = key_ctx(A, P.e);
  P.lo = A.pa.plo[p];
  P.deg = A.pa.pdeg[p];
  P.o = A.pa.off[p];
  P.s = A.pa.off[p + 1] - P.o;
  P.nx = excl_count(A.X, P.e, i);
  return P;
}

__device__ void wave_pair_run(const SampleArgs &A, uint32_t *ck, uint32_t *cj,
                              const WavePair &P) {
  const int lane = lane_id();
  const int e = P.e;
  const EmitCtx &c = P.c;
  const int64_t lo = P.lo, deg = P.deg, o = P.o, s = P.s;
  const int32_t nx = P.nx;
  if (s == deg) {  // every in-edge is kept
    for (int64_t j = lane; j < deg; j += kWave) emit_edge(c, o + j, lo + j);
    return;
  }
  if (nx > 0 && s == deg - nx) {  // every in-edge but the excluded ones
    int64_t emitted = 0;
    for (int64_t j0 = 0; j0 < deg; j0 += kWave) {
      const int64_t j = j0 + lane;
      const bool keep = j < deg && !is_excluded(A.X, e, uint64_t(lo + j));
      const uint64_t bal = __ballot(keep);
      if (keep) emit_edge(c, o + emitted + __popcll(bal & lanes_below()), lo + j);
      emitted += __popcll(bal);
    }
    return;
  }
  const int64_t K = s;
  const uint32_t shift = uint32_t(32 - A.key_bits);
  const uint64_t key_space = uint64_t(1) << A.key_bits;
  const KeyCtx kc = P.kc;
  const PhiloxLine L = philox_line(kc.k0, kc.k1, uint32_t(A.hop), uint32_t(kc.ke));
  const uint64_t g_first = uint64_t(lo) >> 2;
  const uint64_t g_last = uint64_t(lo + deg - 1) >> 2;
  const uint64_t hi = uint64_t(lo + deg);

  // candidates (key < tau), appended in edge order
  const uint64_t tau = cand_threshold(K, deg, key_space);
  int64_t n_cand = 0;
  for (uint64_t gb = g_first; gb <= g_last; gb += kWave) {
    const uint64_t g = gb + lane;
    int mask = 0;
    U32x4 r{0, 0, 0, 0};
    if (g <= g_last) {
      r = edge_keys(L, g, shift);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint64_t ed = 4 * g + q;
        if (ed >= uint64_t(lo) && ed < hi && uint64_t(word_of(r, q)) < tau &&
            !(nx > 0 && is_excluded(A.X, e, ed)))
          mask |= 1 << q;
      }
    }
    int tot;
    int64_t pos = n_cand + wave_prefix_small(__popc(mask), &tot);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (mask & (1 << q)) {
        if (pos < kCandCap) {
          ck[pos] = word_of(r, q);
          cj[pos] = uint32_t(4 * g + q - uint64_t(lo));
        }
        ++pos;
      }
    }
    n_cand += tot;
  }
  wave_sync();

  if (n_cand >= K && n_cand <= kCandCap) {
    // rank each candidate by counting smaller (key, j); keep ranks < K, in
    // list (= edge) order
    const int nc = int(n_cand);
    int64_t emitted = 0;
    for (int q0 = 0; q0 < nc; q0 += kWave) {
      const int q = q0 + lane;
      bool sel = false;
      uint32_t jq = 0;
      if (q < nc) {
        jq = cj[q];
        const uint64_t me = (uint64_t(ck[q]) << 32) | jq;
        int rank = 0;
        for (int t = 0; t < nc; ++t)
          rank += ((uint64_t(ck[t]) << 32) | cj[t]) < me ? 1 : 0;
        sel = rank < K;
      }
      const uint64_t bal = __ballot(sel);
      if (sel) emit_edge(c, o + emitted + __popcll(bal & lanes_below()), lo + jq);
      emitted += __popcll(bal);
    }
    return;
  }
  uint64_t a, b;
  bisection_bounds(n_cand, K, tau, key_space, deg, &a, &b);
  select_by_bisection(c, lo, deg, K, o, a, b, L, shift, A.X, e, nx > 0);
}

__device__ void role_wave_pairs(const SampleArgs &A, uint32_t *ck, uint32_t *cj,
                                int64_t w) {
  WavePair P[kWavePairs];
  int n = 0;
#pragma unroll
  for (int k = 0; k < kWavePairs; ++k) {
    const int64_t x = w * kWavePairs + k;
    if (x < A.n_wave) {
      P[k] = wave_pair(A, A.pa.wlist[x]);
      n = k + 1;
    }
  }
#pragma unroll
  for (int k = 0; k < kWavePairs; ++k) {
    if (k < n) {
      if (k > 0) wave_sync();  // the previous pair's candidate reads are done
      wave_pair_run(A, ck, cj, P[k]);
    }
  }
}

// Role C: wavefront w takes the hub chunks [w * chunks_per_wave, ...) in
// order and appends each chunk's candidates (key < tau) to its hub's list.
// The hub of the first chunk is found by a wavefront-wide search (the last
// hub whose first chunk is not above it); later chunks walk on from there, so
// the search and the hub's parameters are loaded once per run of chunks.
constexpr int64_t kHubWaves = 16384;
constexpr int64_t kMaxChunksPerWave = 16;

struct HubParams {
  int64_t hub, first_chunk, end_chunk, lo, deg, K, o, dst;
  uint64_t tau;
  int e;
  int32_t nx;  // excluded in-edges
  KeyCtx kc;
  PhiloxLine L;
  // every in-edge is kept: chunks are copied to output slots o + (j - lo)
  __device__ bool take_all() const { return K == deg; }
};

// A value that is the same on every lane, in a scalar register.
__device__ __forceinline__ int64_t uniform64(int64_t x) {
  const uint64_t u = uint64_t(x);
  return int64_t(uint64_t(__builtin_amdgcn_readfirstlane(uint32_t(u))) |
                 (uint64_t(__builtin_amdgcn_readfirstlane(uint32_t(u >> 32))) << 32));
}

// A copy of x in a vector register.  The key loop of the hub role reads its
// round keys from vector registers: uniform as they are, in scalar registers
// they outnumber what the role has left, and the compiler would then fetch
// some of them back from vector lanes on every step.
__device__ __forceinline__ uint32_t in_vgpr(uint32_t x) {
  uint32_t y = x;
  asm("" : "+v"(y));
  return y;
}
__device__ __forceinline__ PhiloxLine vgpr_line(PhiloxLine L) {
  L.ek1 = in_vgpr(L.ek1);
  L.x1k0 = in_vgpr(L.x1k0);
  L.hk1 = in_vgpr(L.hk1);
  L.x3k1 = in_vgpr(L.x3k1);
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    L.k0[r] = in_vgpr(L.k0[r]);
    L.k1[r] = in_vgpr(L.k1[r]);
  }
  return L;
}

// A hub's parameters; the same on every lane of the wavefront (scalar
// registers, so that the key loop keeps its vector registers to itself).
__device__ HubParams hub_params(const SampleArgs &A, int64_t hub) {
  HubParams H;
  H.hub = uniform64(hub);
  H.first_chunk = uniform64(A.pa.hub_choff[hub]);
  H.end_chunk = uniform64(hub + 1 < A.n_hubs ? A.pa.hub_choff[hub + 1] : A.n_chunks);
  const int64_t p = uniform64(A.pa.hub_pair[hub]);
  H.e = int(__builtin_amdgcn_readfirstlane(uint32_t(A.pa.pet[p])));
  H.kc = key_ctx(A, H.e);
  H.L = vgpr_line(philox_line(H.kc.k0, H.kc.k1, uint32_t(A.hop), uint32_t(H.kc.ke)));
  H.lo = uniform64(A.pa.plo[p]);
  H.deg = uniform64(A.pa.pdeg[p]);
  H.o = uniform64(A.pa.off[p]);
  H.K = uniform64(A.pa.off[p + 1]) - H.o;
  H.dst = uniform64(p - A.hv.pair_base[H.e]);
  H.tau = uint64_t(uniform64(int64_t(cand_threshold(H.K, H.deg, uint64_t(1) << A.key_bits))));
  H.nx = int32_t(__builtin_amdgcn_readfirstlane(
      uint32_t(excl_count(A.X, H.e, p - A.hv.pair_base[H.e]))));
  return H;
}

// A wavefront's candidates for its current hub wait in LDS (kHubBuf
// entries) and go to the hub's global list in one piece, with one atomic
// for their positions, when the wavefront moves to the next hub, when the
// buffer is full, and at the end: one round trip per (wavefront, hub) instead
// of one per step that finds candidates.
constexpr int kHubBuf = kCandCap;  // uint64 entries: a wavefront's two candidate arrays
struct HubBuf {
  uint64_t *e;  // LDS
  int n;        // entries held (the same on every lane)
};

__device__ void hub_flush(const SampleArgs &A, int64_t hub, HubBuf &B) {
  if (B.n == 0) return;
  wave_sync();
  int base = 0;
  if (lane_id() == 0) base = atomicAdd(A.pa.hub_cnt + hub, B.n);
  base = __shfl(base, 0, kWave);
  uint64_t *list = A.cand + hub * kCandCap;
  for (int i = lane_id(); i < B.n; i += kWave)
    if (base + i < kCandCap) list[base + i] = B.e[i];
  wave_sync();
  B.n = 0;
}

// One wavefront step over the 64 key groups gb .. gb+63 (wave-uniform gb;
// group g holds edges 4g .. 4g+3, g < 2^30) of a hub's edge range
// [c_lo, c_hi): appends the edges with key <= lim to the hub's candidates.
// kChecked: some lanes' edges may lie outside the range.  Otherwise the step
// first asks whether any key of the wavefront is small enough at all, which
// is rarely the case.
template <bool kChecked>
__device__ __forceinline__ void hub_step(const SampleArgs &A, const HubParams &H,
                                         uint32_t gb, int64_t c_lo, int64_t c_hi,
                                         uint32_t lim, uint32_t shift, uint32_t m0v,
                                         HubBuf &B) {
  const int lane = lane_id();
  const uint32_t g = gb + uint32_t(lane);
  // round 0's product M0 * (gb + lane) as one multiply-add: M0 (m0v, in a
  // vector register) * lane plus the wavefront's M0 * gb (scalar registers),
  // so the step needs no add for g
  const U32x4 r = philox_keys_p0(H.L, uint64_t(m0v) * uint32_t(lane) + uint64_t(0xD2511F53u) * gb);
  if (!kChecked) {
    const uint32_t m = min(min(r.x, r.y), min(r.z, r.w));
    if (__ballot(m <= lim) == 0) return;
  }
  int mask = (r.x <= lim ? 1 : 0) | (r.y <= lim ? 2 : 0) | (r.z <= lim ? 4 : 0) |
             (r.w <= lim ? 8 : 0);
  if (kChecked) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint64_t ed = 4 * uint64_t(g) + q;
      if (ed < uint64_t(c_lo) || ed >= uint64_t(c_hi)) mask &= ~(1 << q);
    }
    if (__ballot(mask != 0) == 0) return;
  }
  if (H.nx > 0) {  // excluded edges are never candidates
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if ((mask & (1 << q)) && is_excluded(A.X, H.e, 4 * uint64_t(g) + q)) mask &= ~(1 << q);
  }
  int tot;
  const int pre = wave_prefix_small(__popc(mask), &tot);
  if (B.n + tot > kHubBuf) hub_flush(A, H.hub, B);  // tot <= 256 < kHubBuf
  int pos = B.n + pre;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if (mask & (1 << q)) {
      B.e[pos] = (uint64_t(word_of(r, q) >> shift) << 32) | (4 * uint64_t(g) + q - uint64_t(H.lo));
      ++pos;
    }
  }
  B.n += tot;
}

// The last hub whose first chunk is not above chunk c (hub_choff strictly
// increases from hub_choff[0] == 0).  A 64-ary search: every lane probes one
// position per round, so the wavefront finds the hub in a few dependent loads
// instead of one per halving.  All lanes of the wavefront must take part.
__device__ int64_t find_hub(const SampleArgs &A, int64_t c) {
  const int lane = lane_id();
  int64_t lo = 0, hi = A.n_hubs;  // hub_choff[lo] <= c, and c < hub_choff[hi] (or hi = n_hubs)
  while (hi - lo > 1) {
    const int64_t step = (hi - lo + kWave - 1) / kWave;
    const int64_t pos = lo + int64_t(lane) * step;
    const bool le = pos < hi && A.pa.hub_choff[pos] <= c;
    // true on a prefix of the lanes, lane 0 always (its position is lo)
    const uint64_t bal = __ballot(le);
    const int last = 63 - __clzll((unsigned long long)bal);
    lo += int64_t(last) * step;
    hi = min(hi, lo + step);
  }
  return lo;
}

__device__ void role_hub_chunks(const SampleArgs &A, int64_t w, uint64_t *buf) {
  const int64_t c_first = w * A.chunks_per_wave;
  const int64_t c_end = min(c_first + A.chunks_per_wave, A.n_chunks);
  HubParams H = hub_params(A, find_hub(A, c_first));
  const uint32_t shift = uint32_t(32 - A.key_bits);
  HubBuf B{buf, 0};
  for (int64_t chunk = c_first; chunk < c_end;) {
    while (chunk >= H.end_chunk) {
      hub_flush(A, H.hub, B);
      H = hub_params(A, H.hub + 1);
    }
    // this wavefront's chunks of the hub are one contiguous range of in-edges
    const int64_t run_end = min(c_end, H.end_chunk);
    const int64_t r_lo = H.lo + (chunk - H.first_chunk) * kHubChunk;
    const int64_t r_hi = min(H.lo + (run_end - H.first_chunk) * kHubChunk, H.lo + H.deg);
    chunk = run_end;
    if (H.take_all()) {
      const EmitCtx c = make_ctx(A.es[H.e], A.src_gid, A.eid, A.dst_local, H.dst, A.bits);
      for (int64_t j = r_lo + lane_id(); j < r_hi; j += kWave) emit_edge(c, H.o + (j - H.lo), j);
      continue;
    }
    // (key >> shift) < tau  <=>  key < tau << shift  <=>  key <= lim
    const uint64_t tau_raw = H.tau << shift;
    const uint32_t lim = tau_raw - 1 >= 0xFFFFFFFFull ? 0xFFFFFFFFu : uint32_t(tau_raw - 1);
    // steps over the key groups g_first .. g_last, 64 at a time; a step whose
    // groups all lie inside the range (g_first <= ... < g_in_end) needs no
    // bounds, so only a partial first and the last steps are checked
    // (wavefront-uniform: scalar registers, so that the loop below is
    // counted and branched on by the scalar unit)
    const uint32_t g_first = __builtin_amdgcn_readfirstlane(uint32_t(uint64_t(r_lo) >> 2));
    const uint32_t g_last = __builtin_amdgcn_readfirstlane(uint32_t(uint64_t(r_hi - 1) >> 2));
    const uint32_t g_in_end = __builtin_amdgcn_readfirstlane(uint32_t(uint64_t(r_hi) >> 2));
    const uint32_t m0v = in_vgpr(0xD2511F53u);
    uint32_t gb = g_first;
    if (4 * uint64_t(gb) < uint64_t(r_lo)) {
      hub_step<true>(A, H, gb, r_lo, r_hi, lim, shift, m0v, B);
      gb += kWave;
    }
    for (; gb + kWave <= g_in_end; gb += kWave)
      hub_step<false>(A, H, gb, r_lo, r_hi, lim, shift, m0v, B);
    for (; gb <= g_last; gb += kWave) hub_step<true>(A, H, gb, r_lo, r_hi, lim, shift, m0v, B);
  }
  hub_flush(A, H.hub, B);
}

// A wavefront per hub: the K smallest (key, j) of the hub's candidate list,
// written in edge order.  The list holds every edge with key < tau, so when
// it has at least K entries they include the K smallest.
__global__ __launch_bounds__(kSampleThreads) void k_hub_finish(SampleArgs A) {
  __shared__ uint32_t s_key[kSampleWaves][kCandCap];
  __shared__ uint32_t s_j[kSampleWaves][kCandCap];
  __shared__ uint8_t s_sel[kSampleWaves][kCandCap];
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int64_t hub = xcd_block(blockIdx.x, gridDim.x, A.xcd) * kSampleWaves + wave;
  if (hub >= A.n_hubs) return;
  uint32_t *ck = s_key[wave];
  uint32_t *cj = s_j[wave];
  uint8_t *sel = s_sel[wave];
  const int64_t p = A.pa.hub_pair[hub];
  const int e = A.pa.pet[p];
  const int64_t lo = A.pa.plo[p];
  const int64_t deg = A.pa.pdeg[p];
  const int64_t o = A.pa.off[p];
  const int64_t K = A.pa.off[p + 1] - o;
  if (K == deg) return;  // a take-all hub: its chunks wrote every edge
  const uint32_t shift = uint32_t(32 - A.key_bits);
  const uint64_t key_space = uint64_t(1) << A.key_bits;
  const KeyCtx kc = key_ctx(A, e);
  const uint64_t tau = cand_threshold(K, deg, key_space);
  const EmitCtx c = make_ctx(A.es[e], A.src_gid, A.eid, A.dst_local,
                             p - A.hv.pair_base[e], A.bits);
  const int64_t n_cand = A.pa.hub_cnt[hub];
  if (n_cand >= K && n_cand <= kCandCap) {
    const uint64_t *list = A.cand + hub * kCandCap;
    const int nc = int(n_cand);
    for (int q = lane; q < nc; q += kWave) {
      const uint64_t v = list[q];
      ck[q] = uint32_t(v >> 32);
      cj[q] = uint32_t(v);
    }
    wave_sync();
    // rank by (key, j): the K smallest are kept
    for (int q = lane; q < nc; q += kWave) {
      const uint64_t me = (uint64_t(ck[q]) << 32) | cj[q];
      int rank = 0;
      for (int t = 0; t < nc; ++t) rank += ((uint64_t(ck[t]) << 32) | cj[t]) < me ? 1 : 0;
      sel[q] = rank < K ? 1 : 0;
    }
    wave_sync();
    // output position = kept candidates with a smaller edge ID (below K
    // while the list holds each edge once; a position past the pair's K
    // slots is reported rather than written)
    for (int q = lane; q < nc; q += kWave) {
      if (!sel[q]) continue;
      const uint32_t jq = cj[q];
      int pos = 0;
      for (int t = 0; t < nc; ++t) pos += (sel[t] && cj[t] < jq) ? 1 : 0;
      if (pos < K)
        emit_edge(c, o + pos, lo + jq);
      else
        atomicOr(reinterpret_cast<int32_t *>(const_cast<int64_t *>(A.small) + kSlotErr), kErrBound);
    }
    return;
  }
  uint64_t a, b;
  bisection_bounds(n_cand, K, tau, key_space, deg, &a, &b);
  const int32_t nx = excl_count(A.X, e, p - A.hv.pair_base[e]);
  select_by_bisection(c, lo, deg, K, o, a, b,
                      philox_line(kc.k0, kc.k1, uint32_t(A.hop), uint32_t(kc.ke)), shift, A.X,
                      e, nx > 0);
}

__global__ __launch_bounds__(kSampleThreads) void k_sample(SampleArgs A) {
  // per wavefront: its candidate keys and edge offsets (or a GroupLds)
  __shared__ __align__(16) uint32_t s_cand[kSampleWaves][2][kCandCap];
  static_assert(sizeof(GroupLds) <= sizeof(s_cand[0]), "a group's table fits a wavefront's LDS");
  const int64_t b = blockIdx.x;
  // the same on every lane: what depends on it stays in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x) / kWave);
  if (b == 0 && int(threadIdx.x) < A.n_src_out)
    A.src_out_slot[threadIdx.x] = A.src_out_new[threadIdx.x];
  // the longest wavefronts first: groups of small take-all pairs (a
  // wavefront per 64 pairs), then hub chunks, then wavefront pairs, so that
  // short wavefronts fill in behind long ones
  // Roles A and C share the first blocks_a + blocks_c blocks.  Ordered per
  // XCD, each role keeps its own range (its block count a multiple of kXcds,
  // xcd_block); otherwise role A's blocks are spread evenly among role C's, so
  // that the pair groups' memory waits overlap the hub chunks' key work:
  // block x of the shared range is role A's block f(x) when f(x + 1) > f(x),
  // with f(x) = floor(x blocks_a / (blocks_a + blocks_c)), else role C's
  // block x - f(x).
  const int64_t n_ac = A.blocks_a + A.blocks_c;
  int64_t ra = -1, rc = -1;
  if (b < n_ac) {
    if (A.xcd) {
      if (b < A.blocks_a)
        ra = xcd_block(b, A.blocks_a, true);
      else
        rc = xcd_block(b - A.blocks_a, A.blocks_c, true);
    } else {
      const int64_t f0 = b * A.blocks_a / n_ac, f1 = (b + 1) * A.blocks_a / n_ac;
      if (f1 > f0)
        ra = f0;
      else
        rc = b - f0;
    }
  }
  if (ra >= 0) {
    // the candidate lists are not used by this role: reuse their LDS
    GroupLds *g = reinterpret_cast<GroupLds *>(&s_cand[wave][0][0]);
    role_pair_groups(A, *g, ra * kSampleWaves + wave, ra == 0);
  } else if (rc >= 0) {
    const int64_t w = rc * kSampleWaves + wave;
    if (w * A.chunks_per_wave < A.n_chunks)
      role_hub_chunks(A, w, reinterpret_cast<uint64_t *>(&s_cand[wave][0][0]));
  } else {
    const int64_t w =
        xcd_block(b - A.blocks_a - A.blocks_c, A.blocks_b, A.xcd) * kSampleWaves + wave;
    if (w * kWavePairs < A.n_wave) role_wave_pairs(A, s_cand[wave][0], s_cand[wave][1], w);
  }
}

// ---- small utilities -------------------------------------------------------

__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v) {
  for (int64_t i = grid_stride_start(); i < n; i += grid_stride_step()) p[i] = v;
}
__global__ void k_fill_u32(uint32_t *p, int64_t n, uint32_t v) {
  for (int64_t i = grid_stride_start(); i < n; i += grid_stride_step()) p[i] = v;
}

// dst[0..n) = src[0..n) for 8-byte aligned dst and src, src in pinned host
// memory (read over the host link).
__global__ void k_upload(uint8_t *dst, const uint8_t *src, int64_t n) {
  const int64_t words = n >> 3;
  for (int64_t i = grid_stride_start(); i < words; i += grid_stride_step())
    reinterpret_cast<uint64_t *>(dst)[i] = reinterpret_cast<const uint64_t *>(src)[i];
  if (blockIdx.x == 0 && int64_t(threadIdx.x) < (n & 7))
    dst[words * 8 + threadIdx.x] = src[words * 8 + threadIdx.x];
}

__global__ void k_check_etype(const int64_t *indptr, int64_t n_dst,
                              const int64_t *indices, int64_t nnz,
                              int64_t n_src, int32_t *err) {
  const int64_t i0 = grid_stride_start();
  if (i0 == 0 && (indptr[0] != 0 || indptr[n_dst] != nnz)) atomicOr(err, 1);
  for (int64_t v = i0; v < n_dst; v += grid_stride_step())
    if (indptr[v + 1] < indptr[v]) atomicOr(err, 1);
  for (int64_t j = i0; j < nnz; j += grid_stride_step()) {
    const int64_t x = indices[j];
    if (x < 0 || x >= n_src) atomicOr(err, 1);
  }
}

// One thread per destination vertex: its row of the non-empty mask, from
// the indptr of every edge type into its node type (coalesced across threads).
__global__ void k_nonempty_mask(const int64_t *const *indptrs, int32_t n_etypes, int32_t words,
                                int64_t n, uint32_t *mask) {
  for (int64_t v = grid_stride_start(); v < n; v += grid_stride_step()) {
    uint32_t w = 0;
    for (int32_t k = 0; k < n_etypes; ++k) {
      const int64_t *ip = indptrs[k];
      if (ip[v + 1] > ip[v]) w |= 1u << (k & 31);
      if ((k & 31) == 31 || k == n_etypes - 1) {
        mask[v * words + (k >> 5)] = w;
        w = 0;
      }
    }
  }
}

__global__ void k_philox(const uint32_t *ctr, uint32_t k0, uint32_t k1,
                         int64_t n, uint32_t *out) {
  for (int64_t i = grid_stride_start(); i < n; i += grid_stride_step()) {
    const U32x4 r = philox4x32_10(
        U32x4{ctr[4 * i], ctr[4 * i + 1], ctr[4 * i + 2], ctr[4 * i + 3]}, k0, k1);
    out[4 * i] = r.x;
    out[4 * i + 1] = r.y;
    out[4 * i + 2] = r.z;
    out[4 * i + 3] = r.w;
  }
}

// The sampler's key loop on its own, for measuring its rate: wavefront w takes
// steps w, w + waves, ... of 64 key groups (256 keys) each and evaluates them
// as a hub chunk does (the line-specialised Philox, then one wavefront test
// whether any key is <= lim); it counts the keys <= lim, so that nothing is
// dead code, and adds its count to *count once.
__global__ __launch_bounds__(256) void k_philox_rate(uint32_t k0, uint32_t k1, uint32_t hop,
                                                     uint32_t etype, int64_t n_steps,
                                                     uint32_t lim,
                                                     unsigned long long *count) {
  const PhiloxLine L = philox_line(k0, k1, hop, etype);
  const int lane = lane_id();
  const int64_t waves = int64_t(gridDim.x) * (256 / kWave);
  uint32_t n = 0;
  for (int64_t st = int64_t(blockIdx.x) * (256 / kWave) + threadIdx.x / kWave; st < n_steps;
       st += waves) {
    const U32x4 r = philox_keys(L, uint32_t(st * kWave + lane));
    const uint32_t m = min(min(r.x, r.y), min(r.z, r.w));
    if (__ballot(m <= lim) == 0) continue;
    n += uint32_t(r.x <= lim) + uint32_t(r.y <= lim) + uint32_t(r.z <= lim) +
         uint32_t(r.w <= lim);
  }
  const int64_t total = wave_sum_i64(int64_t(n));
  if (lane == 0 && total) atomicAdd(count, (unsigned long long)total);
}

// ---- host handshake -----------------------------------------------------------

// Copies the n readback slots to host memory, then sets the flag word
// host[n] to `seq`: a host that sees `seq` there reads the slots as they are
// at this point of the stream (every earlier kernel has finished).
__global__ __launch_bounds__(256) void k_publish(int64_t *small, int64_t *host,
                                                 int32_t n, uint64_t seq, bool clear) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) host[i] = small[i];
  __threadfence_system();
  __syncthreads();
  if (threadIdx.x == 0)
    __hip_atomic_store(reinterpret_cast<uint64_t *>(host + n), seq, __ATOMIC_RELEASE,
                       __HIP_MEMORY_SCOPE_SYSTEM);
  // the call is over: its readback slots start the next call at zero (each
  // thread clears the slots it copied)
  if (clear)
    for (int i = threadIdx.x; i < n; i += blockDim.x) small[i] = 0;
}

// dst[i] = v.p[i] for i < n: small tables written in stream order with the
// values carried in the launch itself.
constexpr int kPtrBatch = 16;
struct PtrBatch {
  void *p[kPtrBatch];
};
__global__ void k_store_ptrs(void **dst, PtrBatch v, int32_t n) {
  if (int(threadIdx.x) < n) dst[threadIdx.x] = v.p[threadIdx.x];
}

}  // namespace

// ---- launchers ---------------------------------------------------------------

hipError_t launch_insert_frontier(HopView hv, const TypeStatic *ts,
                                  int32_t n_types, int64_t total, int64_t *small,
                                  hipStream_t stream) {
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_insert_frontier, dim3(grid_for(total, 256)), dim3(256), 0,
                     stream, hv, ts, n_types, total, small);
  return hipGetLastError();
}

int64_t count_tiles(int64_t n_items) {
  const int64_t per_tile = int64_t(kTileThreads) * pair_items(n_items);
  const int64_t t = (n_items + per_tile - 1) / per_tile;
  return t < 1 ? 1 : t;
}

template <bool kStaged, int kItems>
void count_launch(HopView hv, const EtypeStatic *es, int32_t n_etypes, int32_t n_types,
                  int64_t n_items, PairArrays pa, Lookback lb, uint32_t epoch,
                  uint64_t ticket_base, ExclView X, int64_t *small, hipStream_t stream,
                  StageEv ev) {
  const size_t lds = kStaged ? CountTable::bytes(n_etypes) : 0;
  launch_k(k_count_scan<kStaged, kItems>, dim3(unsigned(count_tiles(n_items))),
           dim3(kTileThreads), lds, stream, ev.start, ev.stop, hv, es, n_etypes, n_types,
           n_items, pa, lb, epoch, ticket_base, X, small);
}

hipError_t launch_count_scan(HopView hv, const EtypeStatic *es, int32_t n_etypes,
                             int32_t n_types, int64_t n_items, PairArrays pa,
                             Lookback lb, uint32_t epoch, uint64_t ticket_base,
                             ExclView X, int64_t *small, hipStream_t stream, StageEv ev) {
  const bool staged = n_etypes <= kCountMaxEtypes;
  const bool large = pair_items(n_items) == kPairItemsLarge;
  if (staged && large)
    count_launch<true, kPairItemsLarge>(hv, es, n_etypes, n_types, n_items, pa, lb, epoch,
                                        ticket_base, X, small, stream, ev);
  else if (staged)
    count_launch<true, kPairItemsSmall>(hv, es, n_etypes, n_types, n_items, pa, lb, epoch,
                                        ticket_base, X, small, stream, ev);
  else if (large)
    count_launch<false, kPairItemsLarge>(hv, es, n_etypes, n_types, n_items, pa, lb, epoch,
                                         ticket_base, X, small, stream, ev);
  else
    count_launch<false, kPairItemsSmall>(hv, es, n_etypes, n_types, n_items, pa, lb, epoch,
                                         ticket_base, X, small, stream, ev);
  return hipGetLastError();
}

hipError_t launch_sample(HopView hv, const EtypeStatic *es, int32_t n_etypes,
                         int32_t n_types, int64_t n_pairs, int64_t n_wave,
                         int64_t n_chunks, int64_t n_hubs, PairArrays pa,
                         uint64_t *cand, const int64_t *small, const uint64_t *sigmas,
                         int32_t key_R, int32_t hop, int32_t key_bits, int64_t *src_gid,
                         int64_t *eid, int32_t *dst_local, int64_t *indptr_all,
                         int64_t **src_out_slot, int64_t *const *src_out, int32_t n_src_out,
                         ExclView X, hipStream_t stream, StageEv ev_sample,
                         StageEv ev_select, bool bit_mode, bool xcd_order) {
  if (n_src_out > kInlineSrcOut) return hipErrorInvalidValue;
  SampleArgs A;
  A.X = X;
  A.src_out_slot = src_out_slot;
  A.n_src_out = n_src_out;
  for (int32_t t = 0; t < kInlineSrcOut; ++t) A.src_out_new[t] = t < n_src_out ? src_out[t] : nullptr;
  A.hv = hv;
  A.es = es;
  A.n_etypes = n_etypes;
  A.n_types = n_types;
  A.n_pairs = n_pairs;
  A.n_wave = n_wave;
  A.n_chunks = n_chunks;
  A.n_hubs = n_hubs;
  // role A always has blocks, for the closing CSC entries; every role's block
  // count is rounded up to a multiple of kXcds (its spare blocks find no work)
  A.blocks_a = xcd_round(std::max<int64_t>(1, (n_pairs + kSampleThreads - 1) / kSampleThreads));
  A.blocks_b = xcd_round(((n_wave + kWavePairs - 1) / kWavePairs + kSampleWaves - 1) / kSampleWaves);
  // runs of chunks per wavefront: long enough to amortise finding the hub,
  // short enough to leave about kHubWaves wavefronts for the chip
  A.chunks_per_wave = std::min<int64_t>(kMaxChunksPerWave, std::max<int64_t>(1, n_chunks / kHubWaves));
  const int64_t waves_c = (n_chunks + A.chunks_per_wave - 1) / A.chunks_per_wave;
  const int64_t blocks_c = xcd_round((waves_c + kSampleWaves - 1) / kSampleWaves);
  A.blocks_c = blocks_c;
  A.pa = pa;
  A.cand = cand;
  A.small = small;
  A.sigmas = sigmas;
  A.key_R = key_R > 0 ? key_R : 1;
  A.hop = hop;
  A.key_bits = key_bits;
  A.bits = bit_mode;
  A.xcd = xcd_order;
  A.src_gid = src_gid;
  A.eid = eid;
  A.dst_local = dst_local;
  A.indptr_all = indptr_all;
  const int64_t blocks = A.blocks_a + A.blocks_b + blocks_c;
  launch_k(k_sample, dim3(unsigned(blocks)), dim3(kSampleThreads), 0, stream, ev_sample.start,
           ev_sample.stop, A);
  if (n_hubs > 0) {
    // the hub lists are complete once the first launch has finished
    const int64_t hb = xcd_round((n_hubs + kSampleWaves - 1) / kSampleWaves);
    launch_k(k_hub_finish, dim3(unsigned(hb)), dim3(kSampleThreads), 0, stream,
             ev_select.start, ev_select.stop, A);
  } else if (ev_select.any()) {
    hipError_t e = record_empty_stage(ev_select, stream);
    if (e != hipSuccess) return e;
  }
  return hipGetLastError();
}

hipError_t record_empty_stage(const StageEv &ev, hipStream_t stream) {
  hipError_t e = hipSuccess;
  if (ev.start) e = hipEventRecord(ev.start, stream);
  if (e == hipSuccess && ev.stop) e = hipEventRecord(ev.stop, stream);
  return e;
}

hipError_t launch_publish(int64_t *small, int64_t *host, int32_t n, uint64_t seq, bool clear,
                          hipStream_t stream) {
  hipLaunchKernelGGL(k_publish, dim3(1), dim3(256), 0, stream, small, host, n, seq, clear);
  return hipGetLastError();
}

hipError_t launch_store_ptrs(void **dst, void *const *vals, int32_t n, hipStream_t stream) {
  for (int32_t i = 0; i < n; i += kPtrBatch) {
    PtrBatch v{};
    const int32_t m = n - i < kPtrBatch ? n - i : kPtrBatch;
    for (int32_t k = 0; k < m; ++k) v.p[k] = vals[i + k];
    hipLaunchKernelGGL(k_store_ptrs, dim3(1), dim3(64), 0, stream, dst + i, v, m);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_i32, dim3(grid_for(n, 256, 8192)), dim3(256), 0,
                     stream, p, n, v);
  return hipGetLastError();
}

hipError_t launch_fill_u32(uint32_t *p, int64_t n, uint32_t v, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_u32, dim3(grid_for(n, 256, 8192)), dim3(256), 0,
                     stream, p, n, v);
  return hipGetLastError();
}

hipError_t launch_upload(void *dst, const void *src, int64_t n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  if ((reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src)) & 7)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_upload, dim3(grid_for((n >> 3) + 1, 256, 64)), dim3(256), 0, stream,
                     static_cast<uint8_t *>(dst), static_cast<const uint8_t *>(src), n);
  return hipGetLastError();
}

hipError_t launch_check_etype(const int64_t *indptr, int64_t n_dst,
                              const int64_t *indices, int64_t nnz,
                              int64_t n_src, int32_t *err, hipStream_t stream) {
  const int64_t n = n_dst > nnz ? n_dst : nnz;
  hipLaunchKernelGGL(k_check_etype, dim3(grid_for(n, 256, 8192)), dim3(256), 0,
                     stream, indptr, n_dst, indices, nnz, n_src, err);
  return hipGetLastError();
}

hipError_t launch_nonempty_mask(const int64_t *const *indptrs, int32_t n_etypes, int32_t words,
                                int64_t n, uint32_t *mask, hipStream_t stream) {
  if (n <= 0 || n_etypes <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_nonempty_mask, dim3(grid_for(n, 256, 16384)), dim3(256), 0, stream,
                     indptrs, n_etypes, words, n, mask);
  return hipGetLastError();
}

hipError_t launch_philox_rate(uint64_t key, int32_t hop, int32_t etype, int64_t n_groups,
                              uint32_t lim, uint64_t *count, hipEvent_t start,
                              hipEvent_t stop, hipStream_t stream) {
  const int64_t steps = n_groups / kWave;
  // as many wavefronts as the hub role launches at most
  const unsigned blocks = unsigned(std::min<int64_t>(std::max<int64_t>(steps / 4, 1), 4096));
  hipExtLaunchKernelGGL(k_philox_rate, dim3(blocks), dim3(256), 0, stream, start, stop, 0,
                        uint32_t(key), uint32_t(key >> 32), uint32_t(hop), uint32_t(etype),
                        steps, lim, reinterpret_cast<unsigned long long *>(count));
  return hipGetLastError();
}

hipError_t launch_philox(const uint32_t *ctr, uint64_t key, int64_t n,
                         uint32_t *out, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_philox, dim3(grid_for(n, 256)), dim3(256), 0, stream, ctr,
                     uint32_t(key), uint32_t(key >> 32), n, out);
  return hipGetLastError();
}

}  // namespace hg
