// Layer-wise (LADIES) sampling on gfx950.  DistDGLv2 (arXiv 2112.15345, Sec.
// 4.2.2) names layer-wise sampling as fitting the same decomposition of
// sampling, compaction and feature copy; the algorithm is LADIES (Zou et al.,
// NeurIPS 2019, Algorithm 1).  Each hop draws a fixed number of vertices per
// node type for the whole layer, with probability proportional to their
// importance, and keeps every in-edge of the frontier from the next frontier.
//
// One hop, after the counting pass has numbered every in-edge of the frontier
// (fanout -1: pair p's in-edges are positions off[p] .. off[p+1]-1); no
// sampler runs, and the edges are read from the CSC where needed:
//  1. k_lw_tile_pairs, k_lw_weights : the first pair of every 512-position
//                    tile; then the importance of every candidate (a source
//                    not in the frontier, which is marked reached): sum of
//                    floor(2^32 / deg(v)^2) over its edges into the frontier,
//                    64-bit atomics (exact in any order), blocks over tiles of
//                    positions whose etypes and pairs are staged in LDS once
//                    per tile (as in the kept-edge scans);
//  2. compaction   : (collect mode) the candidates of each type, ascending;
//  3. k_lw_scan_*  : exclusive prefix of their importance per type
//                    (reduce-then-scan over 512-candidate tiles);
//  4. k_lw_draw    : draw k takes r = floor(x * total / 2^64), x from
//                    Philox4x32-10 at (k, 2^30 | hop, type), and marks the
//                    candidate whose interval [prefix, prefix + weight) holds
//                    r (binary search);
//  5. compaction   : the drawn vertices join the frontier (ascending);
//  6. k_lw_scan_*  : the kept in-edges (source in the next frontier) by an
//                    exclusive scan of their flags, emitted in order;
//  7. k_lw_indptr  : the block CSC, the kept edge starts per etype, and the
//                    next hop's plan.
#include "hg_device.hpp"
#include "hg_internal.hpp"

namespace hg {

namespace {

constexpr int kLwThreads = 256;
constexpr int kLwItems = 2;
constexpr int64_t kLwTile = int64_t(kLwThreads) * kLwItems;
static_assert(kLwTile == kLayerTile, "the runtime sizes the scans in these tiles");

__device__ __forceinline__ int64_t gs_start() {
  return int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
}
__device__ __forceinline__ int64_t gs_step() {
  return int64_t(gridDim.x) * blockDim.x;
}

unsigned grid_for(int64_t n, int threads, int64_t cap = 1 << 16) {
  int64_t b = (n + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return unsigned(b);
}

__device__ __forceinline__ bool in_frontier(const uint32_t *fbits, int64_t v) {
  return (fbits[v >> 5] >> (v & 31)) & 1u;
}

// floor(2^32 / d^2) for d >= 1 (zero once d^2 > 2^32).  The correctly
// rounded double quotient lies between the two integers around the exact one,
// so its floor is the exact floor or one above; integer checks settle it.
__device__ __forceinline__ uint64_t layer_weight(int64_t d) {
  const uint64_t d2 = uint64_t(d) * uint64_t(d);
  constexpr uint64_t kOne = uint64_t(1) << 32;
  if (d2 > kOne) return 0;
  uint64_t q = uint64_t(4294967296.0 / double(d2));
  if (q * d2 > kOne) --q;
  else if ((q + 1) * d2 <= kOne) ++q;
  return q;
}

__device__ __forceinline__ const int64_t *ebase_of(const LayerArgs &A) {
  return A.small + kSlotNew + A.n_types;  // starts of each etype's emitted edges
}
__device__ __forceinline__ int64_t *kept_base_of(const LayerArgs &A) {
  return A.small + kSlotNew + A.n_types + A.n_etypes + 1;
}

// The in-edges of the frontier are never written out.  The counting pass
// numbers them: pair p's in-edges are positions off[p] .. off[p+1]-1, at CSC
// slots plo[p] + (i - off[p]); position i lies in the last pair with
// off[p] <= i (empty pairs share the offset of the pair after them).  The
// kernels below read the source of position i from the CSC where they need it.

// The etypes that a block's contiguous range [j0, j1) of positions spans,
// resolved once per block: their starts and what the per-edge work reads of
// them.  A range over more than kTileSegs etypes leaves n = 0 and its edges
// search the etype starts one by one.
constexpr int kTileSegs = 32;
struct TileSegs {
  int64_t start[kTileSegs + 1];
  const uint32_t *fbits[kTileSegs];  // frontier bits of the source type
  void *per_seg[kTileSegs];          // importance array of the source type, or source map
  const int64_t *indices[kTileSegs];
  uint8_t *reached[kTileSegs];       // reached flags of the source type
  int64_t pair_base[kTileSegs];
  int e0, n;
};

// kKind 0: per_seg = importance array of the source type; 1: source map.
template <int kKind>
__device__ void tile_segs_load(const LayerArgs &A, int64_t j0, int64_t j1, TileSegs &T) {
  const int64_t *ebase = ebase_of(A);
  if (threadIdx.x == 0) {
    const int a = find_segment(ebase, A.n_etypes, j0);
    const int b = find_segment(ebase, A.n_etypes, j1 - 1);
    T.e0 = a;
    T.n = b - a + 1 <= kTileSegs ? b - a + 1 : 0;
  }
  __syncthreads();
  const int n = T.n;
  if (int(threadIdx.x) <= n && n > 0) {
    const int e = T.e0 + int(threadIdx.x);
    T.start[threadIdx.x] = ebase[e];
    if (int(threadIdx.x) < n) {
      const EtypeStatic &E = A.es[e];
      T.fbits[threadIdx.x] = A.ts[E.src_type].fbits;
      if (kKind == 0)
        T.per_seg[threadIdx.x] = A.wt[E.src_type];
      else
        T.per_seg[threadIdx.x] = E.src_map;
      T.indices[threadIdx.x] = E.indices;
      T.reached[threadIdx.x] = E.src_reached;
      T.pair_base[threadIdx.x] = A.hv.pair_base[e];
    }
  }
  __syncthreads();
}

// Segment of position j in the block's table, from a hint not above it (the
// positions of one thread come in ascending order).
__device__ __forceinline__ int tile_seg(const TileSegs &T, int s, int64_t j) {
  while (s + 1 < T.n && T.start[s + 1] <= j) ++s;
  return s;
}

// What a position needs of its etype.
struct SegView {
  const uint32_t *fbits;
  void *per_seg;
  const int64_t *indices;
  uint8_t *reached;
  int64_t pair_base;
};
template <int kKind>
__device__ __forceinline__ SegView seg_view(const LayerArgs &A, const TileSegs &T, int &s,
                                            int64_t j) {
  if (T.n > 0) {
    s = tile_seg(T, s, j);
    return SegView{T.fbits[s], T.per_seg[s], T.indices[s], T.reached[s], T.pair_base[s]};
  }
  const int e = find_segment(ebase_of(A), A.n_etypes, j);
  const EtypeStatic &E = A.es[e];
  return SegView{A.ts[E.src_type].fbits,
                 kKind == 0 ? static_cast<void *>(A.wt[E.src_type]) : static_cast<void *>(E.src_map),
                 E.indices, E.src_reached, A.hv.pair_base[e]};
}

// tile_pair[t] = the last pair p with off[p] <= t * kLwTile, for every tile t
// of positions; tile_pair[n_tiles] = the last pair.  Each non-empty pair writes
// the tiles that start inside it.
__global__ __launch_bounds__(256) void k_lw_tile_pairs(LayerArgs A) {
  for (int64_t p = gs_start(); p < A.n_pairs; p += gs_step()) {
    const int64_t lo = A.pa.off[p], hi = A.pa.off[p + 1];
    for (int64_t t = (lo + kLwTile - 1) / kLwTile; t * kLwTile < hi; ++t) A.tile_pair[t] = p;
  }
  if (gs_start() == 0) A.tile_pair[A.n_keep_tiles] = A.n_pairs - 1;
}

// The pairs of a block's positions [j0, j1) in LDS: from tile_pair of the tile
// holding j0 to tile_pair of the tile after j1 - 1 (which may hold one pair
// past j1).  More than kTilePairs pairs (runs of empty pairs) leave n = 0, and
// each position then searches the pair offsets.
constexpr int kTilePairs = 1024;
template <int N>
struct TilePairs {
  int64_t off[N], plo[N], deg[N];
};
struct PairRange {
  int64_t p0;
  int n;
};
template <int N>
__device__ PairRange tile_pairs_load(const LayerArgs &A, int64_t j0, int64_t j1,
                                     TilePairs<N> &Q) {
  const int64_t pa = A.tile_pair[j0 / kLwTile];
  const int64_t pb = A.tile_pair[(j1 - 1) / kLwTile + 1];
  const int n = pb - pa + 1 <= N ? int(pb - pa + 1) : 0;
  for (int k = threadIdx.x; k < n; k += blockDim.x) {
    Q.off[k] = A.pa.off[pa + k];
    Q.plo[k] = A.pa.plo[pa + k];
    Q.deg[k] = A.pa.pdeg[pa + k];
  }
  __syncthreads();
  return PairRange{pa, n};
}

// Position j: its pair, its CSC slot and the pair's in-degree.
struct EdgeAt {
  int64_t p, slot, deg;
};
template <int N>
__device__ __forceinline__ EdgeAt edge_at(const LayerArgs &A, const TilePairs<N> &Q,
                                          const PairRange &R, int64_t j) {
  if (R.n > 0) {
    int lo = 0, hi = R.n;  // Q.off[lo] <= j
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (Q.off[mid] <= j)
        lo = mid;
      else
        hi = mid;
    }
    return EdgeAt{R.p0 + lo, Q.plo[lo] + (j - Q.off[lo]), Q.deg[lo]};
  }
  int64_t lo = 0, hi = A.n_pairs;
  while (hi - lo > 1) {
    const int64_t mid = (lo + hi) >> 1;
    if (A.pa.off[mid] <= j)
      lo = mid;
    else
      hi = mid;
  }
  return EdgeAt{lo, A.pa.plo[lo] + (j - A.pa.off[lo]), A.pa.pdeg[lo]};
}

// Blocks of 256 threads take tiles of kLwWeightTile positions (whole scan
// tiles), each thread every 256th position of the tile.
constexpr int kLwWeightItems = 8;
constexpr int64_t kLwWeightTile = 256 * kLwWeightItems;
static_assert(kLwWeightTile % kLwTile == 0, "weight tiles are whole scan tiles");

__global__ __launch_bounds__(256) void k_lw_weights(LayerArgs A) {
  __shared__ TileSegs T;
  __shared__ TilePairs<kTilePairs> Q;
  const int64_t n_tiles = (A.n_all + kLwWeightTile - 1) / kLwWeightTile;
  for (int64_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
    const int64_t j0 = tile * kLwWeightTile;
    const int64_t j1 = j0 + kLwWeightTile < A.n_all ? j0 + kLwWeightTile : A.n_all;
    tile_segs_load<0>(A, j0, j1, T);
    const PairRange R = tile_pairs_load(A, j0, j1, Q);
    int s = 0;
    for (int64_t j = j0 + threadIdx.x; j < j1; j += 256) {
      const SegView v = seg_view<0>(A, T, s, j);
      const EdgeAt x = edge_at(A, Q, R, j);
      const int64_t u = v.indices[x.slot];
      if (in_frontier(v.fbits, u)) continue;
      v.reached[u] = 1;  // a candidate
      const uint64_t w = layer_weight(x.deg);
      if (w)
        atomicAdd(reinterpret_cast<unsigned long long *>(static_cast<uint64_t *>(v.per_seg) + u),
                  (unsigned long long)w);
    }
    __syncthreads();  // T and Q are rebuilt for the next tile
  }
}

// ---- reduce-then-scan over tiles of kLwTile values --------------------------
// kind 0: the candidates' importance, one segment per node type (tiles
//         cand_tile[t] .. cand_tile[t+1]; the type's candidates are counted in
//         small[kSlotNew + t] by the collect compaction);
// kind 1: the kept flags of the emitted edges, one segment.
template <int kKind>
struct ScanSeg {
  int seg;
  int64_t first_tile, n;
};

template <int kKind>
__device__ __forceinline__ ScanSeg<kKind> seg_of(const LayerArgs &A, int64_t tile) {
  if (kKind == 0) {
    const int t = find_segment(A.cand_tile, A.n_types, tile);
    return ScanSeg<kKind>{t, A.cand_tile[t], A.small[kSlotNew + t]};
  }
  return ScanSeg<kKind>{0, 0, A.n_all};
}

// Position i of a scan: its value (kind 0: the candidate's importance; kind 1:
// whether the in-edge's source is in the next frontier) and, for kind 1, what
// the apply pass writes of a kept edge.
struct ScanItem {
  int64_t v;
  int64_t slot, dst, u;  // kind 1: CSC slot (edge ID), destination local ID, source
  const int32_t *src_map;
};

// The pair table of a scan tile: kind 1 only.
template <int kKind>
using ScanPairs = TilePairs<kKind == 1 ? kTilePairs : 1>;

template <int kKind>
__device__ __forceinline__ ScanItem scan_item(const LayerArgs &A, const ScanSeg<kKind> &S,
                                              const TileSegs &T, const ScanPairs<kKind> &Q,
                                              const PairRange &R, int &s, int64_t i) {
  ScanItem it{0, 0, 0, 0, nullptr};
  if (i >= S.n) return it;
  if (kKind == 0) {
    it.v = int64_t(A.wt[S.seg][A.cand[S.seg][i]]);
    return it;
  }
  const SegView sv = seg_view<1>(A, T, s, i);
  const EdgeAt x = edge_at(A, Q, R, i);
  it.u = sv.indices[x.slot];
  it.v = in_frontier(sv.fbits, it.u) ? 1 : 0;
  it.slot = x.slot;
  it.dst = x.p - sv.pair_base;
  it.src_map = static_cast<const int32_t *>(sv.per_seg);
  return it;
}

// The block's etype and pair tables for a kind-1 tile.
template <int kKind>
__device__ __forceinline__ PairRange scan_tables(const LayerArgs &A, int64_t tile, TileSegs &T,
                                                 ScanPairs<kKind> &Q) {
  if (kKind == 1) {
    const int64_t j0 = tile * kLwTile;
    const int64_t j1 = j0 + kLwTile < A.n_all ? j0 + kLwTile : A.n_all;
    tile_segs_load<1>(A, j0, j1, T);
    return tile_pairs_load(A, j0, j1, Q);
  }
  return PairRange{0, 0};
}

template <int kKind>
__global__ __launch_bounds__(kLwThreads) void k_lw_scan_reduce(LayerArgs A) {
  __shared__ int64_t lds[8];
  __shared__ TileSegs T;
  __shared__ ScanPairs<kKind> Q;
  const int64_t tile = blockIdx.x;
  const PairRange R = scan_tables<kKind>(A, tile, T, Q);
  const ScanSeg<kKind> S = seg_of<kKind>(A, tile);
  const int64_t i0 = (tile - S.first_tile) * kLwTile + threadIdx.x * kLwItems;
  int64_t v = 0;
  int s = 0;
#pragma unroll
  for (int k = 0; k < kLwItems; ++k) v += scan_item<kKind>(A, S, T, Q, R, s, i0 + k).v;
  int64_t total;
  block_excl_scan_256(v, lds, &total);
  if (threadIdx.x == 0) A.tile_sum[tile] = total;
}

// One block: tile_pre = exclusive scan of tile_sum over all n_tiles tiles,
// tile_pre[n_tiles] = the grand total.  Each thread takes kLwScanPer
// consecutive tiles of a chunk.
constexpr int kLwScanThreads = 1024;
constexpr int kLwScanPer = 8;
__global__ __launch_bounds__(kLwScanThreads) void k_lw_scan_tiles(int64_t *tile_sum,
                                                                  int64_t *tile_pre,
                                                                  int64_t n_tiles) {
  constexpr int kWaves = kLwScanThreads / kWave;
  constexpr int64_t kChunk = int64_t(kLwScanThreads) * kLwScanPer;
  __shared__ int64_t s_wave[kWaves];
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  int64_t carry = 0;
  for (int64_t c0 = 0; c0 < n_tiles; c0 += kChunk) {
    const int64_t i0 = c0 + int64_t(threadIdx.x) * kLwScanPer;
    int64_t x[kLwScanPer];
    int64_t mine = 0;
#pragma unroll
    for (int k = 0; k < kLwScanPer; ++k) {
      x[k] = i0 + k < n_tiles ? tile_sum[i0 + k] : 0;
      mine += x[k];
    }
    const int64_t inc = wave_incl_scan_i64(mine);
    if (lane == kWave - 1) s_wave[wave] = inc;
    __syncthreads();
    int64_t before = 0, sum = 0;
    for (int w = 0; w < kWaves; ++w) {
      const int64_t y = s_wave[w];
      if (w < wave) before += y;
      sum += y;
    }
    int64_t run = carry + before + inc - mine;
#pragma unroll
    for (int k = 0; k < kLwScanPer; ++k) {
      if (i0 + k < n_tiles) tile_pre[i0 + k] = run;
      run += x[k];
    }
    carry += sum;
    __syncthreads();
  }
  if (threadIdx.x == 0) tile_pre[n_tiles] = carry;
}

// Each tile's values get their exclusive prefix within the segment.
template <int kKind>
__global__ __launch_bounds__(kLwThreads) void k_lw_scan_apply(LayerArgs A) {
  __shared__ int64_t lds[8];
  __shared__ TileSegs T;
  __shared__ ScanPairs<kKind> Q;
  const int64_t tile = blockIdx.x;
  const PairRange R = scan_tables<kKind>(A, tile, T, Q);
  const ScanSeg<kKind> S = seg_of<kKind>(A, tile);
  const int64_t i0 = (tile - S.first_tile) * kLwTile + threadIdx.x * kLwItems;
  ScanItem it[kLwItems];
  int64_t sum = 0;
  int s = 0;
#pragma unroll
  for (int k = 0; k < kLwItems; ++k) {
    it[k] = scan_item<kKind>(A, S, T, Q, R, s, i0 + k);
    sum += it[k].v;
  }
  int64_t total;
  int64_t pre = block_excl_scan_256(sum, lds, &total) +
                (A.tile_pre[tile] - A.tile_pre[S.first_tile]);
#pragma unroll
  for (int k = 0; k < kLwItems; ++k) {
    const int64_t i = i0 + k;
    if (i < S.n) {
      if (kKind == 0) {
        A.prefix[S.seg][i] = uint64_t(pre);
        A.wt[S.seg][A.cand[S.seg][i]] = 0;  // clean for the next hop and call
      } else {
        A.pos[i] = pre;
        if (it[k].v) {
          A.out_eid[pre] = it[k].slot;
          A.out_dst_local[pre] = int32_t(it[k].dst);
          A.out_src_local[pre] = it[k].src_map[it[k].u];
        }
      }
    }
    pre += it[k].v;
  }
  if (kKind == 1 && tile == int64_t(gridDim.x) - 1 && threadIdx.x == kLwThreads - 1)
    A.pos[A.n_all] = pre;  // the last thread of the last tile ends past n_all
}

// Draws: thread x of type t's range draw_base[t] .. draw_base[t+1] makes draw
// x - draw_base[t] (or, for a type that takes every candidate, marks
// candidate x - draw_base[t]).
__global__ __launch_bounds__(256) void k_lw_draw(LayerArgs A) {
  const int64_t n = A.draw_base[A.n_types];
  for (int64_t x = gs_start(); x < n; x += gs_step()) {
    const int t = find_segment(A.draw_base, A.n_types, x);
    const int64_t k = x - A.draw_base[t];
    const int copy = t / A.key_T;
    const uint64_t sigma = A.sigmas[copy];
    const int64_t nc = A.small[kSlotNew + t];
    const int64_t *cand = A.cand[t];
    uint8_t *reached = A.ts[t].reached;
    if (A.draws[t] < 0) {
      if (k < nc) reached[cand[k]] = 1;
      continue;
    }
    const uint64_t total = uint64_t(A.tile_pre[A.cand_tile[t + 1]] - A.tile_pre[A.cand_tile[t]]);
    if (total == 0 || nc == 0) continue;
    const U32x4 r4 = philox4x32_10(U32x4{uint32_t(k), uint32_t(uint64_t(k) >> 32),
                                         0x40000000u | uint32_t(A.hop),
                                         uint32_t(t - copy * A.key_T)},
                                   uint32_t(sigma), uint32_t(sigma >> 32));
    const uint64_t r = __umul64hi(uint64_t(r4.x) | (uint64_t(r4.y) << 32), total);
    // the last candidate whose prefix is not above r (zero-weight candidates
    // share the prefix of the next one and are never the last)
    const uint64_t *pre = A.prefix[t];
    int64_t a = 0, b = nc - 1;
    while (a < b) {
      const int64_t m = a + (b - a + 1) / 2;
      if (pre[m] <= r)
        a = m;
      else
        b = m - 1;
    }
    reached[cand[a]] = 1;
  }
}

// Per pair its block-CSC entry from the kept positions; the closing entry and
// the kept edge start of every etype; block 0 plans the next hop.
__global__ __launch_bounds__(256) void k_lw_indptr(LayerArgs A) {
  const int64_t *ebase = ebase_of(A);
  const int64_t *pb = A.hv.pair_base;
  // kept edges before emitted edge i (no edges: no scan ran, and none are kept)
  auto pos = [&](int64_t i) { return A.n_all > 0 ? A.pos[i] : int64_t(0); };
  if (blockIdx.x == 0) {
    int64_t *kept = kept_base_of(A);
    for (int e = threadIdx.x; e <= A.n_etypes; e += blockDim.x) {
      kept[e] = pos(ebase[e]);
      if (e < A.n_etypes) A.out_indptr[pb[e + 1] + e] = pos(ebase[e + 1]) - pos(ebase[e]);
    }
    plan_next_hop(A.hv, A.next, A.es, A.tile_base, A.small, A.n_types, A.n_etypes);
  }
  for (int64_t p = gs_start(); p < A.n_pairs; p += gs_step()) {
    const int e = A.pa.pet[p];
    A.out_indptr[pb[e] + e + (p - pb[e])] = pos(A.pa.off[p]) - pos(ebase[e]);
  }
}

}  // namespace

hipError_t launch_lw_weights(const LayerArgs &A, hipStream_t stream) {
  if (A.n_all <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_lw_tile_pairs, dim3(grid_for(A.n_pairs, 256)), dim3(256), 0, stream, A);
  hipLaunchKernelGGL(k_lw_weights, dim3(grid_for(A.n_all, kLwWeightTile)), dim3(256), 0, stream,
                     A);
  return hipGetLastError();
}

hipError_t launch_lw_prefix(const LayerArgs &A, hipStream_t stream) {
  const int64_t tiles = A.cand_tiles;
  if (tiles <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_lw_scan_reduce<0>, dim3(unsigned(tiles)), dim3(kLwThreads), 0, stream, A);
  hipLaunchKernelGGL(k_lw_scan_tiles, dim3(1), dim3(kLwScanThreads), 0, stream, A.tile_sum,
                     A.tile_pre, tiles);
  hipLaunchKernelGGL(k_lw_scan_apply<0>, dim3(unsigned(tiles)), dim3(kLwThreads), 0, stream, A);
  return hipGetLastError();
}

hipError_t launch_lw_draw(const LayerArgs &A, hipStream_t stream) {
  const int64_t n = A.draw_threads;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_lw_draw, dim3(grid_for(n, 256)), dim3(256), 0, stream, A);
  return hipGetLastError();
}

hipError_t launch_lw_keep(const LayerArgs &A, hipStream_t stream) {
  const int64_t tiles = A.n_keep_tiles;
  if (tiles > 0) {
    hipLaunchKernelGGL(k_lw_scan_reduce<1>, dim3(unsigned(tiles)), dim3(kLwThreads), 0, stream,
                       A);
    hipLaunchKernelGGL(k_lw_scan_tiles, dim3(1), dim3(kLwScanThreads), 0, stream, A.tile_sum,
                       A.tile_pre, tiles);
    hipLaunchKernelGGL(k_lw_scan_apply<1>, dim3(unsigned(tiles)), dim3(kLwThreads), 0, stream,
                       A);
  }
  // at least one block: block 0 writes the etype entries and plans the next hop
  hipLaunchKernelGGL(k_lw_indptr, dim3(grid_for(A.n_pairs, 256)), dim3(256), 0, stream, A);
  return hipGetLastError();
}

}  // namespace hg
