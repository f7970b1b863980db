// Per-hop compaction on gfx950 (DistDGLv2, arXiv 2112.15345, Sec. 4.2.2: the
// frontier of the next hop is the unique set of this hop's vertices, and
// compaction relabels vertices and edges).
//
// The newly reached vertices of a node type are deduplicated and put in
// ascending ID order with one mark per vertex: the sampler marks every kept
// source v reached (a byte, or a bit laid out as the frontier bits), and the
// new vertices are the reached vertices whose frontier bit is clear; a prefix
// count of those (per node type) then gives each one its rank, which is its
// position among the new vertices.
// The count is a reduce-then-scan over kTile-word tiles in three launches
// (count per tile; scan of the tile counts; rank and assign), which needs no
// inter-block waiting.  A dense int32 map (vertex -> local ID, meaningful while
// the vertex's frontier bit is set) holds the local IDs of the frontier and of
// the new vertices for the relabel.
#include "hg_device.hpp"
#include "hg_internal.hpp"

namespace hg {

namespace {

__device__ __forceinline__ int64_t gs_step() {
  return int64_t(gridDim.x) * blockDim.x;
}

unsigned grid_for(int64_t n, int threads, int64_t cap = 1 << 20) {
  int64_t b = (n + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return unsigned(b);
}

struct CompactArgs {
  HopView hv;
  const TypeStatic *ts;
  int32_t n_types;
  uint8_t *reached;  // reached this hop (one byte per vertex)
  uint32_t *fbits;   // in the frontier (one bit per vertex)
  uint32_t *rbits;   // non-NULL: the hop marked reached bits (laid out as fbits) instead
  const int64_t *tile_base;
  int64_t n_tiles;
  int64_t copy_total;
  int64_t *tile_pre;  // [n_tiles + 1] set bits in earlier tiles, of any type (or look-back words)
  int32_t *tile_cnt;  // per tile: set bits
  int64_t *small;
  bool collect;       // only list the vertices (no map, no frontier bits)
};

// Four flag bytes (each 0 or 1) as four bits: byte k of x lands on bit 24 + k
// of x * 0x01020408, with no carries from the other partial products.
__device__ __forceinline__ uint32_t pack4(uint32_t x) {
  return ((x & 0x01010101u) * 0x01020408u) >> 24;
}
__device__ __forceinline__ uint32_t pack16(uint4 v) {
  return pack4(v.x) | (pack4(v.y) << 4) | (pack4(v.z) << 8) | (pack4(v.w) << 12);
}

// A thread's share of a tile (kTileItems * 32 vertices): their reached flags
// as bits, and their frontier words.
struct TileWords {
  uint2 reached, front;
  __device__ uint2 fresh() const {  // reached, not yet in the frontier
    return uint2{reached.x & ~front.x, reached.y & ~front.y};
  }
};
static_assert(kTileItems == 2, "a thread covers 64 vertices");
__device__ __forceinline__ const uint4 *reached_of(const CompactArgs &A, int64_t tile) {
  return reinterpret_cast<const uint4 *>(A.reached + (tile * kTile + threadIdx.x * kTileItems) * 32);
}
__device__ __forceinline__ TileWords tile_words(const CompactArgs &A, int64_t tile) {
  const int64_t w = tile * kTile + threadIdx.x * kTileItems;
  const uint2 front = *reinterpret_cast<const uint2 *>(A.fbits + w);
  if (A.rbits) return TileWords{*reinterpret_cast<const uint2 *>(A.rbits + w), front};
  const uint4 *r = reached_of(A, tile);
  const uint4 r0 = r[0], r1 = r[1], r2 = r[2], r3 = r[3];
  return TileWords{uint2{pack16(r0) | (pack16(r1) << 16), pack16(r2) | (pack16(r3) << 16)},
                   front};
}
// Clears the thread's reached bytes or bits (when any is set).
__device__ __forceinline__ void clear_reached(const CompactArgs &A, int64_t tile,
                                              const TileWords &tw) {
  if (A.rbits) {
    if ((tw.reached.x | tw.reached.y) != 0)
      *reinterpret_cast<uint2 *>(A.rbits + tile * kTile + threadIdx.x * kTileItems) =
          uint2{0, 0};
    return;
  }
  if ((tw.reached.x | tw.reached.y) != 0) {
    uint4 *r = const_cast<uint4 *>(reached_of(A, tile));
    const uint4 z{0, 0, 0, 0};
    r[0] = z;
    r[1] = z;
    r[2] = z;
    r[3] = z;
  }
}

// Copies kTile frontier entries into the head of the source lists.
__device__ void copy_tile(const CompactArgs &A, int64_t ct) {
  for (int k = 0; k < kTileItems; ++k) {
    const int64_t x = ct * kTile + k * kTileThreads + threadIdx.x;
    if (x >= A.copy_total) return;
    int64_t acc = 0;
    int t = 0;
    for (; t < A.n_types - 1; ++t) {
      if (x < acc + A.hv.nF[t]) break;
      acc += A.hv.nF[t];
    }
    A.hv.src_out[t][x - acc] = A.hv.frontier[t][x - acc];
  }
}

// 1. Set bits per tile; the blocks past the tiles copy the frontier.
__global__ __launch_bounds__(kTileThreads) void k_bits_count(CompactArgs A) {
  __shared__ int64_t lds[8];
  const int64_t tile = blockIdx.x;
  if (tile >= A.n_tiles) {
    copy_tile(A, tile - A.n_tiles);
    return;
  }
  static_assert(kTileItems == 2, "one 8-byte load per thread");
  const TileWords tw = tile_words(A, tile);
  const uint2 w = tw.fresh();
  int64_t total;
  block_excl_scan_256(__popc(w.x) + __popc(w.y), lds, &total);
  if (threadIdx.x == 0) A.tile_cnt[tile] = int32_t(total);
  // a tile without new vertices is done: the assign pass skips it
  if (total == 0) clear_reached(A, tile, tw);
}

// 2. Exclusive scan of the tile counts over all tiles, in one block: tile_pre
// gets the set bits of every earlier tile (of any type), and tile_pre[n_tiles]
// the total.  A tile's prefix within its type is then tile_pre[tile] -
// tile_pre[first tile of the type]; each type's count of new vertices is the
// difference at its bounds.
constexpr int kScanThreads = 1024;
// Tile counts per thread and pass: all of a pass's loads are issued before
// the block scan, so a pass costs one memory round trip (11k tiles of the
// billion-edge share in one pass instead of eleven).
constexpr int kScanItems = 16;
__global__ __launch_bounds__(kScanThreads) void k_bits_scan(CompactArgs A) {
  constexpr int kWaves = kScanThreads / kWave;
  __shared__ int64_t s_wave[kWaves];
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  int64_t carry = 0;
  for (int64_t c0 = 0; c0 < A.n_tiles; c0 += int64_t(kScanThreads) * kScanItems) {
    const int64_t base = c0 + int64_t(threadIdx.x) * kScanItems;
    int32_t x[kScanItems];
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) x[k] = base + k < A.n_tiles ? A.tile_cnt[base + k] : 0;
    int64_t mine = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) mine += x[k];
    const int64_t inc = wave_incl_scan_i64(mine);
    if (lane == kWave - 1) s_wave[wave] = inc;
    __syncthreads();
    int64_t before = 0, sum = 0;
    for (int v = 0; v < kWaves; ++v) {
      const int64_t y = s_wave[v];
      if (v < wave) before += y;
      sum += y;
    }
    int64_t run = carry + before + inc - mine;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
      if (base + k < A.n_tiles) A.tile_pre[base + k] = run;
      run += x[k];
    }
    carry += sum;
    __syncthreads();
  }
  if (threadIdx.x == 0) A.tile_pre[A.n_tiles] = carry;
  __syncthreads();
  // new vertices of each type (the block's own stores are visible to it)
  for (int t = threadIdx.x; t < A.n_types; t += kScanThreads)
    A.small[kSlotNew + t] = A.tile_pre[A.tile_base[t + 1]] - A.tile_pre[A.tile_base[t]];
}

// Gives the new vertices of the thread's share of a tile (the first has local
// ID `local`) their local IDs, adds them to the frontier bits and clears the
// reached bits.
__device__ __forceinline__ void assign_bits(const CompactArgs &A, int t, int64_t first,
                                            int64_t tile, const TileWords &tw, int64_t local) {
  clear_reached(A, tile, tw);
  const uint2 ab = tw.fresh();
  if ((ab.x | ab.y) == 0) return;
  if (!A.collect)
    *reinterpret_cast<uint2 *>(A.fbits + tile * kTile + threadIdx.x * kTileItems) =
        uint2{tw.front.x | ab.x, tw.front.y | ab.y};
  int32_t *map = A.ts[t].map;
  int64_t *out = A.hv.src_out[t];
  const uint32_t words[kTileItems] = {ab.x, ab.y};
  const int64_t v0 = ((tile - first) * kTile + threadIdx.x * kTileItems) * 32;
#pragma unroll
  for (int k = 0; k < kTileItems; ++k) {
    uint32_t m = words[k];
    while (m) {
      const int bit = __ffs(m) - 1;
      m &= m - 1;
      const int64_t v = v0 + k * 32 + bit;
      if (!A.collect) map[v] = int32_t(local);
      out[local] = v;
      ++local;
    }
  }
}

// 3. Ranks the set bits of a tile within its node type, gives each new vertex
// its local ID and clears the tile's words.
__global__ __launch_bounds__(kTileThreads) void k_bits_assign(CompactArgs A) {
  __shared__ int64_t lds[8];
  const int64_t tile = blockIdx.x;
  if (A.tile_cnt[tile] == 0) return;
  const int t = find_segment(A.tile_base, A.n_types, tile);
  const TileWords tw = tile_words(A, tile);
  const uint2 ab = tw.fresh();
  int64_t total;
  const int64_t pre = block_excl_scan_256(__popc(ab.x) + __popc(ab.y), lds, &total);
  const int64_t first = A.tile_base[t];
  assign_bits(A, t, first, tile, tw,
              A.hv.nF[t] + (A.tile_pre[tile] - A.tile_pre[first]) + pre);
}

// The three steps in one launch for a few tiles: tiles in ticket order, each
// tile's prefix within its type by decoupled look-back (words in tile_pre);
// the last tile of a type writes the type's count.  Tickets past the tiles
// copy the frontier.
__global__ __launch_bounds__(kTileThreads) void k_bits_single(CompactArgs A, uint32_t epoch,
                                                              uint64_t ticket_base) {
  __shared__ int64_t lds[8];
  const int64_t tile = take_ticket(A.small, ticket_base, lds);
  if (tile >= A.n_tiles) {
    copy_tile(A, tile - A.n_tiles);
    return;
  }
  const int t = find_segment(A.tile_base, A.n_types, tile);
  const int64_t first = A.tile_base[t];
  const TileWords tw = tile_words(A, tile);
  const uint2 ab = tw.fresh();
  int64_t agg[1];
  const int64_t pre = block_excl_scan_256(__popc(ab.x) + __popc(ab.y), lds, &agg[0]);
  int64_t ex[1];
  tile_lookback<1>(Lookback{reinterpret_cast<uint64_t *>(A.tile_pre)}, tile, first, epoch, agg,
                   ex, A.small);
  if (tile == A.tile_base[t + 1] - 1 && threadIdx.x == 0)
    A.small[kSlotNew + t] = ex[0] + agg[0];  // new vertices of type t
  assign_bits(A, t, first, tile, tw, A.hv.nF[t] + ex[0] + pre);
}

// Edge types whose edge starts and source maps the relabel stages in LDS.
constexpr int kRelabelMaxEtypes = 2048;
constexpr int kRelabelItems = 1;

// src_local[j] = map of edge j's source type at src_gid[j].  The etype of an
// edge is found by binary search over the edge starts (in LDS when staged);
// each thread looks up kRelabelItems edges at once.
template <bool kStaged>
__global__ __launch_bounds__(256) void k_relabel(HopView hv, HopView next, const EtypeStatic *es,
                                                 const int64_t *tile_base, const int64_t *small,
                                                 int32_t n_types, int32_t n_etypes,
                                                 int64_t n_edges, const int64_t *src_gid,
                                                 int32_t *src_local, bool xcd) {
  extern __shared__ __align__(16) char relabel_lds[];
  if (blockIdx.x == 0)
    plan_next_hop(hv, next, es, tile_base, small, n_types, n_etypes);
  const int64_t *ebase = small + kSlotNew + n_types;
  int64_t *s_eb = reinterpret_cast<int64_t *>(relabel_lds);
  int32_t **s_map = reinterpret_cast<int32_t **>(s_eb + n_etypes + 1);
  if (kStaged) {
    for (int e = threadIdx.x; e <= n_etypes; e += blockDim.x) {
      s_eb[e] = ebase[e];
      if (e < n_etypes) s_map[e] = es[e].src_map;
    }
    __syncthreads();
  }
  // the grid is a multiple of kXcds blocks, so that its blocks can be ordered
  // per XCD (xcd_block): a mini-batch's map lines then stay in one L2
  const int64_t step = gs_step();
  for (int64_t j0 = xcd_block(blockIdx.x, gridDim.x, xcd) * blockDim.x + threadIdx.x;
       j0 < n_edges; j0 += kRelabelItems * step) {
    int64_t g[kRelabelItems];
    int32_t *m[kRelabelItems];
#pragma unroll
    for (int u = 0; u < kRelabelItems; ++u) {
      const int64_t j = j0 + u * step;
      g[u] = 0;
      m[u] = nullptr;
      if (j < n_edges) {
        g[u] = src_gid[j];
        const int e = find_segment(kStaged ? s_eb : ebase, n_etypes, j);
        m[u] = kStaged ? s_map[e] : es[e].src_map;
      }
    }
    int32_t l[kRelabelItems];
#pragma unroll
    for (int u = 0; u < kRelabelItems; ++u) l[u] = m[u] ? m[u][g[u]] : 0;
#pragma unroll
    for (int u = 0; u < kRelabelItems; ++u)
      if (m[u]) src_local[j0 + u * step] = l[u];
  }
}

}  // namespace

hipError_t launch_compact(HopView hv, const TypeStatic *ts, int32_t n_types,
                          uint8_t *reached, uint32_t *fbits, const int64_t *tile_base,
                          int64_t n_tiles, int64_t copy_total, int64_t *tile_sums,
                          uint32_t epoch, uint64_t ticket_base, int64_t *small,
                          int64_t *ticketed, hipStream_t stream, bool collect, StageEv ev,
                          uint32_t *rbits) {
  CompactArgs A{hv, ts, n_types, reached, fbits, rbits, tile_base, n_tiles, copy_total, tile_sums,
                reinterpret_cast<int32_t *>(tile_sums + n_tiles + 1), small, collect};
  const int64_t copy_blocks = (copy_total + kTile - 1) / kTile;
  *ticketed = 0;
  if (n_tiles <= kSinglePassTiles) {
    const int64_t blocks = n_tiles + copy_blocks;
    if (blocks > 0) {
      launch_k(k_bits_single, dim3(unsigned(blocks)), dim3(kTileThreads), 0, stream, ev.start,
               ev.stop, A, epoch, ticket_base);
      *ticketed = blocks;
    } else if (ev.any()) {
      hipError_t e = record_empty_stage(ev, stream);
      if (e != hipSuccess) return e;
    }
    return hipGetLastError();
  }
  // n_tiles > kSinglePassTiles here, so every launch has blocks
  launch_k(k_bits_count, dim3(unsigned(n_tiles + copy_blocks)), dim3(kTileThreads), 0, stream,
           ev.start, nullptr, A);
  hipLaunchKernelGGL(k_bits_scan, dim3(1), dim3(kScanThreads), 0, stream, A);
  launch_k(k_bits_assign, dim3(unsigned(n_tiles)), dim3(kTileThreads), 0, stream, nullptr,
           ev.stop, A);
  return hipGetLastError();
}

hipError_t launch_relabel(HopView hv, HopView next, const EtypeStatic *es,
                          const int64_t *tile_base, const int64_t *small,
                          int32_t n_types, int32_t n_etypes, int64_t n_edges,
                          const int64_t *src_gid, int32_t *src_local,
                          hipStream_t stream, StageEv ev, bool xcd_order) {
  // at least one block: block 0 plans the next hop
  const unsigned grid =
      unsigned(xcd_round(grid_for((n_edges + kRelabelItems - 1) / kRelabelItems, 256, 1 << 20)));
  if (n_etypes <= kRelabelMaxEtypes)
    launch_k(k_relabel<true>, dim3(grid), dim3(256), size_t(16) * (n_etypes + 1), stream,
             ev.start, ev.stop, hv, next, es, tile_base, small, n_types, n_etypes, n_edges,
             src_gid, src_local, xcd_order);
  else
    launch_k(k_relabel<false>, dim3(grid), dim3(256), 0, stream, ev.start, ev.stop, hv, next,
             es, tile_base, small, n_types, n_etypes, n_edges, src_gid, src_local, xcd_order);
  return hipGetLastError();
}

}  // namespace hg
