// Per-hop compaction on gfx950 (DistDGLv2, arXiv 2112.15345, Sec. 4.2.2: the
// frontier of the next hop is the unique set of this hop's vertices, and
// compaction relabels vertices and edges).
//
// The newly reached vertices of a node type are deduplicated and put in
// ascending ID order with one bit per vertex: the sampler sets bit v for every
// kept source v that is not in the frontier yet; here a single-pass prefix
// count of the set bits (per node type) gives each one its rank, which is its
// position among the new vertices.  A dense int32 map (vertex -> local ID,
// -1 when absent) holds the local IDs of the frontier and of the new vertices
// for the relabel.
#include "hg_device.hpp"
#include "hg_internal.hpp"

namespace hg {

namespace {

__device__ __forceinline__ int64_t gs_start() {
  return int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
}
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
  uint32_t *bitmap;
  const int64_t *tile_base;
  int64_t n_tiles;
  int64_t copy_total;
  Lookback lb;
  uint32_t epoch;
  uint64_t ticket_base;
  int64_t *small;
};

// Ranks the set bits of one 512-word tile within its node type and gives
// each new vertex its local ID.
__device__ void bitmap_tile(const CompactArgs &A, int64_t tile, int64_t *lds) {
  const int t = find_segment(A.tile_base, A.n_types, tile);
  const int64_t first = A.tile_base[t];
  uint32_t *w = A.bitmap + tile * kTile + threadIdx.x * kTileItems;
  const uint2 ab = *reinterpret_cast<const uint2 *>(w);
  const uint32_t words[kTileItems] = {ab.x, ab.y};
  int64_t s = 0;
#pragma unroll
  for (int k = 0; k < kTileItems; ++k) s += __popc(words[k]);
  int64_t agg[1];
  const int64_t pre = block_excl_scan_256(s, lds, &agg[0]);
  int64_t ex[1];
  tile_lookback<1>(A.lb, tile, first, A.epoch, agg, ex, A.small, lds);
  if (tile == A.tile_base[t + 1] - 1 && threadIdx.x == 0)
    A.small[kSlotNew + t] = ex[0] + agg[0];  // new vertices of type t
  if (s == 0) return;
  int32_t *map = A.ts[t].map;
  int64_t *out = A.hv.src_out[t];
  int64_t local = A.hv.nF[t] + ex[0] + pre;
  const int64_t v0 = ((tile - first) * kTile + threadIdx.x * kTileItems) * 32;
#pragma unroll
  for (int k = 0; k < kTileItems; ++k) {
    uint32_t m = words[k];
    while (m) {
      const int bit = __ffs(m) - 1;
      m &= m - 1;
      const int64_t v = v0 + k * 32 + bit;
      map[v] = int32_t(local);
      out[local] = v;
      ++local;
    }
  }
  *reinterpret_cast<uint2 *>(w) = uint2{0, 0};
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

__global__ __launch_bounds__(kTileThreads) void k_compact(CompactArgs A) {
  __shared__ int64_t lds[8];
  const int64_t tile = take_ticket(A.small, A.ticket_base, lds);
  if (tile < A.n_tiles)
    bitmap_tile(A, tile, lds);
  else
    copy_tile(A, tile - A.n_tiles);
}

// Next hop's frontier sizes (this hop's plus the new vertices of each type)
// and pair layout (pairs of etype e: frontier of its destination type).
__device__ void plan_next_hop(HopView hv, HopView next, const EtypeStatic *es,
                              const int64_t *tile_base, const int64_t *small,
                              int32_t n_types, int32_t n_etypes) {
  if (threadIdx.x != 0) return;
  for (int t = 0; t < n_types; ++t) {
    // a type without bitmap tiles (no vertices) gains nothing
    const int64_t u = tile_base[t + 1] > tile_base[t] ? small[kSlotNew + t] : 0;
    next.nF[t] = hv.nF[t] + u;
  }
  int64_t acc = 0;
  for (int e = 0; e < n_etypes; ++e) {
    next.pair_base[e] = acc;
    acc += next.nF[es[e].dst_type];
  }
  next.pair_base[n_etypes] = acc;
}

__global__ void k_relabel(HopView hv, HopView next, const EtypeStatic *es,
                          const int64_t *tile_base, const int64_t *small,
                          int32_t n_types, int32_t n_etypes, int64_t n_edges,
                          const int64_t *src_gid, int32_t *src_local) {
  if (blockIdx.x == 0)
    plan_next_hop(hv, next, es, tile_base, small, n_types, n_etypes);
  const int64_t *ebase = small + kSlotNew + n_types;
  for (int64_t j = gs_start(); j < n_edges; j += gs_step()) {
    const int e = find_segment(ebase, n_etypes, j);
    src_local[j] = es[e].src_map[src_gid[j]];
  }
}

}  // namespace

hipError_t launch_compact(HopView hv, const TypeStatic *ts, int32_t n_types,
                          uint32_t *bitmap, const int64_t *tile_base,
                          int64_t n_tiles, int64_t copy_total, Lookback lb,
                          uint32_t epoch, uint64_t ticket_base, int64_t *small,
                          int32_t *blocks_launched, hipStream_t stream) {
  CompactArgs A{hv, ts, n_types, bitmap, tile_base, n_tiles, copy_total, lb, epoch,
                ticket_base, small};
  const int64_t copy_blocks = (copy_total + kTile - 1) / kTile;
  const int64_t blocks = n_tiles + copy_blocks;
  *blocks_launched = int32_t(blocks);
  if (blocks <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_compact, dim3(unsigned(blocks)), dim3(kTileThreads), 0,
                     stream, A);
  return hipGetLastError();
}

hipError_t launch_relabel(HopView hv, HopView next, const EtypeStatic *es,
                          const int64_t *tile_base, const int64_t *small,
                          int32_t n_types, int32_t n_etypes, int64_t n_edges,
                          const int64_t *src_gid, int32_t *src_local,
                          hipStream_t stream) {
  // at least one block: block 0 plans the next hop
  hipLaunchKernelGGL(k_relabel, dim3(grid_for(n_edges, 256)), dim3(256), 0, stream, hv,
                     next, es, tile_base, small, n_types, n_etypes, n_edges, src_gid,
                     src_local);
  return hipGetLastError();
}

}  // namespace hg
