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
  HopView hv, next;
  const TypeStatic *ts;
  const EtypeStatic *es;
  int32_t n_types, n_etypes;
  uint32_t *bitmap;
  const int64_t *tile_base;
  int64_t n_tiles;
  int64_t copy_total;
  Lookback lb;
  uint32_t epoch;
  uint64_t ticket_base, done_base;
  int64_t *small;
};

// Ranks the set bits of one 2048-word tile within its node type and gives
// each new vertex its local ID.
__device__ void bitmap_tile(const CompactArgs &A, int64_t tile, int64_t *lds) {
  const int t = find_segment(A.tile_base, A.n_types, tile);
  const int64_t first = A.tile_base[t];
  uint32_t *w = A.bitmap + tile * kTile + threadIdx.x * kTileItems;
  const uint4 a = *reinterpret_cast<const uint4 *>(w);
  const uint4 b = *reinterpret_cast<const uint4 *>(w + 4);
  const uint32_t words[kTileItems] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
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
  *reinterpret_cast<uint4 *>(w) = uint4{0, 0, 0, 0};
  *reinterpret_cast<uint4 *>(w + 4) = uint4{0, 0, 0, 0};
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

// The next hop's frontier sizes and pair layout (run by the last block).
__device__ void plan_next_hop(const CompactArgs &A) {
  if (threadIdx.x != 0) return;
  for (int t = 0; t < A.n_types; ++t) {
    int64_t u = 0;
    if (A.tile_base[t + 1] > A.tile_base[t])
      u = __hip_atomic_load(A.small + kSlotNew + t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
      A.small[kSlotNew + t] = 0;
    A.next.nF[t] = A.hv.nF[t] + u;
  }
  int64_t acc = 0;
  for (int e = 0; e < A.n_etypes; ++e) {
    A.next.pair_base[e] = acc;
    acc += A.next.nF[A.es[e].dst_type];
  }
  A.next.pair_base[A.n_etypes] = acc;
}

__global__ __launch_bounds__(kTileThreads) void k_compact(CompactArgs A) {
  __shared__ int64_t lds[8];
  const int64_t tile = take_ticket(A.small, A.ticket_base, lds);
  if (tile < A.n_tiles)
    bitmap_tile(A, tile, lds);
  else
    copy_tile(A, tile - A.n_tiles);
  // the last block to finish plans the next hop
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0)
    lds[0] = int64_t(atomicAdd(reinterpret_cast<unsigned long long *>(A.small + kSlotDone),
                               1ull) - A.done_base) == int64_t(gridDim.x) - 1;
  __syncthreads();
  if (lds[0]) {
    __threadfence();
    plan_next_hop(A);
  }
}

__global__ void k_relabel(const EtypeStatic *es, const int64_t *ebase,
                          int32_t n_etypes, int64_t n_edges,
                          const int64_t *src_gid, int32_t *src_local) {
  for (int64_t j = gs_start(); j < n_edges; j += gs_step()) {
    const int e = find_segment(ebase, n_etypes, j);
    src_local[j] = es[e].src_map[src_gid[j]];
  }
}

}  // namespace

hipError_t launch_compact(HopView hv, HopView next, const TypeStatic *ts,
                          const EtypeStatic *es, int32_t n_types,
                          int32_t n_etypes, uint32_t *bitmap,
                          const int64_t *tile_base, int64_t n_tiles,
                          int64_t copy_total, Lookback lb, uint32_t epoch,
                          uint64_t ticket_base, uint64_t done_base,
                          int64_t *small, int32_t *blocks_launched,
                          hipStream_t stream) {
  CompactArgs A{hv, next, ts, es, n_types, n_etypes, bitmap, tile_base, n_tiles,
                copy_total, lb, epoch, ticket_base, done_base, small};
  const int64_t copy_blocks = (copy_total + kTile - 1) / kTile;
  int64_t blocks = n_tiles + copy_blocks;
  if (blocks < 1) blocks = 1;  // the plan always runs
  *blocks_launched = int32_t(blocks);
  hipLaunchKernelGGL(k_compact, dim3(unsigned(blocks)), dim3(kTileThreads), 0,
                     stream, A);
  return hipGetLastError();
}

hipError_t launch_relabel(const EtypeStatic *es, const int64_t *small,
                          int32_t n_types, int32_t n_etypes, int64_t n_edges,
                          const int64_t *src_gid, int32_t *src_local,
                          hipStream_t stream) {
  if (n_edges <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_relabel, dim3(grid_for(n_edges, 256)), dim3(256), 0,
                     stream, es, small + kSlotNew + n_types, n_etypes, n_edges,
                     src_gid, src_local);
  return hipGetLastError();
}

}  // namespace hg
