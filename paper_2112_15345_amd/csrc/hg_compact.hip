// Per-hop compaction on gfx950 (DistDGLv2, arXiv 2112.15345, Sec. 4.2.2: the
// frontier of the next hop is the unique set of this hop's vertices, and
// compaction relabels vertices and edges).
//
// The newly reached vertices of a node type are deduplicated and ordered by
// ID with one bit per vertex: the sampler sets bit v for every kept source v
// that is not in the frontier yet; a popcount scan over the bitmap then gives
// each set bit its rank, which is its position among the new vertices in
// ascending ID.  A dense int32 map (vertex -> local ID, -1 when absent) holds
// the local IDs of the frontier and of the new vertices for the relabel.
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

// One block per 2048-word tile; thread t reads words [8t, 8t+8).
__global__ __launch_bounds__(kTileThreads) void k_bm_tile_counts(
    const uint32_t *bitmap, int64_t *tile_cnt) {
  __shared__ int64_t lds[4];
  const uint32_t *w = bitmap + int64_t(blockIdx.x) * kTile + threadIdx.x * kTileItems;
  const uint4 a = *reinterpret_cast<const uint4 *>(w);
  const uint4 b = *reinterpret_cast<const uint4 *>(w + 4);
  int64_t s = __popc(a.x) + __popc(a.y) + __popc(a.z) + __popc(a.w) +
              __popc(b.x) + __popc(b.y) + __popc(b.z) + __popc(b.w);
  s = wave_sum_i64(s);
  if (lane_id() == 0) lds[threadIdx.x / kWave] = s;
  __syncthreads();
  if (threadIdx.x == 0) tile_cnt[blockIdx.x] = lds[0] + lds[1] + lds[2] + lds[3];
}

// One block: per node type, exclusive scan of its tiles' counts in place.
__global__ __launch_bounds__(kTileThreads) void k_bm_scan(
    int64_t *tile_cnt, const int64_t *tile_base, int32_t n_types,
    int64_t *n_new) {
  __shared__ int64_t lds[4];
  for (int t = 0; t < n_types; ++t) {
    const int64_t t0 = tile_base[t], t1 = tile_base[t + 1];
    int64_t carry = 0;
    for (int64_t base = t0; base < t1; base += kTile) {
      const int64_t b = base + threadIdx.x * kTileItems;
      int64_t v[kTileItems];
      int64_t s = 0;
#pragma unroll
      for (int k = 0; k < kTileItems; ++k) {
        v[k] = (b + k < t1) ? tile_cnt[b + k] : 0;
        s += v[k];
      }
      int64_t total;
      int64_t pre = block_excl_scan_256(s, lds, &total) + carry;
#pragma unroll
      for (int k = 0; k < kTileItems; ++k) {
        if (b + k < t1) tile_cnt[b + k] = pre;
        pre += v[k];
      }
      carry += total;
    }
    if (threadIdx.x == 0) n_new[t] = carry;
    __syncthreads();
  }
}

__global__ __launch_bounds__(kTileThreads) void k_bm_assign(
    uint32_t *bitmap, const int64_t *tile_cnt, const int64_t *tile_base,
    const HopNtype *types, int32_t n_types) {
  __shared__ int64_t lds[4];
  const int64_t tile = blockIdx.x;
  const int t = find_segment(tile_base, n_types, tile);
  uint32_t *w = bitmap + tile * kTile + threadIdx.x * kTileItems;
  uint4 a = *reinterpret_cast<const uint4 *>(w);
  uint4 b = *reinterpret_cast<const uint4 *>(w + 4);
  uint32_t words[kTileItems] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  int64_t s = 0;
#pragma unroll
  for (int k = 0; k < kTileItems; ++k) s += __popc(words[k]);
  int64_t total;
  const int64_t pre = block_excl_scan_256(s, lds, &total);
  if (total == 0) return;  // uniform over the block
  const HopNtype &T = types[t];
  int64_t local = T.n_frontier + tile_cnt[tile] + pre;
  // first vertex ID covered by this thread's first word
  const int64_t v0 = ((tile - tile_base[t]) * kTile + threadIdx.x * kTileItems) * 32;
#pragma unroll
  for (int k = 0; k < kTileItems; ++k) {
    uint32_t m = words[k];
    while (m) {
      const int bit = __ffs(m) - 1;
      m &= m - 1;
      const int64_t v = v0 + k * 32 + bit;
      T.map[v] = int32_t(local);
      T.src_out[local] = v;
      ++local;
    }
  }
  if (s) {
    *reinterpret_cast<uint4 *>(w) = uint4{0, 0, 0, 0};
    *reinterpret_cast<uint4 *>(w + 4) = uint4{0, 0, 0, 0};
  }
}

__global__ void k_copy_frontier(const HopNtype *types, const int64_t *type_base,
                                int32_t n_types, int64_t total) {
  for (int64_t x = gs_start(); x < total; x += gs_step()) {
    const int t = find_segment(type_base, n_types, x);
    const int64_t i = x - type_base[t];
    types[t].src_out[i] = types[t].frontier[i];
  }
}

__global__ void k_relabel(const HopEtype *et, const int64_t *ebase,
                          int32_t n_etypes, int64_t n_edges,
                          const int64_t *src_gid, int32_t *src_local) {
  for (int64_t j = gs_start(); j < n_edges; j += gs_step()) {
    const int e = find_segment(ebase, n_etypes, j);
    src_local[j] = et[e].src_map[src_gid[j]];
  }
}

}  // namespace

hipError_t launch_bitmap_tile_counts(const uint32_t *bitmap, int64_t n_tiles,
                                     int64_t *tile_cnt, hipStream_t stream) {
  if (n_tiles <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_bm_tile_counts, dim3(unsigned(n_tiles)), dim3(kTileThreads),
                     0, stream, bitmap, tile_cnt);
  return hipGetLastError();
}

hipError_t launch_bitmap_scan(int64_t *tile_cnt, const int64_t *tile_base,
                              int32_t n_types, int64_t *n_new,
                              hipStream_t stream) {
  hipLaunchKernelGGL(k_bm_scan, dim3(1), dim3(kTileThreads), 0, stream, tile_cnt,
                     tile_base, n_types, n_new);
  return hipGetLastError();
}

hipError_t launch_bitmap_assign(uint32_t *bitmap, int64_t n_tiles,
                                const int64_t *tile_cnt,
                                const int64_t *tile_base, const HopNtype *types,
                                int32_t n_types, hipStream_t stream) {
  if (n_tiles <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_bm_assign, dim3(unsigned(n_tiles)), dim3(kTileThreads), 0,
                     stream, bitmap, tile_cnt, tile_base, types, n_types);
  return hipGetLastError();
}

hipError_t launch_copy_frontier(const HopNtype *types, const int64_t *type_base,
                                int32_t n_types, int64_t total,
                                hipStream_t stream) {
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_copy_frontier, dim3(grid_for(total, 256)), dim3(256), 0,
                     stream, types, type_base, n_types, total);
  return hipGetLastError();
}

hipError_t launch_relabel(const HopEtype *et, const int64_t *ebase,
                          int32_t n_etypes, int64_t n_edges,
                          const int64_t *src_gid, int32_t *src_local,
                          hipStream_t stream) {
  if (n_edges <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_relabel, dim3(grid_for(n_edges, 256)), dim3(256), 0,
                     stream, et, ebase, n_etypes, n_edges, src_gid, src_local);
  return hipGetLastError();
}

}  // namespace hg
