// Internal interface between the host runtime (hg_runtime.cpp) and the gfx950
// kernels (hg_sample.hip, hg_compact.hip, hg_gather.hip).  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace hg {

// Items of one scan / bitmap tile: 256 threads x 8 items.
constexpr int kTileThreads = 256;
constexpr int kTileItems = 8;
constexpr int64_t kTile = int64_t(kTileThreads) * kTileItems;  // 2048

// Candidate capacity of one wavefront's bottom-K selection (LDS entries).
constexpr int kCandCap = 512;

// Per hop, per edge type: where the pairs (frontier vertex of the
// destination type x edge type) of this edge type sit and what they read.
struct HopEtype {
  const int64_t *frontier;  // frontier of dst_type at this hop (device)
  const int64_t *indptr;    // CSC of the edge type
  const int64_t *indices;
  int32_t *src_map;         // dense vertex -> local-ID map of src_type
  uint32_t *src_bitmap;     // new-vertex bitmap of src_type
  int64_t pair_base;        // global index of this etype's first pair
  int64_t n_pairs;          // frontier size of dst_type
  int64_t n_dst_nodes;      // vertex count of dst_type (range check)
  int32_t fanout;           // -1 = all
  int32_t src_type;
};

// Per hop, per node type.
struct HopNtype {
  const int64_t *frontier;  // current frontier (device)
  int64_t n_frontier;
  int64_t num_nodes;
  int32_t *map;             // dense map of the type
  int64_t *src_out;         // source list being built (frontier ++ new)
  int64_t new_base;         // running offset of this type in a concatenation
};

// ---- launchers (all asynchronous on `stream`) -------------------------------

// Seeds of hop 0: map[seed] = position; flags an out-of-range or repeated seed.
hipError_t launch_insert_frontier(const HopNtype *types, const int64_t *type_base,
                                  int32_t n_types, int64_t total, int32_t *err,
                                  hipStream_t stream);
// map[v] = -1 for every vertex of the given lists (in-range entries only).
hipError_t launch_reset_map(const HopNtype *types, const int64_t *type_base,
                            int32_t n_types, int64_t total, hipStream_t stream);

// Per pair: its kept-edge count min(deg, K) (deg if K == -1), its first slot
// and its degree.
hipError_t launch_count(const HopEtype *et, const int64_t *pair_base,
                        int32_t n_etypes, int64_t n_pairs, int64_t *cnt,
                        int64_t *plo, int64_t *pdeg, int32_t *err,
                        hipStream_t stream);

// out[0..n] = exclusive prefix sums of in[0..n-1]; out[n] = total.
// `scratch` holds at least scan_scratch_elems(n) int64.
int64_t scan_scratch_elems(int64_t n);
hipError_t launch_scan_i64(const int64_t *in, int64_t n, int64_t *out,
                           int64_t *scratch, hipStream_t stream);

// ebase[e] = off[pair_base[e]] for e <= n_etypes (edge start of each etype).
hipError_t launch_edge_bases(const int64_t *pair_base, const int64_t *off,
                             int32_t n_etypes, int64_t *ebase,
                             hipStream_t stream);

// The sampler: one wavefront per pair, writes the kept edges of the pair at
// off[p]: source vertex, edge ID and destination local ID, and marks sources
// that are not yet in the frontier in the bitmap.
hipError_t launch_sample(const HopEtype *et, const int64_t *pair_base,
                         int32_t n_etypes, int64_t n_pairs, const int64_t *cnt,
                         const int64_t *plo, const int64_t *pdeg,
                         const int64_t *off, uint64_t sigma, int32_t hop,
                         int32_t key_bits, int64_t *src_gid, int64_t *eid,
                         int32_t *dst_local, hipStream_t stream);

// Block CSC per etype: indptr_all[pair_base[e] + e + i] =
//   off[pair_base[e] + i] - off[pair_base[e]],  i = 0..n_pairs(e).
hipError_t launch_block_indptr(const int64_t *pair_base, const int64_t *off,
                               int32_t n_etypes, int64_t n_pairs,
                               int64_t *indptr_all, hipStream_t stream);

// Popcount of each 2048-word bitmap tile.
hipError_t launch_bitmap_tile_counts(const uint32_t *bitmap, int64_t n_tiles,
                                     int64_t *tile_cnt, hipStream_t stream);
// Per node type t owning tiles [tile_base[t], tile_base[t+1]): exclusive scan
// of its tile counts in place; n_new[t] = its total.
hipError_t launch_bitmap_scan(int64_t *tile_cnt, const int64_t *tile_base,
                              int32_t n_types, int64_t *n_new,
                              hipStream_t stream);
// For every set bit v of type t: local = n_frontier[t] + rank; map[v] = local;
// src_out[local] = v; clears the tile.
hipError_t launch_bitmap_assign(uint32_t *bitmap, int64_t n_tiles,
                                const int64_t *tile_cnt,
                                const int64_t *tile_base, const HopNtype *types,
                                int32_t n_types, hipStream_t stream);
// src_out[i] = frontier[i] for every type (the destination prefix).
hipError_t launch_copy_frontier(const HopNtype *types, const int64_t *type_base,
                                int32_t n_types, int64_t total,
                                hipStream_t stream);
// src_local[j] = map_{src_type(e)}[src_gid[j]] for the edges of etype e,
// which are [ebase[e], ebase[e+1]).
hipError_t launch_relabel(const HopEtype *et, const int64_t *ebase,
                          int32_t n_etypes, int64_t n_edges,
                          const int64_t *src_gid, int32_t *src_local,
                          hipStream_t stream);

// Fill helpers (kernels, so that they are safe under graph capture).
hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t stream);
hipError_t launch_fill_u32(uint32_t *p, int64_t n, uint32_t v, hipStream_t stream);

// Graph check of one edge type: indptr[0] == 0, non-decreasing,
// indptr[n_dst] == nnz, indices in [0, n_src).  Sets *err on a violation.
hipError_t launch_check_etype(const int64_t *indptr, int64_t n_dst,
                              const int64_t *indices, int64_t nnz,
                              int64_t n_src, int32_t *err, hipStream_t stream);

// Row gather: out[i] = table[ids[i]] (row_bytes bytes), zero row when out of
// range.  Picks the widest vector width that divides row_bytes and the
// alignment of both pointers.
hipError_t launch_gather(const void *table, int64_t n_rows, int64_t row_bytes,
                         const int64_t *ids, int64_t n, void *out,
                         hipStream_t stream);

// Philox4x32-10 on n counters.
hipError_t launch_philox(const uint32_t *ctr, uint64_t key, int64_t n,
                         uint32_t *out, hipStream_t stream);

}  // namespace hg
