// Edge-seeded mini-batches on gfx950 (link prediction).  DistDGLv2 (arXiv
// 2112.15345) lets its scheduler pick target edges as well as target vertices
// (Sec. 4.2.1) and runs the same sampling decomposition from them (Sec.
// 4.2.2).  The targets' endpoints become the seeds:
//  1. k_edge_targets: a wavefront per target edge: its source (indices[eid])
//     and its destination (the vertex whose in-edge slots hold eid, by a
//     64-ary search over indptr), its negative destinations (one per lane) (Philox4x32-10 at counter
//     (eid, 2^31 | k, etype), words 0 and 1 as u, destination
//     floor(u * n / 2^64)), and its reverse edge under exclusion 2 (checked
//     to run the other way).  Every endpoint sets its reached flag.
//  2. The compaction pass of the hops (hg_compact.hip) then ranks the reached
//     vertices from an empty frontier: the seeds of each type in ascending
//     ID, with their local IDs in the map.
//  3. k_edge_relabel: the pair graphs' local IDs, the exclusion hash tables
//     (the excluded edges, and per pair with excluded in-edges their number),
//     and hop 0's frontier sizes and pair layout.
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

unsigned grid_for(int64_t n, int threads, int64_t cap = 1 << 16) {
  int64_t b = (n + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return unsigned(b);
}

// The destination of CSC slot eid: the largest v in [0, n_dst) with
// indptr[v] <= eid (for 0 <= eid < indptr[n_dst]).  Searched by a wavefront:
// every lane probes one of 64 positions per round, so about log64(n_dst)
// dependent loads instead of log2(n_dst).  All lanes take part and get the
// result.
__device__ int64_t wave_edge_dst(const int64_t *indptr, int64_t n_dst, int64_t eid) {
  const int lane = lane_id();
  int64_t a = 0, b = n_dst;  // indptr[a] <= eid; the answer is in [a, b)
  while (b - a > 1) {
    const int64_t step = (b - a + kWave - 1) / kWave;
    const int64_t pos = a + int64_t(lane) * step;
    // true on a prefix of the lanes (indptr never decreases), lane 0 always
    const uint64_t bal = __ballot(pos < b && indptr[pos] <= eid);
    const int last = 63 - __clzll((unsigned long long)bal);
    a += int64_t(last) * step;
    b = min(b, a + step);
  }
  return a;
}

__device__ __forceinline__ void mark(uint8_t *reached, int64_t v) { reached[v] = 1; }

__device__ __forceinline__ void flag(int64_t *small, int32_t bits) {
  atomicOr(reinterpret_cast<int32_t *>(small + kSlotErr), bits);
}

// A wavefront per target (the target index is the same on all its lanes).
__global__ __launch_bounds__(256) void k_edge_targets(EdgeBatchArgs A) {
  const int lane = lane_id();
  const int64_t waves = int64_t(gridDim.x) * (blockDim.x / kWave);
  for (int64_t x = gs_start() / kWave; x < A.n_targets; x += waves) {
    const int e = find_segment(A.tbase, A.n_etypes, x);
    const EdgeEtype &T = A.et[e];
    const EtypeStatic &E = A.es[e];
    const int64_t j = T.eids[x - A.tbase[e]];
    if (lane == 0) {
      A.tsrc[x] = -1;
      A.tdst[x] = -1;
      A.trev[x] = -1;
    }
    if (lane < A.n_neg) A.tneg[x * A.n_neg + lane] = -1;
    if (j < 0 || j >= T.nnz) {
      if (lane == 0) flag(A.small, kErrTarget);
      continue;
    }
    const int64_t u = E.indices[j];
    const int64_t v = wave_edge_dst(E.indptr, E.n_dst_nodes, j);
    if (lane == 0) {
      A.tsrc[x] = u;
      A.tdst[x] = v;
      mark(E.src_reached, u);
      mark(A.ts[E.dst_type].reached, v);
    }
    if (lane < A.n_neg) {  // negative k = lane
      const int copy = e / A.key_R;
      const uint64_t sigma = A.sigmas[copy];
      const U32x4 r = philox4x32_10(U32x4{uint32_t(j), uint32_t(uint64_t(j) >> 32),
                                          0x80000000u | uint32_t(lane), uint32_t(e - copy * A.key_R)},
                                    uint32_t(sigma), uint32_t(sigma >> 32));
      const uint64_t w = uint64_t(r.x) | (uint64_t(r.y) << 32);
      const int64_t nv = int64_t(__umul64hi(w, uint64_t(E.n_dst_nodes)));
      A.tneg[x * A.n_neg + lane] = nv;
      mark(A.ts[E.dst_type].reached, nv);
    }
    if (A.exclude == 2 && T.rev >= 0) {
      // the reverse edge must run from v back to u in the reverse type
      const int64_t rj = T.rev_eid[j];
      const EdgeEtype &RT = A.et[T.rev];
      const EtypeStatic &RE = A.es[T.rev];
      if (rj < 0 || rj >= RT.nnz || RE.indices[rj] != v ||
          wave_edge_dst(RE.indptr, RE.n_dst_nodes, rj) != u) {
        if (lane == 0) flag(A.small, kErrTarget);
        continue;
      }
      if (lane == 0) A.trev[x] = rj;
    }
  }
}

// Inserts `key` into the edge table; true when it was not there yet.
__device__ bool edge_insert(const EdgeBatchArgs &A, uint64_t key) {
  for (uint32_t h = hash_slot(key, A.edge_mask);; h = (h + 1) & A.edge_mask) {
    const uint64_t prev = atomicCAS(reinterpret_cast<unsigned long long *>(A.edge_keys + h),
                                    (unsigned long long)kHashEmpty, (unsigned long long)key);
    if (prev == kHashEmpty) return true;
    if (prev == key) return false;
  }
}

// Adds one excluded in-edge to the pair `key`.
__device__ void pair_add(const EdgeBatchArgs &A, uint64_t key) {
  for (uint32_t h = hash_slot(key, A.pair_mask);; h = (h + 1) & A.pair_mask) {
    const uint64_t prev = atomicCAS(reinterpret_cast<unsigned long long *>(A.pair_keys + h),
                                    (unsigned long long)kHashEmpty, (unsigned long long)key);
    if (prev == kHashEmpty || prev == key) {
      atomicAdd(A.pair_cnt + h, 1);
      return;
    }
  }
}

__device__ __forceinline__ uint64_t hkey(int e, int64_t v) {
  return (uint64_t(uint32_t(e)) << 32) | uint64_t(uint32_t(v));
}

__global__ __launch_bounds__(256) void k_edge_relabel(EdgeBatchArgs A, HopView first,
                                                      const int64_t *tile_base) {
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    // hop 0: the seeds are the frontier; pairs of etype e are its
    // destination type's seeds
    for (int t = 0; t < A.n_types; ++t)
      first.nF[t] = tile_base[t + 1] > tile_base[t] ? A.small[kSlotNew + t] : 0;
    int64_t acc = 0;
    for (int e = 0; e < A.n_etypes; ++e) {
      const int64_t n = first.nF[A.es[e].dst_type];
      first.pair_base[e] = acc;
      A.n_seed[e] = n;
      acc += n;
    }
    first.pair_base[A.n_etypes] = acc;
  }
  for (int64_t x = gs_start(); x < A.n_targets; x += gs_step()) {
    const int e = find_segment(A.tbase, A.n_etypes, x);
    const EtypeStatic &E = A.es[e];
    const int64_t u = A.tsrc[x], v = A.tdst[x];
    if (u < 0) continue;  // an invalid target: the call fails
    const int32_t lu = E.src_map[u];
    const int32_t lv = A.ts[E.dst_type].map[v];
    A.pos_src[x] = lu;
    A.pos_dst[x] = lv;
    for (int k = 0; k < A.n_neg; ++k)
      A.neg_dst[x * A.n_neg + k] = A.ts[E.dst_type].map[A.tneg[x * A.n_neg + k]];
    if (A.exclude >= 1) {
      const int64_t j = A.et[e].eids[x - A.tbase[e]];
      if (edge_insert(A, hkey(e, j))) pair_add(A, hkey(e, lv));
      const int64_t rj = A.trev[x];
      if (A.exclude == 2 && rj >= 0) {
        // the reverse edge ends at u, a seed of the reverse type's destination type
        const int r = A.et[e].rev;
        if (edge_insert(A, hkey(r, rj))) pair_add(A, hkey(r, lu));
      }
    }
  }
}

}  // namespace

hipError_t launch_edge_targets(const EdgeBatchArgs &A, hipStream_t stream) {
  if (A.n_targets <= 0) return hipSuccess;
  // a wavefront per target
  hipLaunchKernelGGL(k_edge_targets, dim3(grid_for(A.n_targets * kWave, 256)), dim3(256), 0, stream,
                     A);
  return hipGetLastError();
}

hipError_t launch_edge_relabel(const EdgeBatchArgs &A, HopView first,
                               const int64_t *tile_base, hipStream_t stream) {
  // at least one block: block 0 plans hop 0
  hipLaunchKernelGGL(k_edge_relabel, dim3(grid_for(A.n_targets, 256)), dim3(256), 0, stream, A,
                     first, tile_base);
  return hipGetLastError();
}

}  // namespace hg
