// Per-hop neighbour sampling on gfx950: pair counting, device-wide scan and the
// fanout sampler (DistDGLv2, arXiv 2112.15345, Sec. 3.2 and Sec. 4.2.2).
//
// A "pair" is (frontier vertex v of the destination type, edge type e).  Each
// pair keeps min(deg, K) of its in-edges: all of them when deg <= K (or
// K == -1), else the K with the smallest (key, edge ID), where the key of edge
// `eid` is word (eid & 3) of Philox4x32-10 at counter (eid >> 2, hop, e) under
// the sampling seed.  Kept edges are written grouped by pair, ascending edge
// ID within a pair.
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

// ---- frontier map maintenance --------------------------------------------

__global__ void k_insert_frontier(const HopNtype *types, const int64_t *type_base,
                                  int32_t n_types, int64_t total, int32_t *err) {
  for (int64_t x = grid_stride_start(); x < total; x += grid_stride_step()) {
    const int t = find_segment(type_base, n_types, x);
    const int64_t i = x - type_base[t];
    const int64_t v = types[t].frontier[i];
    if (v < 0 || v >= types[t].num_nodes) {
      atomicOr(err, 1);
      continue;
    }
    const int old = atomicCAS(&types[t].map[v], -1, int(i));
    if (old != -1) atomicOr(err, 2);
  }
}

__global__ void k_reset_map(const HopNtype *types, const int64_t *type_base,
                            int32_t n_types, int64_t total) {
  for (int64_t x = grid_stride_start(); x < total; x += grid_stride_step()) {
    const int t = find_segment(type_base, n_types, x);
    const int64_t v = types[t].frontier[x - type_base[t]];
    if (v >= 0 && v < types[t].num_nodes) types[t].map[v] = -1;
  }
}

// ---- pair counting -------------------------------------------------------

__global__ void k_count(const HopEtype *et, const int64_t *pair_base,
                        int32_t n_etypes, int64_t n_pairs, int64_t *cnt,
                        int64_t *plo, int64_t *pdeg, int32_t *err) {
  for (int64_t p = grid_stride_start(); p < n_pairs; p += grid_stride_step()) {
    const int e = find_segment(pair_base, n_etypes, p);
    const HopEtype &E = et[e];
    const int64_t v = E.frontier[p - E.pair_base];
    int64_t lo = 0, deg = 0;
    if (v >= 0 && v < E.n_dst_nodes) {
      lo = E.indptr[v];
      deg = E.indptr[v + 1] - lo;
    } else {
      atomicOr(err, 1);
    }
    const int64_t k = E.fanout;
    cnt[p] = (k < 0 || deg <= k) ? deg : k;
    plo[p] = lo;
    pdeg[p] = deg;
  }
}

// ---- device-wide exclusive scan (reduce, scan tile sums, down-sweep) -----

__global__ __launch_bounds__(kTileThreads) void k_scan_reduce(
    const int64_t *in, int64_t n, int64_t *tile_sum) {
  __shared__ int64_t lds[4];
  const int64_t base = int64_t(blockIdx.x) * kTile + threadIdx.x * kTileItems;
  int64_t s = 0;
#pragma unroll
  for (int k = 0; k < kTileItems; ++k)
    if (base + k < n) s += in[base + k];
  s = wave_sum_i64(s);
  if (lane_id() == 0) lds[threadIdx.x / kWave] = s;
  __syncthreads();
  if (threadIdx.x == 0) tile_sum[blockIdx.x] = lds[0] + lds[1] + lds[2] + lds[3];
}

// One block: exclusive scan of ts[0..nt) in place, ts[nt] = total.
__global__ __launch_bounds__(kTileThreads) void k_scan_tiles(int64_t *ts,
                                                             int64_t nt) {
  __shared__ int64_t lds[4];
  int64_t carry = 0;
  for (int64_t base = 0; base < nt; base += kTile) {
    const int64_t b = base + threadIdx.x * kTileItems;
    int64_t v[kTileItems];
    int64_t s = 0;
#pragma unroll
    for (int k = 0; k < kTileItems; ++k) {
      v[k] = (b + k < nt) ? ts[b + k] : 0;
      s += v[k];
    }
    int64_t total;
    int64_t pre = block_excl_scan_256(s, lds, &total) + carry;
#pragma unroll
    for (int k = 0; k < kTileItems; ++k) {
      if (b + k < nt) ts[b + k] = pre;
      pre += v[k];
    }
    carry += total;
  }
  if (threadIdx.x == 0) ts[nt] = carry;
}

__global__ __launch_bounds__(kTileThreads) void k_scan_down(
    const int64_t *in, int64_t n, const int64_t *ts, int64_t nt, int64_t *out) {
  __shared__ int64_t lds[4];
  const int64_t b = int64_t(blockIdx.x) * kTile + threadIdx.x * kTileItems;
  int64_t v[kTileItems];
  int64_t s = 0;
#pragma unroll
  for (int k = 0; k < kTileItems; ++k) {
    v[k] = (b + k < n) ? in[b + k] : 0;
    s += v[k];
  }
  int64_t total;
  int64_t pre = block_excl_scan_256(s, lds, &total) + ts[blockIdx.x];
#pragma unroll
  for (int k = 0; k < kTileItems; ++k) {
    if (b + k < n) out[b + k] = pre;
    pre += v[k];
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) out[n] = ts[nt];
}

__global__ void k_set_i64(int64_t *p, int64_t v) { *p = v; }

__global__ void k_edge_bases(const int64_t *pair_base, const int64_t *off,
                             int32_t n_etypes, int64_t *ebase) {
  for (int64_t e = grid_stride_start(); e <= n_etypes; e += grid_stride_step())
    ebase[e] = off[pair_base[e]];
}

// ---- the sampler -----------------------------------------------------------

struct EmitCtx {
  const int64_t *indices;
  const int32_t *src_map;
  uint32_t *src_bitmap;
  int64_t *src_gid;
  int64_t *eid;
  int32_t *dst_local;
  int32_t dst;
};

// Writes kept edge `e` at output slot `pos` and marks its source as new when
// it is not in the frontier of its type yet.
__device__ __forceinline__ void emit_edge(const EmitCtx &c, int64_t pos,
                                          int64_t e) {
  const int64_t g = c.indices[e];
  c.src_gid[pos] = g;
  c.eid[pos] = e;
  c.dst_local[pos] = c.dst;
  if (c.src_map[g] < 0) {
    uint32_t *w = c.src_bitmap + (g >> 5);
    const uint32_t bit = 1u << (g & 31);
    if ((*w & bit) == 0) atomicOr(w, bit);
  }
}

// Keys of the four edges 4g .. 4g+3.
__device__ __forceinline__ U32x4 edge_keys(uint64_t g, int32_t hop, int32_t e,
                                           uint32_t k0, uint32_t k1,
                                           uint32_t shift) {
  U32x4 r = philox4x32_10(
      U32x4{uint32_t(g), uint32_t(g >> 32), uint32_t(hop), uint32_t(e)}, k0, k1);
  r.x >>= shift;
  r.y >>= shift;
  r.z >>= shift;
  r.w >>= shift;
  return r;
}

__device__ __forceinline__ uint32_t word_of(const U32x4 &r, int w) {
  return w == 0 ? r.x : (w == 1 ? r.y : (w == 2 ? r.z : r.w));
}

constexpr int kSampleWaves = 4;

__global__ __launch_bounds__(kSampleWaves *kWave) void k_sample(
    const HopEtype *et, const int64_t *pair_base, int32_t n_etypes,
    int64_t n_pairs, const int64_t *cnt, const int64_t *plo,
    const int64_t *pdeg, const int64_t *off, uint64_t sigma, int32_t hop,
    int32_t key_bits, int64_t *src_gid, int64_t *eid_out, int32_t *dst_local) {
  __shared__ uint32_t s_key[kSampleWaves][kCandCap];
  __shared__ uint32_t s_j[kSampleWaves][kCandCap];
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int64_t p = int64_t(blockIdx.x) * kSampleWaves + wave;
  if (p >= n_pairs) return;
  const int64_t s = cnt[p];
  if (s == 0) return;
  const int e = find_segment(pair_base, n_etypes, p);
  EmitCtx c;
  c.indices = et[e].indices;
  c.src_map = et[e].src_map;
  c.src_bitmap = et[e].src_bitmap;
  c.src_gid = src_gid;
  c.eid = eid_out;
  c.dst_local = dst_local;
  c.dst = int32_t(p - et[e].pair_base);
  const int64_t lo = plo[p];
  const int64_t deg = pdeg[p];
  const int64_t o = off[p];

  if (s == deg) {  // every in-edge is kept
    for (int64_t j = lane; j < deg; j += kWave) emit_edge(c, o + j, lo + j);
    return;
  }

  // ---- keep the K = s in-edges with the smallest (key, edge ID) ----------
  const int K = int(s);
  const uint32_t shift = uint32_t(32 - key_bits);
  const uint64_t key_space = uint64_t(1) << key_bits;
  const uint32_t k0 = uint32_t(sigma), k1 = uint32_t(sigma >> 32);
  const uint64_t g_first = uint64_t(lo) >> 2;
  const uint64_t g_last = uint64_t(lo + deg - 1) >> 2;
  const uint64_t hi = uint64_t(lo + deg);

  // Pass 1: keys are uniform, so about deg * tau / 2^bits of them fall below
  // tau; tau is set for K + 4 sqrt(K) + 16 expected candidates.  Candidates
  // (key < tau) are appended in edge order to this wave's LDS list.
  uint64_t tau = uint64_t(
      ceil((double(K) + 4.0 * sqrt(double(K)) + 16.0) / double(deg) *
           double(key_space)));
  if (tau < 1) tau = 1;
  if (tau > key_space) tau = key_space;
  uint32_t *ck = s_key[wave];
  uint32_t *cj = s_j[wave];
  int64_t n_cand = 0;
  for (uint64_t gb = g_first; gb <= g_last; gb += kWave) {
    const uint64_t g = gb + lane;
    int mask = 0;
    U32x4 r{0, 0, 0, 0};
    if (g <= g_last) {
      r = edge_keys(g, hop, e, k0, k1, shift);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint64_t ed = 4 * g + w;
        if (ed >= uint64_t(lo) && ed < hi && uint64_t(word_of(r, w)) < tau)
          mask |= 1 << w;
      }
    }
    int tot;
    int64_t pos = n_cand + wave_prefix_small(__popc(mask), &tot);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      if (mask & (1 << w)) {
        if (pos < kCandCap) {
          ck[pos] = word_of(r, w);
          cj[pos] = uint32_t(4 * g + w - uint64_t(lo));
        }
        ++pos;
      }
    }
    n_cand += tot;
  }
  wave_sync();

  if (n_cand >= K && n_cand <= kCandCap) {
    // The K smallest all lie among the candidates: rank each candidate by
    // counting smaller (key, j) pairs, keep ranks < K, in list (edge) order.
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

  // Exact fallback (too few or too many candidates): bisect the composite
  // (key << 32 | j) for the K-th smallest value T, then keep every edge with
  // composite <= T, in edge order.
  uint64_t a = 0;
  uint64_t b = ((key_space - 1) << 32) | uint64_t(deg - 1);
  if (tau < key_space) {
    if (n_cand >= K)
      b = min(b, (tau << 32) - 1);
    else
      a = tau << 32;
  }
  while (a < b) {
    const uint64_t mid = a + ((b - a) >> 1);
    int64_t le = 0;
    for (uint64_t gb = g_first; gb <= g_last; gb += kWave) {
      const uint64_t g = gb + lane;
      if (g > g_last) continue;
      const U32x4 r = edge_keys(g, hop, e, k0, k1, shift);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint64_t ed = 4 * g + w;
        if (ed >= uint64_t(lo) && ed < hi &&
            ((uint64_t(word_of(r, w)) << 32) | (ed - uint64_t(lo))) <= mid)
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
      const U32x4 r = edge_keys(g, hop, e, k0, k1, shift);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint64_t ed = 4 * g + w;
        if (ed >= uint64_t(lo) && ed < hi &&
            ((uint64_t(word_of(r, w)) << 32) | (ed - uint64_t(lo))) <= T)
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

// ---- block CSC -------------------------------------------------------------

// Segment starts of the per-etype indptr arrays: st[e] = pair_base[e] + e.
__device__ __forceinline__ int find_indptr_segment(const int64_t *pair_base,
                                                   int n, int64_t x) {
  int lo = 0, hi = n;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (pair_base[mid] + mid <= x)
      lo = mid;
    else
      hi = mid;
  }
  return lo;
}

__global__ void k_block_indptr(const int64_t *pair_base, const int64_t *off,
                               int32_t n_etypes, int64_t total,
                               int64_t *indptr_all) {
  for (int64_t q = grid_stride_start(); q < total; q += grid_stride_step()) {
    const int e = find_indptr_segment(pair_base, n_etypes, q);
    const int64_t first = pair_base[e];
    const int64_t i = q - (first + e);
    indptr_all[q] = off[first + i] - off[first];
  }
}

// ---- small utilities -------------------------------------------------------

__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v) {
  for (int64_t i = grid_stride_start(); i < n; i += grid_stride_step()) p[i] = v;
}
__global__ void k_fill_u32(uint32_t *p, int64_t n, uint32_t v) {
  for (int64_t i = grid_stride_start(); i < n; i += grid_stride_step()) p[i] = v;
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

}  // namespace

// ---- launchers ---------------------------------------------------------------

hipError_t launch_insert_frontier(const HopNtype *types, const int64_t *type_base,
                                  int32_t n_types, int64_t total, int32_t *err,
                                  hipStream_t stream) {
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_insert_frontier, dim3(grid_for(total, 256)), dim3(256), 0,
                     stream, types, type_base, n_types, total, err);
  return hipGetLastError();
}

hipError_t launch_reset_map(const HopNtype *types, const int64_t *type_base,
                            int32_t n_types, int64_t total, hipStream_t stream) {
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_reset_map, dim3(grid_for(total, 256)), dim3(256), 0,
                     stream, types, type_base, n_types, total);
  return hipGetLastError();
}

hipError_t launch_count(const HopEtype *et, const int64_t *pair_base,
                        int32_t n_etypes, int64_t n_pairs, int64_t *cnt,
                        int64_t *plo, int64_t *pdeg, int32_t *err,
                        hipStream_t stream) {
  if (n_pairs <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_count, dim3(grid_for(n_pairs, 256)), dim3(256), 0, stream,
                     et, pair_base, n_etypes, n_pairs, cnt, plo, pdeg, err);
  return hipGetLastError();
}

int64_t scan_scratch_elems(int64_t n) { return (n + kTile - 1) / kTile + 1; }

hipError_t launch_scan_i64(const int64_t *in, int64_t n, int64_t *out,
                           int64_t *scratch, hipStream_t stream) {
  if (n <= 0) {
    hipLaunchKernelGGL(k_set_i64, dim3(1), dim3(1), 0, stream, out, int64_t(0));
    return hipGetLastError();
  }
  const int64_t nt = (n + kTile - 1) / kTile;
  hipLaunchKernelGGL(k_scan_reduce, dim3(unsigned(nt)), dim3(kTileThreads), 0,
                     stream, in, n, scratch);
  hipLaunchKernelGGL(k_scan_tiles, dim3(1), dim3(kTileThreads), 0, stream,
                     scratch, nt);
  hipLaunchKernelGGL(k_scan_down, dim3(unsigned(nt)), dim3(kTileThreads), 0,
                     stream, in, n, scratch, nt, out);
  return hipGetLastError();
}

hipError_t launch_edge_bases(const int64_t *pair_base, const int64_t *off,
                             int32_t n_etypes, int64_t *ebase,
                             hipStream_t stream) {
  hipLaunchKernelGGL(k_edge_bases, dim3(grid_for(n_etypes + 1, 256)), dim3(256),
                     0, stream, pair_base, off, n_etypes, ebase);
  return hipGetLastError();
}

hipError_t launch_sample(const HopEtype *et, const int64_t *pair_base,
                         int32_t n_etypes, int64_t n_pairs, const int64_t *cnt,
                         const int64_t *plo, const int64_t *pdeg,
                         const int64_t *off, uint64_t sigma, int32_t hop,
                         int32_t key_bits, int64_t *src_gid, int64_t *eid,
                         int32_t *dst_local, hipStream_t stream) {
  if (n_pairs <= 0) return hipSuccess;
  const int64_t blocks = (n_pairs + kSampleWaves - 1) / kSampleWaves;
  hipLaunchKernelGGL(k_sample, dim3(unsigned(blocks)), dim3(kSampleWaves * kWave),
                     0, stream, et, pair_base, n_etypes, n_pairs, cnt, plo, pdeg,
                     off, sigma, hop, key_bits, src_gid, eid, dst_local);
  return hipGetLastError();
}

hipError_t launch_block_indptr(const int64_t *pair_base, const int64_t *off,
                               int32_t n_etypes, int64_t n_pairs,
                               int64_t *indptr_all, hipStream_t stream) {
  const int64_t total = n_pairs + n_etypes;
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_block_indptr, dim3(grid_for(total, 256)), dim3(256), 0,
                     stream, pair_base, off, n_etypes, total, indptr_all);
  return hipGetLastError();
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

hipError_t launch_check_etype(const int64_t *indptr, int64_t n_dst,
                              const int64_t *indices, int64_t nnz,
                              int64_t n_src, int32_t *err, hipStream_t stream) {
  const int64_t n = n_dst > nnz ? n_dst : nnz;
  hipLaunchKernelGGL(k_check_etype, dim3(grid_for(n, 256, 8192)), dim3(256), 0,
                     stream, indptr, n_dst, indices, nnz, n_src, err);
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
