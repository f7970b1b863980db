// Feature gather on gfx950: out[i, :] = table[ids[i], :], bits copied
// unchanged.  This is the feature-copy stage of DistDGLv2's mini-batch
// pipeline (arXiv 2112.15345, Sec. 4.2.1), done as a copy inside HBM: the
// rows of the input frontier are read from the per-type table and written
// contiguously.
//
// Each lane moves one vector (16 bytes when the row size and both pointers
// allow it) of a row; a block covers several rows per pass and keeps kUnroll
// passes of loads in flight before storing.  Stores bypass the caches
// (non-temporal), since the output is not re-read by this kernel.
#include <hip/hip_ext.h>

#include <map>
#include <mutex>

#include "hg_device.hpp"
#include "hg_internal.hpp"

namespace hg {

// Scratch of the allocation-free row pull (hg_gather_rows_noalloc): the count
// of out-of-range IDs of the call running on this GPU.  Every GPU the library
// runs on holds its own copy until the process ends.  Host code never uses
// this name as an address: it uses the per-device address that
// hipGetSymbolAddress gives (noalloc_scratch_init).
static __device__ __align__(256) unsigned long long scratch[kNoAllocScratchBytes / 8];

namespace {
std::mutex g_scratch_mu;
std::map<int, unsigned long long *> g_scratch_ptr;  // device -> address of `scratch`
}  // namespace

hipError_t noalloc_scratch_init(int device) {
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr.count(device)) return hipSuccess;
  void *p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess || !p) return e != hipSuccess ? e : hipErrorInvalidSymbol;
  g_scratch_ptr[device] = static_cast<unsigned long long *>(p);
  return hipSuccess;
}

unsigned long long *noalloc_scratch(int device) {
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  auto it = g_scratch_ptr.find(device);
  return it == g_scratch_ptr.end() ? nullptr : it->second;
}

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

template <typename V>
__device__ __forceinline__ V zero_vec() {
  return V(0);
}

// Rows of a gather: n, or min(*n_dev, n) when the count is on the device.
__device__ __forceinline__ int64_t rows_of(int64_t n, const int64_t *n_dev) {
  return n_dev ? min(*n_dev, n) : n;
}

// rv = vectors per row, rv <= kThreads.
template <typename V>
__global__ __launch_bounds__(kThreads) void k_gather(
    const V *__restrict__ table, int64_t n_rows, int32_t rv,
    const int64_t *__restrict__ ids, int64_t n_max, V *__restrict__ out,
    const int64_t *n_dev, unsigned long long *bad) {
  const int64_t n = rows_of(n_max, n_dev);
  const int rpp = kThreads / rv;  // rows per pass
  const int r_in = threadIdx.x / rv;
  const int col = threadIdx.x - r_in * rv;
  if (r_in >= rpp) return;
  const int64_t rows_per_block = int64_t(rpp) * kUnroll;
  for (int64_t r0 = int64_t(blockIdx.x) * rows_per_block; r0 < n;
       r0 += int64_t(gridDim.x) * rows_per_block) {
    V v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t row = r0 + int64_t(u) * rpp + r_in;
      v[u] = zero_vec<V>();
      if (row < n) {
        const int64_t id = ids[row];
        if (id >= 0 && id < n_rows)
          v[u] = table[id * rv + col];
        else if (bad && col == 0)
          atomicAdd(bad, 1ull);
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t row = r0 + int64_t(u) * rpp + r_in;
      if (row < n) __builtin_nontemporal_store(v[u], out + row * rv + col);
    }
  }
}

// Rows wider than kThreads vectors: one block walks the columns of a row.
template <typename V>
__global__ __launch_bounds__(kThreads) void k_gather_wide(
    const V *__restrict__ table, int64_t n_rows, int64_t rv,
    const int64_t *__restrict__ ids, int64_t n_max, V *__restrict__ out,
    const int64_t *n_dev, unsigned long long *bad) {
  const int64_t n = rows_of(n_max, n_dev);
  for (int64_t row = blockIdx.x; row < n; row += gridDim.x) {
    const int64_t id = ids[row];
    const bool ok = id >= 0 && id < n_rows;
    if (!ok && bad && threadIdx.x == 0) atomicAdd(bad, 1ull);
    for (int64_t c = threadIdx.x; c < rv; c += kThreads) {
      V x = zero_vec<V>();
      if (ok) x = table[id * rv + c];
      __builtin_nontemporal_store(x, out + row * rv + c);
    }
  }
}

template <typename V>
hipError_t launch_typed(const void *table, int64_t n_rows, int64_t row_bytes,
                        const int64_t *ids, int64_t n, void *out,
                        hipStream_t stream, const int64_t *n_dev, unsigned long long *bad) {
  const int64_t rv = row_bytes / int64_t(sizeof(V));
  if (rv <= kThreads) {
    const int64_t rows_per_block = int64_t(kThreads / rv) * kUnroll;
    int64_t blocks = (n + rows_per_block - 1) / rows_per_block;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(k_gather<V>, dim3(unsigned(blocks)), dim3(kThreads), 0,
                       stream, static_cast<const V *>(table), n_rows, int32_t(rv),
                       ids, n, static_cast<V *>(out), n_dev, bad);
  } else {
    int64_t blocks = n < 65536 ? n : 65536;
    hipLaunchKernelGGL(k_gather_wide<V>, dim3(unsigned(blocks)), dim3(kThreads),
                       0, stream, static_cast<const V *>(table), n_rows, rv, ids,
                       n, static_cast<V *>(out), n_dev, bad);
  }
  return hipGetLastError();
}

// Several gathers in one launch: segment s owns blocks
// [block_base[s], block_base[s+1]) and moves its rows as k_gather does.
constexpr int kMaxSegs = 32;
// A segment whose row count is on the device pays one dependent load per
// block before its first rows: when such segments would have more than
// kDevCountBlocks blocks in all, each block makes up to kDevCountPasses passes
// (at the capacity) instead of one, so that fewer blocks pay it.
constexpr int64_t kDevCountPasses = 4;
constexpr int64_t kDevCountBlocks = 8192;

struct GatherSeg {
  const void *table;
  int64_t n_rows;
  const int64_t *ids;
  int64_t n;  // rows, or their bound with n_dev
  void *out;
  int64_t rv;
  int64_t block_base;
  const int64_t *n_dev;
};

struct GatherBatch {
  GatherSeg seg[kMaxSegs];
  int64_t block_end;
  int32_t n_seg;
};

template <typename V>
__global__ __launch_bounds__(kThreads) void k_gather_multi(GatherBatch B) {
  int s = 0;
  while (s + 1 < B.n_seg && int64_t(blockIdx.x) >= B.seg[s + 1].block_base) ++s;
  const GatherSeg &G = B.seg[s];
  const int64_t nb = (s + 1 < B.n_seg ? B.seg[s + 1].block_base : B.block_end) - G.block_base;
  const int64_t blk = int64_t(blockIdx.x) - G.block_base;
  const int rv = int(G.rv);
  const V *__restrict__ table = static_cast<const V *>(G.table);
  V *__restrict__ out = static_cast<V *>(G.out);
  const int rpp = kThreads / rv;
  const int r_in = threadIdx.x / rv;
  const int col = threadIdx.x - r_in * rv;
  if (r_in >= rpp) return;
  // (a device count costs each block one dependent load before its first
  // rows: such segments get fewer blocks, each looping over more rows)
  const int64_t n = rows_of(G.n, G.n_dev);
  const int64_t rows_per_block = int64_t(rpp) * kUnroll;
  for (int64_t r0 = blk * rows_per_block; r0 < n; r0 += nb * rows_per_block) {
    V v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t row = r0 + int64_t(u) * rpp + r_in;
      v[u] = zero_vec<V>();
      if (row < n) {
        const int64_t id = G.ids[row];
        if (id >= 0 && id < G.n_rows) v[u] = table[id * rv + col];
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t row = r0 + int64_t(u) * rpp + r_in;
      if (row < n) __builtin_nontemporal_store(v[u], out + row * rv + col);
    }
  }
}

int vec_bytes(const void *table, const void *out, int64_t row_bytes) {
  const uint64_t align = uint64_t(reinterpret_cast<uintptr_t>(table)) |
                         uint64_t(reinterpret_cast<uintptr_t>(out)) | uint64_t(row_bytes);
  if ((align & 15) == 0) return 16;
  if ((align & 7) == 0) return 8;
  if ((align & 3) == 0) return 4;
  if ((align & 1) == 0) return 2;
  return 1;
}

}  // namespace

hipError_t launch_gather(const void *table, int64_t n_rows, int64_t row_bytes,
                         const int64_t *ids, int64_t n, void *out,
                         hipStream_t stream, const int64_t *n_dev, unsigned long long *bad) {
  if (n <= 0 || row_bytes <= 0) return hipSuccess;
  switch (vec_bytes(table, out, row_bytes)) {
    case 16: return launch_typed<u32x4>(table, n_rows, row_bytes, ids, n, out, stream, n_dev, bad);
    case 8: return launch_typed<u32x2>(table, n_rows, row_bytes, ids, n, out, stream, n_dev, bad);
    case 4: return launch_typed<uint32_t>(table, n_rows, row_bytes, ids, n, out, stream, n_dev, bad);
    case 2: return launch_typed<uint16_t>(table, n_rows, row_bytes, ids, n, out, stream, n_dev, bad);
    default: return launch_typed<uint8_t>(table, n_rows, row_bytes, ids, n, out, stream, n_dev, bad);
  }
}

hipError_t launch_gather_multi(const GatherJob *jobs, int32_t n_jobs, hipStream_t stream,
                               hipEvent_t start, hipEvent_t stop) {
  // 16-byte rows of at most kThreads vectors share one launch, up to kMaxSegs
  // per launch; anything else goes through launch_gather.  With events, the
  // batched launches carry them (start on the first, stop on the last), so
  // they time the kernels themselves.
  GatherBatch B{};
  int64_t blocks = 0;
  int launches = 0;
  int64_t pending = 0;  // batched segments still to launch
  int64_t dev_blocks = 0;  // one-pass blocks of the device-count segments
  for (int32_t k = 0; k < n_jobs; ++k) {
    const GatherJob &J = jobs[k];
    if (J.n > 0 && J.row_bytes > 0 && vec_bytes(J.table, J.out, J.row_bytes) == 16 &&
        J.row_bytes / 16 <= kThreads) {
      ++pending;
      const int64_t rpb = int64_t(kThreads / (J.row_bytes / 16)) * kUnroll;
      if (J.n_dev) dev_blocks += (J.n + rpb - 1) / rpb;
    }
  }
  const int64_t passes =
      std::min<int64_t>(kDevCountPasses, std::max<int64_t>(1, dev_blocks / kDevCountBlocks));
  auto flush = [&]() -> hipError_t {
    if (B.n_seg == 0) return hipSuccess;
    B.block_end = blocks;
    pending -= B.n_seg;
    hipEvent_t e0 = launches == 0 ? start : nullptr;
    hipEvent_t e1 = pending == 0 ? stop : nullptr;
    if (e0 || e1)
      hipExtLaunchKernelGGL(k_gather_multi<u32x4>, dim3(unsigned(blocks)), dim3(kThreads), 0,
                            stream, e0, e1, 0, B);
    else
      hipLaunchKernelGGL(k_gather_multi<u32x4>, dim3(unsigned(blocks)), dim3(kThreads), 0,
                         stream, B);
    ++launches;
    B = GatherBatch{};
    blocks = 0;
    return hipGetLastError();
  };
  for (int32_t k = 0; k < n_jobs; ++k) {
    const GatherJob &J = jobs[k];
    if (J.n <= 0 || J.row_bytes <= 0) continue;
    const int64_t rv = J.row_bytes / 16;
    if (vec_bytes(J.table, J.out, J.row_bytes) != 16 || rv > kThreads) {
      hipError_t e =
          launch_gather(J.table, J.n_rows, J.row_bytes, J.ids, J.n, J.out, stream, J.n_dev);
      if (e != hipSuccess) return e;
      continue;
    }
    if (B.n_seg == kMaxSegs) {
      hipError_t e = flush();
      if (e != hipSuccess) return e;
    }
    const int64_t rows_per_block = int64_t(kThreads / rv) * kUnroll;
    int64_t nb = (J.n + rows_per_block - 1) / rows_per_block;
    if (J.n_dev) nb = (nb + passes - 1) / passes;
    if (nb > 65536) nb = 65536;
    B.seg[B.n_seg++] = GatherSeg{J.table, J.n_rows, J.ids, J.n, J.out, rv, blocks, J.n_dev};
    blocks += nb;
  }
  return flush();
}

}  // namespace hg
