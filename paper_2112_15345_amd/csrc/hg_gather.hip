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
#include "hg_device.hpp"
#include "hg_internal.hpp"

namespace hg {

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

template <typename V>
__device__ __forceinline__ V zero_vec() {
  return V(0);
}

// rv = vectors per row, rv <= kThreads.
template <typename V>
__global__ __launch_bounds__(kThreads) void k_gather(
    const V *__restrict__ table, int64_t n_rows, int32_t rv,
    const int64_t *__restrict__ ids, int64_t n, V *__restrict__ out) {
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
        if (id >= 0 && id < n_rows) v[u] = table[id * rv + col];
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
    const int64_t *__restrict__ ids, int64_t n, V *__restrict__ out) {
  for (int64_t row = blockIdx.x; row < n; row += gridDim.x) {
    const int64_t id = ids[row];
    const bool ok = id >= 0 && id < n_rows;
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
                        hipStream_t stream) {
  const int64_t rv = row_bytes / int64_t(sizeof(V));
  if (rv <= kThreads) {
    const int64_t rows_per_block = int64_t(kThreads / rv) * kUnroll;
    int64_t blocks = (n + rows_per_block - 1) / rows_per_block;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(k_gather<V>, dim3(unsigned(blocks)), dim3(kThreads), 0,
                       stream, static_cast<const V *>(table), n_rows, int32_t(rv),
                       ids, n, static_cast<V *>(out));
  } else {
    int64_t blocks = n < 65536 ? n : 65536;
    hipLaunchKernelGGL(k_gather_wide<V>, dim3(unsigned(blocks)), dim3(kThreads),
                       0, stream, static_cast<const V *>(table), n_rows, rv, ids,
                       n, static_cast<V *>(out));
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gather(const void *table, int64_t n_rows, int64_t row_bytes,
                         const int64_t *ids, int64_t n, void *out,
                         hipStream_t stream) {
  if (n <= 0 || row_bytes <= 0) return hipSuccess;
  const uint64_t align = uint64_t(reinterpret_cast<uintptr_t>(table)) |
                         uint64_t(reinterpret_cast<uintptr_t>(out)) |
                         uint64_t(row_bytes);
  if ((align & 15) == 0)
    return launch_typed<u32x4>(table, n_rows, row_bytes, ids, n, out, stream);
  if ((align & 7) == 0)
    return launch_typed<u32x2>(table, n_rows, row_bytes, ids, n, out, stream);
  if ((align & 3) == 0)
    return launch_typed<uint32_t>(table, n_rows, row_bytes, ids, n, out, stream);
  if ((align & 1) == 0)
    return launch_typed<uint16_t>(table, n_rows, row_bytes, ids, n, out, stream);
  return launch_typed<uint8_t>(table, n_rows, row_bytes, ids, n, out, stream);
}

}  // namespace hg
