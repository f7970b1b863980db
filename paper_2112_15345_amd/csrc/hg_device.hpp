// Device-side helpers for the gfx950 kernels: 64-lane wavefront primitives,
// segment lookup and the Philox4x32-10 counter-based generator.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>

#include "hg_internal.hpp"

namespace hg {

constexpr int kWave = 64;

// A kernel launch that carries timestamps when asked (e0 when the kernel
// starts, e1 when it ends), else a plain launch.
template <typename K, typename... Args>
inline void launch_k(K kernel, dim3 grid, dim3 block, size_t lds, hipStream_t stream,
                     hipEvent_t e0, hipEvent_t e1, Args... args) {
  if (e0 || e1)
    hipExtLaunchKernelGGL(kernel, grid, block, lds, stream, e0, e1, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, lds, stream, args...);
}

// Workgroup b goes to XCD b % kXcds.  A range of n blocks that starts at a
// multiple of kXcds, with n a multiple of kXcds, is reordered by xcd_block so
// that XCD x runs the x-th eighth of the range's work, in order: lines that a
// stretch of consecutive work shares (reached marks and map entries of the same
// mini-batch) are then cached, and written back, by one L2 instead of all
// eight.  A bijection of [0, n): any dispatch order still does every block once.
// With `on` false it is the identity.
inline int64_t xcd_round(int64_t n) { return (n + kXcds - 1) / kXcds * kXcds; }
__device__ __forceinline__ int64_t xcd_block(int64_t r, int64_t n, bool on) {
  return on ? (r % kXcds) * (n / kXcds) + r / kXcds : r;
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Bit mask of the lanes below this one.
__device__ __forceinline__ uint64_t lanes_below() {
  return (uint64_t(1) << lane_id()) - 1;
}

// Orders LDS traffic between the lanes of one wavefront (no block barrier).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Exclusive prefix over the lanes of a small per-lane count (0..7) and the
// wave total, from three ballots.
__device__ __forceinline__ int wave_prefix_small(int v, int *total) {
  const uint64_t below = lanes_below();
  const uint64_t b0 = __ballot(v & 1);
  const uint64_t b1 = __ballot(v & 2);
  const uint64_t b2 = __ballot(v & 4);
  *total = __popcll(b0) + 2 * __popcll(b1) + 4 * __popcll(b2);
  return __popcll(b0 & below) + 2 * __popcll(b1 & below) +
         4 * __popcll(b2 & below);
}

__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, kWave);
  return v;
}

// Inclusive scan over the lanes of a wavefront.
__device__ __forceinline__ int64_t wave_incl_scan_i64(int64_t v) {
  const int lane = lane_id();
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int64_t o = __shfl_up(v, d, kWave);
    if (lane >= d) v += o;
  }
  return v;
}

// Exclusive scan of one value per thread over a 256-thread block; returns the
// thread's exclusive prefix and writes the block total.  `lds` holds 4 int64.
__device__ __forceinline__ int64_t block_excl_scan_256(int64_t v, int64_t *lds,
                                                       int64_t *total) {
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int64_t inc = wave_incl_scan_i64(v);
  if (lane == kWave - 1) lds[wave] = inc;
  __syncthreads();
  int64_t before = 0, sum = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const int64_t s = lds[w];
    if (w < wave) before += s;
    sum += s;
  }
  __syncthreads();
  *total = sum;
  return before + inc - v;
}

// Four exclusive scans at once over a 256-thread block (one pass of
// barriers); `lds` holds 16 int64.
__device__ __forceinline__ void block_excl_scan4_256(const int64_t (&v)[4],
                                                     int64_t (&pre)[4],
                                                     int64_t (&total)[4],
                                                     int64_t *lds) {
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  int64_t inc[4];
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    inc[a] = wave_incl_scan_i64(v[a]);
    if (lane == kWave - 1) lds[a * 4 + wave] = inc[a];
  }
  __syncthreads();
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    int64_t before = 0, sum = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const int64_t s = lds[a * 4 + w];
      if (w < wave) before += s;
      sum += s;
    }
    total[a] = sum;
    pre[a] = before + inc[a] - v[a];
  }
  __syncthreads();
}

// A load through a pointer known to address global memory (device memory),
// so that the compiler issues a global rather than a flat access and does
// not wait on LDS traffic for it.
template <typename T>
__device__ __forceinline__ T load_global(const T *p) {
  return *(const __attribute__((address_space(1))) T *)(p);
}

// Largest s in [0, n) with base[s] <= x, for a non-decreasing base[0..n]
// with base[0] <= x < base[n]: the segment that holds item x.
__device__ __forceinline__ int find_segment(const int64_t *base, int n,
                                            int64_t x) {
  int lo = 0, hi = n;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (base[mid] <= x)
      lo = mid;
    else
      hi = mid;
  }
  return lo;
}

// Takes this block's tile of a single-pass scan: tiles are handed out in the
// order blocks start, so every lower tile belongs to a block already running.
__device__ __forceinline__ int64_t take_ticket(int64_t *small,
                                               uint64_t ticket_base,
                                               int64_t *lds) {
  if (threadIdx.x == 0)
    lds[0] = int64_t(atomicAdd(reinterpret_cast<unsigned long long *>(small + kSlotTicket),
                               1ull) - ticket_base);
  __syncthreads();
  const int64_t t = lds[0];
  __syncthreads();
  return t;
}

// Upper bound on polls of one predecessor's word (well under a second); past
// it the scan gives up, flags kErrLookback and the call reports a device error.
constexpr int kSpinLimit = 1 << 21;

// A look-back word: epoch (20 bits) | state (2 bits) | value (42 bits).
// Each word carries its own epoch, so a reader needs no fence: it polls the
// word until it carries the current epoch.  A tile has one word per scanned
// value: first its aggregate (state 1), later overwritten in place by its
// inclusive prefix (state 2); a reader sees one or the other.
constexpr int kLbValueBits = 42;
constexpr uint32_t kLbAggregate = 1, kLbInclusive = 2;
__device__ __forceinline__ uint64_t lb_word(uint32_t epoch, uint32_t state, int64_t v) {
  return (uint64_t(epoch) << (kLbValueBits + 2)) | (uint64_t(state) << kLbValueBits) |
         (uint64_t(v) & ((uint64_t(1) << kLbValueBits) - 1));
}
__device__ __forceinline__ bool lb_ready(uint64_t w, uint32_t epoch) {
  return uint32_t(w >> (kLbValueBits + 2)) == epoch;
}
__device__ __forceinline__ uint32_t lb_state(uint64_t w) {
  return uint32_t(w >> kLbValueBits) & 3u;
}
__device__ __forceinline__ int64_t lb_value(uint64_t w) {
  return int64_t(w & ((uint64_t(1) << kLbValueBits) - 1));
}
__device__ __forceinline__ void lb_store(uint64_t *p, uint64_t w) {
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t lb_load(const uint64_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Decoupled look-back (single-pass prefix scan) of NV values for tile `tile`
// of a segment whose first tile is `first`, in a block of kTileThreads
// threads.  The tile publishes its aggregates; then every thread inspects one
// predecessor per step (kTileThreads predecessors at a time, one round trip),
// and for each value the block sums the aggregates back to the nearest
// predecessor whose inclusive prefix is out, which ends that value's walk.
// The tile then publishes its own inclusive prefixes.  Returns the exclusive
// prefix in every thread.  `agg` must be the same in all threads; every
// thread of the block must call this.
template <int NV>
__device__ void tile_lookback(Lookback lb, int64_t tile, int64_t first,
                              uint32_t epoch, const int64_t (&agg)[NV],
                              int64_t (&excl)[NV], int64_t *small) {
  constexpr int kWaves = kTileThreads / kWave;
  __shared__ int32_t s_stop[kWaves][NV];
  __shared__ int64_t s_sum[kWaves][NV];
  uint64_t *mine = lb.word + tile * NV;
  const int tid = threadIdx.x;
  const int lane = lane_id();
  const int wave = tid / kWave;
#pragma unroll
  for (int k = 0; k < NV; ++k) excl[k] = 0;
  if (tile <= first) {
    if (tid < NV) {
#pragma unroll
      for (int k = 0; k < NV; ++k)
        if (k == tid) lb_store(mine + k, lb_word(epoch, kLbInclusive, agg[k]));
    }
    return;
  }
  if (tid < NV) {
#pragma unroll
    for (int k = 0; k < NV; ++k)
      if (k == tid) lb_store(mine + k, lb_word(epoch, kLbAggregate, agg[k]));
  }
  bool done[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k) done[k] = false;
  bool timed_out = false;
  for (int64_t top = tile - 1;; top -= kTileThreads) {
    // thread i looks at predecessor top - i; tiles before the segment count
    // as published inclusive prefixes of nothing
    const int64_t j = top - tid;
    const bool valid = j >= first;
    uint64_t w[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) w[k] = 0;
    if (valid) {
      const uint64_t *wj = lb.word + j * NV;
      int spins = 0;
      for (;;) {
#pragma unroll
        for (int k = 0; k < NV; ++k) w[k] = lb_load(wj + k);
        bool ready = true;
#pragma unroll
        for (int k = 0; k < NV; ++k) ready = ready && lb_ready(w[k], epoch);
        if (ready) break;
        if (++spins >= kSpinLimit) { timed_out = true; break; }
        __builtin_amdgcn_s_sleep(1);
      }
    }
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      // a timed-out word ends the walk too; the call then reports an error
      const bool inc = !valid || timed_out || lb_state(w[k]) == kLbInclusive;
      const uint64_t bal = __ballot(inc);
      if (lane == 0) s_stop[wave][k] = bal ? __ffsll((unsigned long long)bal) - 1 : kWave;
    }
    __syncthreads();
    int stop[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      stop[k] = kTileThreads;
      for (int v = kWaves - 1; v >= 0; --v)
        if (s_stop[v][k] < kWave) stop[k] = v * kWave + s_stop[v][k];
      const int64_t x = (!done[k] && valid && tid <= stop[k]) ? lb_value(w[k]) : 0;
      const int64_t ws = wave_sum_i64(x);
      if (lane == 0) s_sum[wave][k] = ws;
    }
    __syncthreads();
    bool all = true;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      if (!done[k]) {
        for (int v = 0; v < kWaves; ++v) excl[k] += s_sum[v][k];
        done[k] = stop[k] < kTileThreads;
      }
      all = all && done[k];
    }
    __syncthreads();  // s_stop and s_sum are rewritten by the next step
    if (all) break;
  }
  if (__ballot(timed_out) && lane == 0)
    atomicOr(reinterpret_cast<int32_t *>(small + kSlotErr), kErrLookback);
  if (tid < NV) {
#pragma unroll
    for (int k = 0; k < NV; ++k)
      if (k == tid) lb_store(mine + k, lb_word(epoch, kLbInclusive, excl[k] + agg[k]));
  }
}

// Next hop's frontier sizes (this hop's plus the new vertices of each type)
// and pair layout (pairs of etype e: frontier of its destination type).  Every
// thread of one 256-thread block calls it; the per-etype pair counts come from
// this hop's sizes directly, and a block scan (in chunks of 256 etypes) lays
// them out.  `next` is another hop's region than `hv`.
__device__ inline int64_t next_frontier_size(const HopView &hv, const int64_t *tile_base,
                                             const int64_t *small, int t) {
  // a type without bitmap tiles (no vertices) gains nothing
  const int64_t u = tile_base[t + 1] > tile_base[t] ? small[kSlotNew + t] : 0;
  return hv.nF[t] + u;
}

__device__ inline void plan_next_hop(HopView hv, HopView next, const EtypeStatic *es,
                                     const int64_t *tile_base, const int64_t *small,
                                     int32_t n_types, int32_t n_etypes) {
  __shared__ int64_t plan_lds[4];
  for (int t = threadIdx.x; t < n_types; t += 256)
    next.nF[t] = next_frontier_size(hv, tile_base, small, t);
  int64_t carry = 0;
  for (int e0 = 0; e0 < n_etypes; e0 += 256) {
    const int e = e0 + int(threadIdx.x);
    const int64_t c = e < n_etypes ? next_frontier_size(hv, tile_base, small, es[e].dst_type) : 0;
    int64_t total;
    const int64_t pre = block_excl_scan_256(c, plan_lds, &total);
    if (e < n_etypes) next.pair_base[e] = carry + pre;
    carry += total;
  }
  if (threadIdx.x == 0) next.pair_base[n_etypes] = carry;
}

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two 32x32
// multiplies, with the round key advanced by the Weyl constants.
struct U32x4 {
  uint32_t x, y, z, w;
};

__device__ __forceinline__ U32x4 philox4x32_10(U32x4 c, uint32_t k0,
                                               uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    // full 64-bit products: one multiply instruction gives both halves
    const uint64_t p0 = uint64_t(0xD2511F53u) * c.x;
    const uint64_t p1 = uint64_t(0xCD9E8D57u) * c.z;
    c = U32x4{uint32_t(p1 >> 32) ^ c.y ^ k0, uint32_t(p1), uint32_t(p0 >> 32) ^ c.w ^ k1,
              uint32_t(p0)};
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

// The edge keys of one (sampling seed, hop, edge type): Philox4x32-10 at
// counter (g, 0, hop, etype) for key groups g < 2^32 (edge IDs are below 2^32,
// so g = eid >> 2 never has a high word).  With the counter's last three words
// the same for every g, the first two rounds are partly the same for all
// lanes: round 0 multiplies the fixed hop word, round 1 the fixed word that
// round 0 made of it.  Those parts are computed once per line (in scalar
// registers), and the 3-input XORs of the later rounds are single bitop3
// instructions (truth table 0x96 = a ^ b ^ c).  The result is exactly
// philox4x32_10({g, 0, hop, etype}, k0, k1): 37 vector operations per four
// keys instead of 58.
struct PhiloxLine {
  uint32_t ek1;    // etype ^ k1 of round 0
  uint32_t x1k0;   // round 1: (round 0's x1) ^ k0 of round 1
  uint32_t hk1;    // round 1: hi(M0 * round 0's x0) ^ k1 of round 1
  uint32_t x3k1;   // round 2: lo(M0 * round 0's x0) ^ k1 of round 2
  uint32_t k0[10], k1[10];
};

__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

// Every argument must be the same on all active lanes.
__device__ __forceinline__ PhiloxLine philox_line(uint32_t k0, uint32_t k1, uint32_t hop,
                                                  uint32_t etype) {
  PhiloxLine L;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    L.k0[r] = __builtin_amdgcn_readfirstlane(k0 + uint32_t(r) * 0x9E3779B9u);
    L.k1[r] = __builtin_amdgcn_readfirstlane(k1 + uint32_t(r) * 0xBB67AE85u);
  }
  // round 0's lane-independent half: p1 = M1 * hop
  const uint64_t p1 = uint64_t(0xCD9E8D57u) * uint32_t(hop);
  const uint32_t x0 = uint32_t(p1 >> 32) ^ L.k0[0];  // counter word 1 is 0
  const uint32_t x1 = uint32_t(p1);
  // round 1's lane-independent product: p0 = M0 * x0
  const uint64_t q0 = uint64_t(0xD2511F53u) * x0;
  L.ek1 = __builtin_amdgcn_readfirstlane(uint32_t(etype) ^ L.k1[0]);
  L.x1k0 = __builtin_amdgcn_readfirstlane(x1 ^ L.k0[1]);
  L.hk1 = __builtin_amdgcn_readfirstlane(uint32_t(q0 >> 32) ^ L.k1[1]);
  L.x3k1 = __builtin_amdgcn_readfirstlane(uint32_t(q0) ^ L.k1[2]);
  return L;
}

// The keys of group g given round 0's product p0 = M0 * g (64 bits).
__device__ __forceinline__ U32x4 philox_keys_p0(const PhiloxLine &L, uint64_t p0) {
  uint32_t x2 = uint32_t(p0 >> 32) ^ L.ek1;
  uint32_t x3 = uint32_t(p0);
  // round 1: p1 = M1 * x2 (p0 is the line's)
  uint64_t p1 = uint64_t(0xCD9E8D57u) * x2;
  uint32_t x0 = uint32_t(p1 >> 32) ^ L.x1k0;
  uint32_t x1 = uint32_t(p1);
  x2 = L.hk1 ^ x3;
  // round 2: x3 of round 1 is the line's
  p0 = uint64_t(0xD2511F53u) * x0;
  p1 = uint64_t(0xCD9E8D57u) * x2;
  x0 = xor3(uint32_t(p1 >> 32), x1, L.k0[2]);
  x1 = uint32_t(p1);
  x2 = uint32_t(p0 >> 32) ^ L.x3k1;
  x3 = uint32_t(p0);
#pragma unroll
  for (int r = 3; r < 10; ++r) {
    p0 = uint64_t(0xD2511F53u) * x0;
    p1 = uint64_t(0xCD9E8D57u) * x2;
    x0 = xor3(uint32_t(p1 >> 32), x1, L.k0[r]);
    x1 = uint32_t(p1);
    x2 = xor3(uint32_t(p0 >> 32), x3, L.k1[r]);
    x3 = uint32_t(p0);
  }
  return U32x4{x0, x1, x2, x3};
}

__device__ __forceinline__ U32x4 philox_keys(const PhiloxLine &L, uint32_t g) {
  return philox_keys_p0(L, uint64_t(0xD2511F53u) * g);  // round 0: p0 = M0 * g
}

}  // namespace hg
