// Host runtime of the C ABI in include/hg.h: argument checks, device
// workspaces, per-hop orchestration of the gfx950 kernels, and error state.
//
// One mini-batch (DistDGLv2, arXiv 2112.15345, Sec. 3.2 and Sec. 4.2.2) runs
// hop by hop, four steps per hop on the caller's stream:
//   1. counting pass : per (frontier vertex, etype) pair its kept-edge count
//                      and output offsets (single-pass scan)   -> wait (sizes)
//   2. sampler       : the kept edges; each stores 1 into the reached flag
//                      of its source
//   3. compaction    : reached vertices not in the frontier are numbered in
//                      ascending ID and join the frontier bitmap; the frontier
//                      is copied to the head of the source lists
//   4. relabel       : edges get local source IDs; the first block plans the
//                      next hop's pairs on the device
// The source list of hop h is the frontier of hop h+1.  The host waits once
// per hop (after 1, for the output sizes) and once at the end.
#include "hg.h"

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <atomic>
#include <map>
#include <memory>
#include <mutex>
#include <thread>
#include <new>
#include <string>
#include <vector>

#include "hg_internal.hpp"

using namespace hg;

// ---------------------------------------------------------------------------
// Error state

namespace {

thread_local std::string g_last_error;

hg_status fail(hg_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

hg_status fail_hip(hipError_t e, const char *what) {
  (void)hipGetLastError();
  return fail(HG_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

// Launch checks read the thread's last HIP error, so an error that other code
// left pending on this thread is cleared when a call starts.
void clear_pending_error() { (void)hipGetLastError(); }

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Makes the graph's device current for the scope of a call.
struct DeviceGuard {
  int prev = -1;
  bool switched = false;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) == hipSuccess && prev != dev) {
      switched = hipSetDevice(dev) == hipSuccess;
    }
  }
  ~DeviceGuard() {
    if (switched) (void)hipSetDevice(prev);
  }
};

struct NTypeInfo {
  int64_t num_nodes;
  const void *feat;  // the address kernels read: device memory, or pinned host
                     // memory through its device mapping
  int32_t dtype;
  int32_t dim;
  int64_t row_bytes;
  bool host;         // the table lives in pinned host memory
};

// A feature table is device memory or pinned host memory (hipHostMalloc):
// kernels read the latter through its device mapping, over the host link.
// Pageable host memory is refused.
hg_status feature_address(int32_t t, const void *feat, const void **addr, bool *host) {
  hipPointerAttribute_t a{};
  if (hipPointerGetAttributes(&a, feat) != hipSuccess ||
      (a.type != hipMemoryTypeHost && a.type != hipMemoryTypeDevice &&
       a.type != hipMemoryTypeManaged)) {
    (void)hipGetLastError();
    return fail(HG_EINVAL, "node type %d: the feature table is neither device memory nor "
                           "pinned host memory", t);
  }
  *host = a.type == hipMemoryTypeHost;
  *addr = feat;
  if (*host) {
    void *d = nullptr;
    if (hipHostGetDevicePointer(&d, const_cast<void *>(feat), 0) != hipSuccess || !d) {
      (void)hipGetLastError();
      return fail(HG_EINVAL, "node type %d: pinned feature table has no device mapping", t);
    }
    *addr = d;
  }
  return HG_OK;
}

struct ETypeInfo {
  int32_t src, dst;
  int64_t nnz;
  const int64_t *indptr;
  const int64_t *indices;
  // the destination type's non-empty mask (owned by the graph), if it has one
  const uint32_t *nz_mask = nullptr;
  int32_t nz_words = 0, nz_slot = 0;
};

// A device buffer that grows (stream-ordered) and is reused across calls.
// The library's stream-ordered pool on a device, for the scratch buffers and
// the default output arrays.  Memory freed into it stays reserved (release
// threshold at its maximum): a call that needs no more than earlier calls maps
// no new memory, where a pool that trims at each synchronisation would map
// gigabytes again (tens of ms) whenever a call outgrows what it kept.  The pool
// lives until the process ends, since blocks handles may outlive their graph.
hipMemPool_t library_pool(int device) {
  static std::mutex mu;
  static std::map<int, hipMemPool_t> pools;
  std::lock_guard<std::mutex> lk(mu);
  auto it = pools.find(device);
  if (it != pools.end()) return it->second;
  hipMemPoolProps props{};
  props.allocType = hipMemAllocationTypePinned;
  props.handleTypes = hipMemHandleTypeNone;
  props.location.type = hipMemLocationTypeDevice;
  props.location.id = device;
  hipMemPool_t pool = nullptr;
  if (hipMemPoolCreate(&pool, &props) != hipSuccess) {
    (void)hipGetLastError();
    pool = nullptr;  // fall back to the device's default pool
  } else {
    uint64_t keep = UINT64_MAX;
    if (hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep) != hipSuccess)
      (void)hipGetLastError();
  }
  pools[device] = pool;
  return pool;
}

// Stream-ordered allocation on the current device from the library's pool.
hipError_t pool_alloc(void **p, size_t bytes, hipStream_t s) {
  int device = 0;
  hipError_t e = hipGetDevice(&device);
  if (e != hipSuccess) return e;
  hipMemPool_t pool = library_pool(device);
  return pool ? hipMallocFromPoolAsync(p, bytes, pool, s) : hipMallocAsync(p, bytes, s);
}

struct Scratch {
  void *p = nullptr;
  size_t cap = 0;
  bool fresh = false;  // reallocated by the last ensure()
  bool ensure(size_t bytes, hipStream_t s) {
    fresh = false;
    if (bytes <= cap) return true;
    fresh = true;
    if (p) (void)hipFreeAsync(p, s);
    p = nullptr;
    cap = 0;
    const size_t want = align_up(std::max(bytes, bytes + bytes / 2));
    if (pool_alloc(&p, want, s) != hipSuccess) {
      (void)hipGetLastError();
      p = nullptr;
      return false;
    }
    cap = want;
    return true;
  }
  void release() {
    if (p) (void)hipFree(p);
    p = nullptr;
    cap = 0;
  }
};

// Per-call device state.  One call uses a workspace at a time; between calls
// both bitmaps are all 0 (so no map entry is meaningful).
struct Workspace {
  int32_t *map = nullptr;          // sum of num_nodes: local IDs
  uint8_t *reached = nullptr;      // n_tiles * kTile * 32 bytes: reached this hop
  uint32_t *fbits = nullptr;       // n_tiles * kTile words: in the frontier
  uint32_t *rbits = nullptr;       // n_tiles * kTile words: reached this hop (bit mode)
  int64_t *dsmall = nullptr;       // readback slots
  int64_t *hsmall = nullptr;       // pinned, coherent mirror of dsmall + a flag word
  uint64_t publish_seq = 0;        // flag value of the last publish
  EtypeStatic *d_es = nullptr;     // static per-etype table
  TypeStatic *d_ts = nullptr;      // static per-type table
  int64_t *tile_sums = nullptr;    // per bitmap tile: prefix and count (compaction)
  Scratch tab;                     // per-hop tables (device)
  char *htab = nullptr;            // per-hop tables (pinned host)
  size_t htab_cap = 0;
  Scratch pairs, lb_pairs, edges, cand;
  Scratch targets;                 // edge-seeded calls: endpoints and exclusion tables
  Scratch lw_weight;               // layer-wise calls: importance per vertex (zero between uses)
  Scratch lw_edges, lw_cand;       // layer-wise calls: every in-edge of a hop; candidates
  uint32_t epoch = 0;              // look-back launches so far (mod kEpochLimit)
  // Recorded at the end of every call on that call's stream (`last`); the
  // next call on another stream waits for it.  An event must never outlive
  // the stream it was last recorded on (waiting on it afterwards reads the
  // destroyed stream's state), so retire_stream() re-creates the events of a
  // stream that is about to be destroyed.
  hipEvent_t done = nullptr;
  hipStream_t last = nullptr;
  bool busy = false;
  bool poisoned = false;           // device state unknown: never reuse
};

}  // namespace

struct hg_graph {
  int device = 0;
  int32_t T = 0, R = 0;
  std::vector<NTypeInfo> nt;
  std::vector<ETypeInfo> et;
  bool has_alloc = false;
  hg_allocator alloc{};
  std::vector<int64_t> map_off;    // [T+1]
  std::vector<int64_t> tile_base;  // [T+1] bitmap tiles of each type
  int64_t n_tiles = 0;
  int64_t *d_tile_base = nullptr;  // device copy of tile_base
  int64_t total_nnz = 0;
  std::vector<uint32_t *> nz_masks;  // owned non-empty masks (not by bundle graphs)
  // A bundle of B mini-batches samples a virtual graph made of B copies of
  // this one (copy b of type x is type b * T + x, over the same arrays): its
  // key_R is this graph's R, so that every copy keys its edges as the real
  // edge type.  Made on first use, kept until hg_destroy.
  int32_t key_R = 0;
  std::map<int32_t, hg_graph *> bundles;
  std::mutex mu;
  std::vector<Workspace *> ws;
};

namespace {
void layout_types(hg_graph *g);
void free_graph(hg_graph *g);
// Mini-batches per bundle at most.
constexpr int32_t kMaxBundle = 32;
}  // namespace

// Output arrays of one sampling call; shared by the handles of a bundle and
// released with the last of them.  Holds its device and allocator by value:
// a blocks handle may outlive its graph.
struct OutAllocs {
  int device = 0;
  bool has_alloc = false;
  hg_allocator alloc{};
  hipStream_t stream = nullptr;
  std::vector<void *> ptrs;
  ~OutAllocs();
};

struct hg_blocks {
  hg_graph *g = nullptr;
  hipStream_t stream = nullptr;
  int32_t H = 0, T = 0, R = 0;
  std::vector<int64_t> n_dst, n_src;  // [H*T]
  std::vector<int64_t *> src_gid;     // [H*T]
  std::vector<int64_t> n_edges;       // [H*R]
  // random keys the sampler evaluated per hop, for the whole call (a bundle's
  // handles each hold the bundle's totals)
  std::vector<int64_t> keys;          // [H]
  std::vector<int64_t *> indptr;
  std::vector<int32_t *> src_local, dst_local;
  std::vector<int64_t *> eid;
  std::vector<int64_t> in_n;          // [T]
  std::vector<const int64_t *> in_gid;
  std::vector<void *> feat;           // [T] gathered rows (hg_sample_blocks_gather), or NULL
  // edge-seeded mini-batches (hg_sample_edge_blocks)
  bool edge_seeded = false;
  int32_t n_neg = 0;
  std::vector<int64_t> seed_n;        // [T]
  std::vector<const int64_t *> seed_gid;
  std::vector<int64_t> pair_n;        // [R]
  std::vector<const int32_t *> pos_src, pos_dst, neg_dst;
  std::shared_ptr<OutAllocs> mem;     // the arrays above
};

// ---------------------------------------------------------------------------
// Device memory

namespace {

// Pool requests of 1 MiB and more are rounded up to m * 2^k with m in 8..15
// (at most 1/8 more): calls of similar size then reuse the blocks that earlier
// calls freed instead of making the pool map new memory.
size_t size_class(size_t bytes) {
  if (bytes < (size_t(1) << 20)) return bytes;
  int k = 0;
  while ((bytes >> k) >= 16) ++k;
  size_t m = bytes >> k;
  if ((m << k) < bytes) ++m;
  return m << k;
}

// Output arrays of a blocks handle: the caller's allocator, or the library's
// stream-ordered pool.
void *dev_alloc(hg_graph *g, size_t bytes, hipStream_t s) {
  bytes = align_up(bytes ? bytes : 1);
  if (g->has_alloc) return g->alloc.alloc(g->alloc.ctx, bytes, s);
  void *p = nullptr;
  if (pool_alloc(&p, size_class(bytes), s) != hipSuccess) {
    (void)hipGetLastError();
    return nullptr;
  }
  return p;
}

}  // namespace

OutAllocs::~OutAllocs() {
  DeviceGuard dg(device);
  for (void *p : ptrs) {
    if (!p) continue;
    if (has_alloc)
      alloc.free(alloc.ctx, p, stream);
    else
      (void)hipFreeAsync(p, stream);
  }
  (void)hipGetLastError();
}

namespace {

// Several arrays carved out of one buffer.
struct Carve {
  struct Req {
    void **slot;
    size_t bytes;
  };
  std::vector<Req> reqs;
  template <typename T>
  void add(T **slot, int64_t n) {
    reqs.push_back({reinterpret_cast<void **>(slot),
                    align_up(size_t(std::max<int64_t>(n, 1)) * sizeof(T))});
  }
  size_t bytes() const {
    size_t total = 0;
    for (auto &r : reqs) total += r.bytes;
    return total;
  }
  void assign(void *base) const {
    size_t off = 0;
    for (auto &r : reqs) {
      *r.slot = static_cast<char *>(base) + off;
      off += r.bytes;
    }
  }
  void *allocate(hg_graph *g, hipStream_t s) const {
    void *base = dev_alloc(g, bytes(), s);
    if (base) assign(base);
    return base;
  }
  bool in_scratch(Scratch &sc, hipStream_t s) const {
    if (!sc.ensure(bytes(), s)) return false;
    assign(sc.p);
    return true;
  }
};

// Layout of one hop's table region: [nF T][pair_base R+1][frontier T]
// [src_out T][fanout R].  The host writes frontier, src_out and fanout; nF
// and pair_base come from the previous hop's compaction pass (the host
// writes them for hop 0).
struct RegionLayout {
  size_t nf, pbase, frontier, src_out, fanout, size;
  RegionLayout(int32_t T, int32_t R) {
    nf = 0;
    pbase = nf + sizeof(int64_t) * size_t(T);
    frontier = pbase + sizeof(int64_t) * size_t(R + 1);
    src_out = frontier + sizeof(int64_t) * size_t(T);
    fanout = src_out + sizeof(int64_t) * size_t(T);
    size = align_up(fanout + sizeof(int32_t) * size_t(std::max(R, 1)));
  }
};

void free_workspace(Workspace *w) {
  if (w->done) {
    if (w->last) (void)hipEventSynchronize(w->done);
    (void)hipEventDestroy(w->done);
  }
  (void)hipFree(w->map);
  (void)hipFree(w->reached);
  (void)hipFree(w->fbits);
  (void)hipFree(w->rbits);
  (void)hipFree(w->dsmall);
  (void)hipFree(w->d_es);
  (void)hipFree(w->d_ts);
  (void)hipFree(w->tile_sums);
  w->tab.release();
  w->pairs.release();
  w->lb_pairs.release();
  w->edges.release();
  w->cand.release();
  w->targets.release();
  w->lw_weight.release();
  w->lw_edges.release();
  w->lw_cand.release();
  if (w->hsmall) (void)hipHostFree(w->hsmall);
  if (w->htab) (void)hipHostFree(w->htab);
  delete w;
  clear_pending_error();
}

// n_new[T], then ebase[R+1], then the kept ebase[R+1] of layer-wise hops
size_t small_slots(const hg_graph *g) { return size_t(kSlotNew + g->T + 2 * (g->R + 1)); }

// Takes a free workspace (or makes one) with table room for `tab_bytes`.
hg_status acquire_workspace(hg_graph *g, size_t tab_bytes, hipStream_t stream,
                            Workspace **out) {
  Workspace *w = nullptr;
  {
    std::lock_guard<std::mutex> lk(g->mu);
    for (auto *c : g->ws)
      if (!c->busy) {
        w = c;
        w->busy = true;
        break;
      }
  }
  bool fresh = false;
  if (!w) {
    w = new (std::nothrow) Workspace();
    if (!w) return fail(HG_ENOMEM, "workspace: out of host memory");
    fresh = true;
    const int64_t map_n = g->map_off[g->T];
    const size_t small_n = small_slots(g);
    const int64_t n_lb = std::max<int64_t>(g->n_tiles, 1);
    hipError_t e = hipSuccess;
    if (e == hipSuccess) e = hipMalloc(&w->map, sizeof(int32_t) * size_t(std::max<int64_t>(map_n, 1)));
    if (e == hipSuccess)
      e = hipMalloc(&w->reached, size_t(std::max<int64_t>(g->n_tiles * kTile * 32, 1)));
    if (e == hipSuccess)
      e = hipMalloc(&w->fbits, sizeof(uint32_t) * size_t(std::max<int64_t>(g->n_tiles * kTile, 1)));
    if (e == hipSuccess)
      e = hipMalloc(&w->rbits, sizeof(uint32_t) * size_t(std::max<int64_t>(g->n_tiles * kTile, 1)));
    if (e == hipSuccess) e = hipMalloc(&w->dsmall, sizeof(int64_t) * small_n);
    if (e == hipSuccess) e = hipMalloc(&w->d_es, sizeof(EtypeStatic) * size_t(std::max(g->R, 1)));
    if (e == hipSuccess) e = hipMalloc(&w->d_ts, sizeof(TypeStatic) * size_t(g->T));
    if (e == hipSuccess) e = hipMalloc(&w->tile_sums, sizeof(int64_t) * (2 * size_t(n_lb) + 2));
    // coherent: the device writes it while the host polls the flag word
    if (e == hipSuccess)
      e = hipHostMalloc(reinterpret_cast<void **>(&w->hsmall), sizeof(int64_t) * (small_n + 1),
                        hipHostMallocCoherent);
    if (e == hipSuccess) std::memset(w->hsmall, 0, sizeof(int64_t) * (small_n + 1));
    if (e == hipSuccess) e = hipEventCreateWithFlags(&w->done, hipEventDisableTiming);
    if (e == hipSuccess)
      e = launch_fill_i32(reinterpret_cast<int32_t *>(w->dsmall), 2 * int64_t(small_n), 0, stream);
    // look-back words of the single-pass compaction: no stale epoch
    if (e == hipSuccess)
      e = launch_fill_i32(reinterpret_cast<int32_t *>(w->tile_sums), 4 * n_lb + 4, 0, stream);
    if (e == hipSuccess)
      e = launch_fill_u32(reinterpret_cast<uint32_t *>(w->reached), g->n_tiles * kTile * 8, 0u,
                          stream);
    if (e == hipSuccess) e = launch_fill_u32(w->fbits, g->n_tiles * kTile, 0u, stream);
    if (e == hipSuccess) e = launch_fill_u32(w->rbits, g->n_tiles * kTile, 0u, stream);
    if (e == hipSuccess) {
      std::vector<EtypeStatic> es(size_t(std::max(g->R, 1)));
      for (int32_t i = 0; i < g->R; ++i) {
        const ETypeInfo &E = g->et[i];
        es[i] = EtypeStatic{E.indptr, E.indices, w->map + g->map_off[E.src],
                            w->reached + g->tile_base[E.src] * kTile * 32,
                            w->rbits + g->tile_base[E.src] * kTile,
                            g->nt[E.dst].num_nodes, E.src, E.dst,
                            E.nz_mask, E.nz_words, E.nz_slot};
      }
      std::vector<TypeStatic> ts(g->T);
      for (int32_t t = 0; t < g->T; ++t)
        ts[t] = TypeStatic{w->map + g->map_off[t], w->reached + g->tile_base[t] * kTile * 32,
                           w->fbits + g->tile_base[t] * kTile, g->nt[t].num_nodes,
                           w->rbits + g->tile_base[t] * kTile};
      e = hipMemcpy(w->d_es, es.data(), sizeof(EtypeStatic) * es.size(), hipMemcpyHostToDevice);
      if (e == hipSuccess)
        e = hipMemcpy(w->d_ts, ts.data(), sizeof(TypeStatic) * ts.size(), hipMemcpyHostToDevice);
    }
    if (e != hipSuccess) {
      free_workspace(w);
      return fail(HG_ENOMEM, "workspace allocation failed: %s", hipGetErrorString(e));
    }
    w->busy = true;
  } else if (w->last && w->last != stream) {
    // the previous user ran on another stream (on the same stream, stream
    // order is enough)
    if (hipStreamWaitEvent(stream, w->done, 0) != hipSuccess) {
      std::lock_guard<std::mutex> lk(g->mu);
      w->busy = false;
      return fail_hip(hipGetLastError(), "hipStreamWaitEvent");
    }
  }
  bool ok = w->tab.ensure(tab_bytes, stream);
  if (ok && w->htab_cap < tab_bytes) {
    // tables of earlier calls were consumed before those calls returned
    if (w->htab) (void)hipHostFree(w->htab);
    w->htab = nullptr;
    w->htab_cap = 0;
    // coherent: the upload kernel reads it over the host link, and no GPU
    // cache may keep an earlier call's lines of it
    if (hipHostMalloc(reinterpret_cast<void **>(&w->htab), tab_bytes, hipHostMallocCoherent) ==
        hipSuccess)
      w->htab_cap = tab_bytes;
    else
      ok = false;
  }
  if (!ok) {
    (void)hipGetLastError();
    if (fresh) {
      free_workspace(w);
    } else {
      std::lock_guard<std::mutex> lk(g->mu);
      w->busy = false;
    }
    return fail(HG_ENOMEM, "workspace tables: allocation failed");
  }
  if (fresh) {
    std::lock_guard<std::mutex> lk(g->mu);
    g->ws.push_back(w);
  }
  *out = w;
  return HG_OK;
}

void release_workspace(hg_graph *g, Workspace *w, hipStream_t stream) {
  if (w->poisoned) {
    // its map or bitmap may be dirty: drop it; the next call makes a new one
    (void)hipStreamSynchronize(stream);
    {
      std::lock_guard<std::mutex> lk(g->mu);
      g->ws.erase(std::remove(g->ws.begin(), g->ws.end(), w), g->ws.end());
    }
    free_workspace(w);
    return;
  }
  if (hipEventRecord(w->done, stream) == hipSuccess) {
    w->last = stream;
  } else {
    // no event to wait on: wait here, so that the next user finds it idle
    clear_pending_error();
    (void)hipStreamSynchronize(stream);
    clear_pending_error();
    w->last = nullptr;
  }
  std::lock_guard<std::mutex> lk(g->mu);
  w->busy = false;
}

// Detaches the idle workspaces of g (and of its bundle graphs) from `stream`,
// which the caller is about to destroy: their work on it is waited for and
// their events, last recorded on it, are replaced by fresh ones (a workspace
// whose event cannot be re-created is dropped).  Workspaces in use by a call
// are left alone: no call may be running on a stream that is being retired.
void retire_stream(hg_graph *g, hipStream_t stream) {
  std::vector<hg_graph *> bundles;
  std::vector<Workspace *> dropped;
  {
    std::lock_guard<std::mutex> lk(g->mu);
    for (auto &kv : g->bundles) bundles.push_back(kv.second);
    for (size_t i = 0; i < g->ws.size();) {
      Workspace *w = g->ws[i];
      if (w->busy || w->last != stream) {
        ++i;
        continue;
      }
      (void)hipEventSynchronize(w->done);
      (void)hipEventDestroy(w->done);
      w->done = nullptr;
      w->last = nullptr;
      if (hipEventCreateWithFlags(&w->done, hipEventDisableTiming) != hipSuccess) {
        w->done = nullptr;
        g->ws.erase(g->ws.begin() + ptrdiff_t(i));
        dropped.push_back(w);
        continue;
      }
      ++i;
    }
  }
  for (Workspace *w : dropped) free_workspace(w);
  for (hg_graph *v : bundles) retire_stream(v, stream);
  clear_pending_error();
}

// Waits until the publish launch with flag value `seq` has copied the
// readback slots of w into w->hsmall (it writes the flag word after them).
// Every few hundred polls the stream is queried, so a failed kernel (whose
// successors never run) ends the wait with its error.
hipError_t wait_flag(const hg_graph *g, Workspace *w, uint64_t seq, hipStream_t stream) {
  hipError_t e;
  const int32_t n = int32_t(small_slots(g));
  const volatile int64_t *flag = w->hsmall + n;
  for (uint32_t i = 1; uint64_t(*flag) != seq; ++i) {
    if ((i & 255) == 0) {
      e = hipStreamQuery(stream);
      if (e == hipSuccess) {
        if (uint64_t(*flag) == seq) break;
        return hipErrorUnknown;  // the stream drained without the flag
      }
      if (e != hipErrorNotReady) return e;
      if (i >= (1u << 16)) std::this_thread::yield();  // a long kernel
    }
  }
  std::atomic_thread_fence(std::memory_order_acquire);
  return hipSuccess;
}

int64_t dtype_size(int32_t dt) {
  switch (dt) {
    case HG_DT_F32: return 4;
    case HG_DT_F16: return 2;
    case HG_DT_BF16: return 2;
    default: return 0;
  }
}

// ---------------------------------------------------------------------------
// One sampling call

struct SampleRun {
  hg_graph *g;
  hipStream_t stream;
  Workspace *ws = nullptr;
  hg_blocks *b = nullptr;
  int32_t T, R, H;
  std::vector<uint64_t> sigmas;  // per copy of a bundle (one for a plain call)
  int32_t key_bits;
  const int32_t *fanouts;
  RegionLayout lay;
  size_t sig_bytes;              // the sigma table heads the call's tables
  uint64_t ticket_base = 0;

  // the reached flags are clean unless reached_dirty; the readback slots are
  // zero again once a clearing publish has run
  bool reached_dirty = false;
  bool small_clean = false;

  // an edge-seeded call: its batch, the excluded edges and its extra tables
  // (a region for the seeds' compaction after regions 0 .. H+1, then the
  // per-etype target table)
  const hg_edge_batch *eb = nullptr;
  ExclView X{};
  size_t edge_tab = 0;  // bytes of the per-etype target table

  // a layer-wise call: draws per hop and node type (hop-major [H * T]); its
  // candidates are listed through region H+2; the importance array is clean
  // unless wt_dirty
  const int32_t *layer_sizes = nullptr;
  bool wt_dirty = false;

  // the feature gather of the input frontier, launched before the last wait:
  // node types, events carried by its launches, and whether it was launched
  const int32_t *gtypes = nullptr;
  int32_t n_gather = 0;
  hipEvent_t g_start = nullptr, g_stop = nullptr;
  // device timestamps of the stages of every hop (benchmarks), or NULL
  const hg_stage_events *sev = nullptr;
  StageEv stage_ev(int32_t h, int s) const {
    if (!sev || h >= HG_MAX_TIMED_HOPS) return StageEv{};
    return StageEv{sev->start[h][s], sev->stop[h][s]};
  }
  bool gathered = false;
  hg_status early_gather(const std::vector<int64_t *> &ids, const std::vector<int64_t> &cap);
  // a layer-wise hop's kept edges (their per-etype starts are read back at the
  // next wait): the hop and its output arrays
  int32_t lw_hop = -1;
  int64_t *lw_eid = nullptr;
  int32_t *lw_srcl = nullptr, *lw_dstl = nullptr;
  hg_status close_layer_edges();
  hg_status layer_hop(int32_t h, const HopView &hv, const HopView &nv, const PairArrays &pa,
                      int64_t P, int64_t S, const std::vector<int64_t> &nF,
                      const std::vector<int64_t> &cbound, int64_t *indptr_all,
                      int64_t *eid_all, int32_t *srcl_all, int32_t *dstl_all,
                      int64_t **src_slot, std::vector<int64_t *> &src_out, bool inline_ptrs);

  SampleRun(hg_graph *g_, hipStream_t s, int32_t H_, const int32_t *fo,
            const uint64_t *sig, int32_t n_sig, int32_t kb)
      : g(g_), stream(s), T(g_->T), R(g_->R), H(H_), sigmas(sig, sig + n_sig), key_bits(kb),
        fanouts(fo), lay(g_->T, g_->R), sig_bytes(align_up(sizeof(uint64_t) * size_t(n_sig))) {}

  // table bytes of a call: the sigma table, then regions 0 .. H+1 (and for an
  // edge-seeded call the seeds' region H+2 and the target table)
  int32_t n_regions() const { return H + 2 + ((eb || layer_sizes) ? 1 : 0); }
  size_t table_bytes() const {
    return sig_bytes + lay.size * size_t(n_regions()) + edge_tab;
  }
  char *hedge() { return hreg(n_regions()); }
  char *dedge() { return dreg(n_regions()); }
  char *hreg(int r) { return ws->htab + sig_bytes + size_t(r) * lay.size; }
  char *dreg(int r) {
    return static_cast<char *>(ws->tab.p) + sig_bytes + size_t(r) * lay.size;
  }
  const uint64_t *dsigmas() { return static_cast<const uint64_t *>(ws->tab.p); }

  // Region r's frontier is region r-1's source lists (the same table words);
  // region 0's is the seeds.
  HopView view(int r) {
    char *d = dreg(r);
    char *f = r == 0 ? d + lay.frontier : dreg(r - 1) + lay.src_out;
    return HopView{reinterpret_cast<int64_t *>(d + lay.nf),
                   reinterpret_cast<int64_t *>(d + lay.pbase),
                   reinterpret_cast<const int64_t *const *>(f),
                   reinterpret_cast<int64_t *const *>(d + lay.src_out),
                   reinterpret_cast<const int32_t *>(d + lay.fanout)};
  }
  template <typename T>
  T *hfield(int r, size_t off) { return reinterpret_cast<T *>(hreg(r) + off); }

  // The tables' bytes [from, to) to the device copy, read from the pinned,
  // coherent host tables by a kernel: a DMA copy here has stalled every worker
  // stream at once for several ms.  The host rewrites these bytes only in a
  // later call on this workspace, and each call waits on the device (its
  // readbacks) after its upload, so the kernel has read them by then.
  hipError_t upload(size_t from, size_t to) {
    return launch_upload(static_cast<char *>(ws->tab.p) + from, ws->htab + from,
                         int64_t(to - from), stream);
  }

  // A fresh epoch for a look-back launch.  Before epochs repeat, every
  // look-back word is zeroed, so no stale word can pass for a current one.
  hipError_t next_epoch(uint32_t *epoch) {
    ws->epoch += 1;
    if (ws->epoch >= kEpochLimit) {
      ws->epoch = 1;
      hipError_t e = launch_fill_i32(reinterpret_cast<int32_t *>(ws->tile_sums),
                                     4 * std::max<int64_t>(g->n_tiles, 1), 0, stream);
      if (e == hipSuccess && ws->lb_pairs.p)
        e = launch_fill_u32(static_cast<uint32_t *>(ws->lb_pairs.p),
                            int64_t(ws->lb_pairs.cap / sizeof(uint32_t)), 0u, stream);
      if (e != hipSuccess) return e;
    }
    *epoch = ws->epoch;
    return hipSuccess;
  }

  // Waits until the stream has reached this point and the readback slots are
  // in ws->hsmall: a one-block kernel copies them to the coherent host buffer
  // and then sets its flag word, which the host polls (cheaper than a copy
  // plus a stream wait).  Every few hundred polls the stream is queried, so
  // a failed kernel (whose successors never run) ends the wait with its error.
  hipError_t sync_small(bool last = false) {
    uint64_t seq;
    hipError_t e = publish(last, &seq);
    return e == hipSuccess ? wait_published(seq) : e;
  }
  // The two halves of sync_small: the copy launch, and the wait for its flag
  // (work launched in between runs while the host waits).
  hipError_t publish(bool last, uint64_t *seq) {
    const int32_t n = int32_t(small_slots(g));
    *seq = ++ws->publish_seq;
    hipError_t e = launch_publish(ws->dsmall, ws->hsmall, n, *seq, last, stream);
    if (e == hipSuccess && last) small_clean = true;
    return e;
  }
  hipError_t wait_published(uint64_t seq) { return wait_flag(g, ws, seq, stream); }

  hg_status check_flags(const char *where) {
    const int32_t err = int32_t(ws->hsmall[kSlotErr]);
    if (err & (kErrSeedRange | kErrSeedRepeat))
      return fail(HG_EINVAL, "seeds: out of range or repeated within a node type");
    if (err & kErrTarget)
      return fail(HG_EINVAL, "target edges: an edge ID out of range, or a reverse edge that "
                             "does not run back along its target");
    if (err) {
      ws->poisoned = true;
      return fail(HG_EDEVICE, "%s: device check failed (flags %d)", where, err);
    }
    return HG_OK;
  }

  // Leaves the bitmaps and the readback slots clean; releases the workspace.
  // (The map needs nothing: with the frontier bits cleared, no entry is
  // meaningful.)
  void finish(bool ok) {
    if (!ws->poisoned) {
      if (reached_dirty) {
        (void)launch_fill_u32(reinterpret_cast<uint32_t *>(ws->reached), g->n_tiles * kTile * 8, 0u,
                              stream);
        (void)launch_fill_u32(ws->rbits, g->n_tiles * kTile, 0u, stream);
      }
      (void)launch_fill_u32(ws->fbits, g->n_tiles * kTile, 0u, stream);
      if (!small_clean)
        (void)launch_fill_i32(reinterpret_cast<int32_t *>(ws->dsmall),
                              2 * int64_t(small_slots(g)), 0, stream);
      if (wt_dirty)
        (void)launch_fill_u32(static_cast<uint32_t *>(ws->lw_weight.p),
                              2 * g->map_off[g->T], 0u, stream);
    }
    if (!ok && b) {
      delete b;  // and its arrays
      b = nullptr;
    }
    release_workspace(g, ws, stream);
    ws = nullptr;
  }

  // A failed launch, copy or wait: the device state is unknown.
  hg_status fail_device(hipError_t e, const char *what) {
    ws->poisoned = true;
    return fail_hip(e, what);
  }

  void init_blocks();
  hg_status run(const int64_t *const *seeds, const int64_t *n_seeds);
  hg_status run_layers(const int64_t *const *seeds, const int64_t *n_seeds);
  hg_status run_edges();
  hg_status hops(std::vector<int64_t> &nF, int64_t n_items);
};

void SampleRun::init_blocks() {
  b->g = g;
  b->stream = stream;
  b->mem = std::make_shared<OutAllocs>();
  b->mem->device = g->device;
  b->mem->has_alloc = g->has_alloc;
  b->mem->alloc = g->alloc;
  b->mem->stream = stream;
  b->H = H;
  b->T = T;
  b->R = R;
  b->n_dst.assign(size_t(H) * T, 0);
  b->n_src.assign(size_t(H) * T, 0);
  b->src_gid.assign(size_t(H) * T, nullptr);
  b->n_edges.assign(size_t(H) * R, 0);
  b->keys.assign(size_t(H), 0);
  b->indptr.assign(size_t(H) * R, nullptr);
  b->src_local.assign(size_t(H) * R, nullptr);
  b->dst_local.assign(size_t(H) * R, nullptr);
  b->eid.assign(size_t(H) * R, nullptr);
  b->in_n.assign(T, 0);
  b->in_gid.assign(T, nullptr);
  b->feat.assign(T, nullptr);
}

hg_status SampleRun::run(const int64_t *const *seeds, const int64_t *n_seeds) {
  hipError_t e;
  init_blocks();

  // ---- region 0: the seeds are the first frontier -------------------------
  std::vector<int64_t> nF(T);
  int64_t P = 0;
  for (int32_t t = 0; t < T; ++t) {
    nF[t] = n_seeds[t];
    hfield<int64_t>(0, lay.nf)[t] = nF[t];
    hfield<const int64_t *>(0, lay.frontier)[t] = n_seeds[t] > 0 ? seeds[t] : nullptr;
    hfield<int64_t *>(0, lay.src_out)[t] = nullptr;
  }
  for (int32_t i = 0; i < R; ++i) {
    hfield<int64_t>(0, lay.pbase)[i] = P;
    P += nF[g->et[i].dst];
  }
  hfield<int64_t>(0, lay.pbase)[R] = P;
  // every region's fanouts and empty source lists go up now; a hop's nF and
  // pair_base are written by the device, its source lists once allocated
  for (int32_t r = 0; r <= H; ++r) {
    for (int32_t i = 0; i < R; ++i)
      hfield<int32_t>(r, lay.fanout)[i] = r < H ? fanouts[size_t(r) * R + i] : 0;
    for (int32_t t = 0; t < T; ++t) hfield<int64_t *>(r, lay.src_out)[t] = nullptr;
  }
  int64_t n_items = P + 1;  // pair slots of the next counting pass

  // (the readback slots are zero: a new workspace starts so, and every call
  // clears them when it ends)
  std::memcpy(ws->htab, sigmas.data(), sizeof(uint64_t) * sigmas.size());
  if ((e = upload(0, sig_bytes + size_t(H + 1) * lay.size)) != hipSuccess)
    return fail_device(e, "start");
  int64_t total = 0;
  for (int64_t n : nF) total += n;
  if ((e = launch_insert_frontier(view(0), ws->d_ts, T, total, ws->dsmall, stream)) !=
      hipSuccess)
    return fail_device(e, "insert seeds");
  if (H == 0) {
    if ((e = sync_small(true)) != hipSuccess) return fail_device(e, "sync");
    hg_status st = check_flags("seeds");
    if (st != HG_OK) return st;
    Carve a;
    std::vector<int64_t *> cp(T, nullptr);
    for (int32_t t = 0; t < T; ++t) a.add(&cp[t], nF[t]);
    void *base = a.allocate(g, stream);
    if (!base) return fail(HG_ENOMEM, "seed copy");
    b->mem->ptrs.push_back(base);
    for (int32_t t = 0; t < T; ++t) {
      if (nF[t] > 0 &&
          (e = hipMemcpyAsync(cp[t], seeds[t], sizeof(int64_t) * size_t(nF[t]),
                              hipMemcpyDeviceToDevice, stream)) != hipSuccess)
        return fail_device(e, "seed copy");
      b->in_n[t] = nF[t];
      b->in_gid[t] = cp[t];
    }
    return HG_OK;
  }
  return hops(nF, n_items);
}

// An edge-seeded call: the targets' endpoints become the seeds (ranked by the
// compaction pass from an empty frontier, in region H+2), then the hops run
// from them with the excluded edges left out.
hg_status SampleRun::run_edges() {
  hipError_t e;
  init_blocks();
  const int32_t Q = eb->n_neg;
  std::vector<int64_t> tbase(R + 1, 0);
  for (int32_t i = 0; i < R; ++i) tbase[i + 1] = tbase[i] + eb->n_eids[i];
  const int64_t N = tbase[R];
  // seeds of a type: at most its vertices, and at most its endpoints
  std::vector<int64_t> bound(T, 0);
  for (int32_t i = 0; i < R; ++i) {
    bound[g->et[i].src] += eb->n_eids[i];
    bound[g->et[i].dst] += eb->n_eids[i] * (1 + Q);
  }
  for (int32_t t = 0; t < T; ++t) bound[t] = std::min(bound[t], g->nt[t].num_nodes);

  // ---- outputs: the seeds and the pair graphs -------------------------------
  Carve oc;
  std::vector<int64_t *> seeds(T, nullptr);
  int32_t *pos_src, *pos_dst, *neg_dst;
  for (int32_t t = 0; t < T; ++t) oc.add(&seeds[t], bound[t]);
  oc.add(&pos_src, N);
  oc.add(&pos_dst, N);
  oc.add(&neg_dst, N * Q);
  void *ob = oc.allocate(g, stream);
  if (!ob) return fail(HG_ENOMEM, "edge batch: seed and pair arrays");
  b->mem->ptrs.push_back(ob);
  b->edge_seeded = true;
  b->n_neg = Q;
  b->seed_n.assign(T, 0);
  b->seed_gid.assign(seeds.begin(), seeds.end());
  b->pair_n.assign(eb->n_eids, eb->n_eids + R);
  b->pos_src.resize(R);
  b->pos_dst.resize(R);
  b->neg_dst.resize(R);
  for (int32_t i = 0; i < R; ++i) {
    b->pos_src[i] = pos_src + tbase[i];
    b->pos_dst[i] = pos_dst + tbase[i];
    b->neg_dst[i] = neg_dst + tbase[i] * Q;
  }

  // ---- scratch: endpoints, negatives, reverse edges, exclusion tables ---------
  const int64_t n_x = eb->exclude == 0 ? 0 : N * (eb->exclude == 2 ? 2 : 1);
  uint64_t cap = 64;
  while (cap < uint64_t(2 * n_x)) cap <<= 1;  // always an empty slot
  if (cap > (uint64_t(1) << 31)) return fail(HG_EUNSUPPORTED, "edge batch: too many targets");
  Carve sc;
  EdgeBatchArgs A{};
  sc.add(&A.tsrc, N);
  sc.add(&A.tdst, N);
  sc.add(&A.trev, N);
  sc.add(&A.tneg, N * Q);
  sc.add(&A.edge_keys, int64_t(cap));
  sc.add(&A.pair_keys, int64_t(cap));
  sc.add(&A.pair_cnt, int64_t(cap));
  sc.add(&A.n_seed, R);
  if (!sc.in_scratch(ws->targets, stream)) return fail(HG_ENOMEM, "edge batch: scratch");

  // ---- tables: regions 0 .. H+1, the seeds' region H+2, the target table -----
  const int32_t pre = H + 2;
  for (int32_t r = 0; r <= pre; ++r) {
    for (int32_t i = 0; i < R; ++i)
      hfield<int32_t>(r, lay.fanout)[i] = r < H ? fanouts[size_t(r) * R + i] : 0;
    for (int32_t t = 0; t < T; ++t) {
      hfield<int64_t *>(r, lay.src_out)[t] = r == pre ? seeds[t] : nullptr;
      hfield<const int64_t *>(r, lay.frontier)[t] = r == 0 ? seeds[t] : nullptr;
      hfield<int64_t>(r, lay.nf)[t] = 0;  // region 0's are written by the device
    }
  }
  int64_t *h_tbase = reinterpret_cast<int64_t *>(hedge());
  EdgeEtype *h_et = reinterpret_cast<EdgeEtype *>(hedge() + align_up(sizeof(int64_t) * (R + 1)));
  for (int32_t i = 0; i <= R; ++i) h_tbase[i] = tbase[i];
  for (int32_t i = 0; i < R; ++i) {
    const bool rev = eb->exclude == 2 && eb->rev_etype && eb->rev_etype[i] >= 0;
    h_et[i] = EdgeEtype{eb->n_eids[i] > 0 ? eb->eids[i] : nullptr,
                        rev ? eb->rev_eid[i] : nullptr, g->et[i].nnz,
                        rev ? eb->rev_etype[i] : -1};
  }
  std::memcpy(ws->htab, sigmas.data(), sizeof(uint64_t) * sigmas.size());
  if ((e = upload(0, table_bytes())) != hipSuccess) return fail_device(e, "start");

  A.es = ws->d_es;
  A.ts = ws->d_ts;
  A.tbase = reinterpret_cast<const int64_t *>(dedge());
  A.et = reinterpret_cast<const EdgeEtype *>(dedge() + align_up(sizeof(int64_t) * (R + 1)));
  A.n_etypes = R;
  A.n_types = T;
  A.n_targets = N;
  A.n_neg = Q;
  A.exclude = eb->exclude;
  A.sigmas = dsigmas();
  A.key_R = g->key_R > 0 ? g->key_R : std::max(R, 1);
  A.pos_src = pos_src;
  A.pos_dst = pos_dst;
  A.neg_dst = neg_dst;
  A.edge_mask = A.pair_mask = uint32_t(cap - 1);
  A.small = ws->dsmall;
  if (eb->exclude >= 1) {
    if ((e = launch_fill_u32(reinterpret_cast<uint32_t *>(A.edge_keys), 2 * int64_t(cap),
                             0xFFFFFFFFu, stream)) != hipSuccess ||
        (e = launch_fill_u32(reinterpret_cast<uint32_t *>(A.pair_keys), 2 * int64_t(cap),
                             0xFFFFFFFFu, stream)) != hipSuccess ||
        (e = launch_fill_i32(A.pair_cnt, int64_t(cap), 0, stream)) != hipSuccess)
      return fail_device(e, "edge batch: tables");
    X = ExclView{A.edge_keys, A.pair_keys, A.pair_cnt, A.n_seed, A.edge_mask, A.pair_mask};
  }

  // ---- seeds: mark the endpoints, rank them, relabel the pair graphs --------
  reached_dirty = true;
  if ((e = launch_edge_targets(A, stream)) != hipSuccess) return fail_device(e, "edge targets");
  char *d = dreg(pre);
  const HopView pv{reinterpret_cast<int64_t *>(d + lay.nf),
                   reinterpret_cast<int64_t *>(d + lay.pbase),
                   reinterpret_cast<const int64_t *const *>(d + lay.frontier),
                   reinterpret_cast<int64_t *const *>(d + lay.src_out),
                   reinterpret_cast<const int32_t *>(d + lay.fanout)};
  uint32_t epoch;
  int64_t ticketed = 0;
  if ((e = next_epoch(&epoch)) != hipSuccess ||
      (e = launch_compact(pv, ws->d_ts, T, ws->reached, ws->fbits, g->d_tile_base, g->n_tiles, 0,
                          ws->tile_sums, epoch, ticket_base, ws->dsmall, &ticketed,
                          stream)) != hipSuccess)
    return fail_device(e, "edge batch: seeds");
  ticket_base += uint64_t(ticketed);
  reached_dirty = false;
  if ((e = launch_edge_relabel(A, view(0), g->d_tile_base, stream)) != hipSuccess)
    return fail_device(e, "edge batch: pairs");
  std::vector<int64_t> nF(bound);  // bounds until the first wait

  if (H == 0) {
    if ((e = sync_small(true)) != hipSuccess) return fail_device(e, "sync");
    hg_status st = check_flags("targets");
    if (st != HG_OK) return st;
    for (int32_t t = 0; t < T; ++t) {
      b->seed_n[t] = ws->hsmall[kSlotNew + t];
      b->in_n[t] = b->seed_n[t];
      b->in_gid[t] = seeds[t];
    }
    return HG_OK;
  }
  int64_t n_items = 1;
  for (int32_t i = 0; i < R; ++i) n_items += bound[g->et[i].dst];
  return hops(nF, n_items);
}

// A layer-wise call: the seeds as in run(), every fanout -1 (each hop first
// lists every in-edge of its frontier), and region H+2 for the candidate lists.
hg_status SampleRun::run_layers(const int64_t *const *seeds, const int64_t *n_seeds) {
  hipError_t e;
  init_blocks();
  std::vector<int64_t> nF(T);
  int64_t P = 0;
  for (int32_t t = 0; t < T; ++t) {
    nF[t] = n_seeds[t];
    hfield<int64_t>(0, lay.nf)[t] = nF[t];
    hfield<const int64_t *>(0, lay.frontier)[t] = n_seeds[t] > 0 ? seeds[t] : nullptr;
  }
  for (int32_t i = 0; i < R; ++i) {
    hfield<int64_t>(0, lay.pbase)[i] = P;
    P += nF[g->et[i].dst];
  }
  hfield<int64_t>(0, lay.pbase)[R] = P;
  for (int32_t r = 0; r < n_regions(); ++r) {
    for (int32_t i = 0; i < R; ++i) hfield<int32_t>(r, lay.fanout)[i] = -1;
    for (int32_t t = 0; t < T; ++t) {
      hfield<int64_t *>(r, lay.src_out)[t] = nullptr;
      if (r > 0) hfield<const int64_t *>(r, lay.frontier)[t] = nullptr;
      if (r == H + 2) hfield<int64_t>(r, lay.nf)[t] = 0;  // candidates are listed from 0
    }
  }
  std::memcpy(ws->htab, sigmas.data(), sizeof(uint64_t) * sigmas.size());
  if ((e = upload(0, table_bytes())) != hipSuccess) return fail_device(e, "start");
  int64_t total = 0;
  for (int64_t n : nF) total += n;
  if ((e = launch_insert_frontier(view(0), ws->d_ts, T, total, ws->dsmall, stream)) !=
      hipSuccess)
    return fail_device(e, "insert seeds");
  if (H == 0) {
    if ((e = sync_small(true)) != hipSuccess) return fail_device(e, "sync");
    hg_status st = check_flags("seeds");
    if (st != HG_OK) return st;
    Carve a;
    std::vector<int64_t *> cp(T, nullptr);
    for (int32_t t = 0; t < T; ++t) a.add(&cp[t], nF[t]);
    void *base = a.allocate(g, stream);
    if (!base) return fail(HG_ENOMEM, "seed copy");
    b->mem->ptrs.push_back(base);
    for (int32_t t = 0; t < T; ++t) {
      if (nF[t] > 0 &&
          (e = hipMemcpyAsync(cp[t], seeds[t], sizeof(int64_t) * size_t(nF[t]),
                              hipMemcpyDeviceToDevice, stream)) != hipSuccess)
        return fail_device(e, "seed copy");
      b->in_n[t] = nF[t];
      b->in_gid[t] = cp[t];
    }
    return HG_OK;
  }
  // the importance array: one uint64 per vertex, zero between uses
  const int64_t map_n = g->map_off[T];
  if (!ws->lw_weight.ensure(sizeof(uint64_t) * size_t(std::max<int64_t>(map_n, 1)), stream))
    return fail(HG_ENOMEM, "layer-wise: importance array");
  if (ws->lw_weight.fresh &&
      (e = launch_fill_u32(static_cast<uint32_t *>(ws->lw_weight.p),
                           int64_t(ws->lw_weight.cap / sizeof(uint32_t)), 0u, stream)) !=
          hipSuccess)
    return fail_device(e, "fill");
  return hops(nF, P + 1);
}

// The kept edges of the last layer-wise hop, from the per-etype starts that
// its keep pass left in the readback slots.
hg_status SampleRun::close_layer_edges() {
  if (lw_hop < 0) return HG_OK;
  const int64_t *kept = ws->hsmall + kSlotNew + T + R + 1;
  for (int32_t i = 0; i < R; ++i) {
    if (kept[i] > kept[i + 1] || kept[i] < 0)
      return fail(HG_EDEVICE, "hop %d: kept edge count mismatch", lw_hop);
    const size_t k = size_t(lw_hop) * R + i;
    b->n_edges[k] = kept[i + 1] - kept[i];
    b->src_local[k] = lw_srcl + kept[i];
    b->dst_local[k] = lw_dstl + kept[i];
    b->eid[k] = lw_eid + kept[i];
  }
  lw_hop = -1;
  return HG_OK;
}

// One layer-wise hop after its counting pass (which numbers every in-edge of
// the frontier): the candidates' importance and their per-type lists, the
// draws, the next frontier, and the kept in-edges into the block arrays.
hg_status SampleRun::layer_hop(int32_t h, const HopView &hv, const HopView &nv,
                               const PairArrays &pa, int64_t P, int64_t S,
                               const std::vector<int64_t> &nF,
                               const std::vector<int64_t> &cbound, int64_t *indptr_all,
                               int64_t *eid_all, int32_t *srcl_all, int32_t *dstl_all,
                               int64_t **src_slot, std::vector<int64_t *> &src_out,
                               bool inline_ptrs) {
  hipError_t e;
  LayerArgs A{};
  A.hv = hv;
  A.next = nv;
  A.es = ws->d_es;
  A.ts = ws->d_ts;
  A.tile_base = g->d_tile_base;
  A.n_types = T;
  A.n_etypes = R;
  A.pa = pa;
  A.n_pairs = P;
  A.n_all = S;
  A.n_keep_tiles = (S + kLayerTile - 1) / kLayerTile;
  A.sigmas = dsigmas();
  A.key_T = T / int32_t(sigmas.size());  // node types of one copy
  A.hop = h;
  A.small = ws->dsmall;
  A.out_eid = eid_all;
  A.out_src_local = srcl_all;
  A.out_dst_local = dstl_all;
  A.out_indptr = indptr_all;
  // the hop's per-type table, written into its own part of the call's tables
  // and uploaded once
  const size_t tab_off = sig_bytes + lay.size * size_t(n_regions()) +
                         size_t(h) * align_up(layer_table_bytes(T));
  char *ht = ws->htab + tab_off;
  uint64_t **h_wt = reinterpret_cast<uint64_t **>(ht);
  int64_t **h_cand = reinterpret_cast<int64_t **>(h_wt + T);
  uint64_t **h_prefix = reinterpret_cast<uint64_t **>(h_cand + T);
  int64_t *h_ctile = reinterpret_cast<int64_t *>(h_prefix + T);
  int64_t *h_dbase = h_ctile + T + 1;
  int32_t *h_draws = reinterpret_cast<int32_t *>(h_dbase + T + 1);
  h_ctile[0] = 0;
  h_dbase[0] = 0;
  for (int32_t t = 0; t < T; ++t) {
    const int32_t k = layer_sizes[size_t(h) * T + t];
    h_draws[t] = k;
    h_ctile[t + 1] = h_ctile[t] + (cbound[t] + kLayerTile - 1) / kLayerTile;
    h_dbase[t + 1] = h_dbase[t] + (k < 0 ? cbound[t] : (cbound[t] > 0 ? k : 0));
    h_wt[t] = static_cast<uint64_t *>(ws->lw_weight.p) + g->map_off[t];
  }
  A.cand_tiles = h_ctile[T];
  A.draw_threads = h_dbase[T];
  const int64_t scan_tiles = std::max(A.cand_tiles, A.n_keep_tiles) + 1;
  Carve ec;
  ec.add(&A.tile_pair, A.n_keep_tiles + 1);
  ec.add(&A.pos, S + 1);
  Carve cc;
  for (int32_t t = 0; t < T; ++t) {
    cc.add(&h_cand[t], cbound[t]);
    cc.add(&h_prefix[t], cbound[t]);
  }
  cc.add(&A.tile_sum, scan_tiles);
  cc.add(&A.tile_pre, scan_tiles);
  if (!ec.in_scratch(ws->lw_edges, stream) || !cc.in_scratch(ws->lw_cand, stream))
    return fail(HG_ENOMEM, "hop %d: layer-wise scratch", h);
  if ((e = upload(tab_off, tab_off + layer_table_bytes(T))) != hipSuccess)
    return fail_device(e, "layer table");
  char *dt = static_cast<char *>(ws->tab.p) + tab_off;
  A.wt = reinterpret_cast<uint64_t *const *>(dt);
  A.cand = reinterpret_cast<int64_t *const *>(dt + sizeof(void *) * size_t(T));
  A.prefix = reinterpret_cast<uint64_t *const *>(dt + sizeof(void *) * 2 * size_t(T));
  A.cand_tile = reinterpret_cast<const int64_t *>(dt + sizeof(void *) * 3 * size_t(T));
  A.draw_base = A.cand_tile + T + 1;
  A.draws = reinterpret_cast<const int32_t *>(A.draw_base + T + 1);
  // 1. the hop's source lists (the sampler's launch carries them in the other
  // modes, and this mode launches no sampler: the in-edges of the frontier,
  // numbered by the counting pass, are read from the CSC where needed)
  if (inline_ptrs &&
      (e = launch_store_ptrs(reinterpret_cast<void **>(src_slot),
                             reinterpret_cast<void *const *>(src_out.data()), T, stream)) !=
          hipSuccess)
    return fail_device(e, "source lists");
  // 2. importance of the candidates, which marks them reached
  reached_dirty = true;
  wt_dirty = true;
  if ((e = launch_lw_weights(A, stream)) != hipSuccess) return fail_device(e, "weights");
  // 3. the candidates of each type in ascending ID (region H+2 lists them)
  const HopView cv = view(H + 2);
  int64_t ticketed = 0;
  uint32_t epoch;
  if ((e = launch_store_ptrs(reinterpret_cast<void **>(dreg(H + 2) + lay.src_out),
                             reinterpret_cast<void *const *>(h_cand), T, stream)) != hipSuccess ||
      (e = next_epoch(&epoch)) != hipSuccess ||
      (e = launch_compact(cv, ws->d_ts, T, ws->reached, ws->fbits, g->d_tile_base, g->n_tiles, 0,
                          ws->tile_sums, epoch, ticket_base, ws->dsmall, &ticketed, stream,
                          true)) != hipSuccess)
    return fail_device(e, "candidates");
  ticket_base += uint64_t(ticketed);
  // 4. their importance prefix per type (which zeroes the importance array)
  if ((e = launch_lw_prefix(A, stream)) != hipSuccess) return fail_device(e, "prefix");
  wt_dirty = false;
  // 5. the draws set the reached flags of the drawn candidates
  if ((e = launch_lw_draw(A, stream)) != hipSuccess) return fail_device(e, "draw");
  // 6. the drawn vertices join the frontier: the source lists of the hop
  int64_t copy_total = 0;
  for (int64_t n : nF) copy_total += n;
  if ((e = next_epoch(&epoch)) != hipSuccess ||
      (e = launch_compact(hv, ws->d_ts, T, ws->reached, ws->fbits, g->d_tile_base, g->n_tiles,
                          copy_total, ws->tile_sums, epoch, ticket_base, ws->dsmall, &ticketed,
                          stream)) != hipSuccess)
    return fail_device(e, "compact");
  ticket_base += uint64_t(ticketed);
  reached_dirty = false;
  // 7. the kept in-edges, the block CSC and the next hop's plan
  if ((e = launch_lw_keep(A, stream)) != hipSuccess) return fail_device(e, "keep");
  lw_hop = h;
  lw_eid = eid_all;
  lw_srcl = srcl_all;
  lw_dstl = dstl_all;
  return HG_OK;
}

// The gather of the input frontier, launched before the last readback: the
// rows of type t are the first (device) count of region H's frontier sizes,
// at most cap[t]; the feature arrays are sized for cap[t] rows.
hg_status SampleRun::early_gather(const std::vector<int64_t *> &ids,
                                  const std::vector<int64_t> &cap) {
  Carve c;
  std::vector<uint8_t *> dst(T, nullptr);
  for (int32_t k = 0; k < n_gather; ++k) {
    const int32_t t = gtypes[k];
    c.add(&dst[t], cap[t] * g->nt[t].row_bytes);
  }
  void *base = c.allocate(g, stream);
  if (!base) return fail(HG_ENOMEM, "feature arrays");
  b->mem->ptrs.push_back(base);
  const int64_t *counts = reinterpret_cast<const int64_t *>(dreg(H) + lay.nf);
  std::vector<GatherJob> jobs;
  for (int32_t k = 0; k < n_gather; ++k) {
    const int32_t t = gtypes[k];
    const NTypeInfo &N = g->nt[t];
    b->feat[t] = dst[t];
    jobs.push_back(GatherJob{N.feat, N.num_nodes, N.row_bytes, ids[t], cap[t], dst[t], counts + t});
  }
  hipError_t e = launch_gather_multi(jobs.data(), int32_t(jobs.size()), stream, g_start, g_stop);
  if (e != hipSuccess) return fail_device(e, "gather");
  gathered = true;
  return HG_OK;
}

// The hop loop from region 0's frontier (sizes nF, or their bounds for an
// edge-seeded call, whose sizes the device wrote); n_items >= pairs + 1.
hg_status SampleRun::hops(std::vector<int64_t> &nF, int64_t n_items) {
  hipError_t e;
  int64_t P = 0;
  // the last hop's source lists (the input frontier) and their capacities
  std::vector<int64_t *> last_src(T, nullptr);
  std::vector<int64_t> last_bound(T, 0);
  int64_t keys_before = 0;
  for (int32_t h = 0; h < H; ++h) {
    const HopView hv = view(h), nv = view(h + 1);
    // ---- 1. counting pass over at most n_items pair slots ----------------
    const int64_t tiles = count_tiles(n_items);
    Carve pc;
    PairArrays pa;
    pc.add(&pa.plo, n_items);
    pc.add(&pa.pdeg, n_items);
    pc.add(&pa.off, n_items);
    pc.add(&pa.pet, n_items);
    pc.add(&pa.wlist, n_items);
    pc.add(&pa.hub_cnt, n_items);
    pc.add(&pa.hub_pair, n_items);
    pc.add(&pa.hub_choff, n_items);
    if (!pc.in_scratch(ws->pairs, stream) ||
        !ws->lb_pairs.ensure(sizeof(uint64_t) * 4 * size_t(tiles), stream))
      return fail(HG_ENOMEM, "hop %d: pair scratch", h);
    Lookback lb{static_cast<uint64_t *>(ws->lb_pairs.p)};
    // new look-back words start with no tile published
    if (ws->lb_pairs.fresh &&
        (e = launch_fill_u32(static_cast<uint32_t *>(ws->lb_pairs.p),
                             int64_t(ws->lb_pairs.cap / sizeof(uint32_t)), 0u, stream)) != hipSuccess)
      return fail_device(e, "fill");
    uint32_t epoch;
    if ((e = next_epoch(&epoch)) != hipSuccess ||
        (e = launch_count_scan(hv, ws->d_es, R, T, n_items, pa, lb, epoch, ticket_base, X,
                               ws->dsmall, stream, stage_ev(h, HG_STAGE_COUNT))) != hipSuccess)
      return fail_device(e, "count");
    ticket_base += uint64_t(tiles);
    // wait: this hop's sizes (and the previous hop's new-vertex counts)
    if ((e = sync_small()) != hipSuccess) return fail_device(e, "sync");
    hg_status st = check_flags("count");
    if (st != HG_OK) return st;
    const int64_t *hs = ws->hsmall;
    // the keys slot sums over the hops: this hop's share
    b->keys[h] = hs[kSlotKeys] - keys_before;
    keys_before = hs[kSlotKeys];
    if ((st = close_layer_edges()) != HG_OK) return st;
    if (h == 0 && eb) {
      // the seeds of an edge-seeded call: the compaction counted them
      for (int32_t t = 0; t < T; ++t) {
        nF[t] = hs[kSlotNew + t];
        b->seed_n[t] = nF[t];
      }
    }
    if (h > 0) {
      // close the previous hop: its source lists are this hop's frontier
      for (int32_t t = 0; t < T; ++t) {
        const int64_t u = hs[kSlotNew + t];
        const size_t k = size_t(h - 1) * T + t;
        b->n_src[k] = b->n_dst[k] + u;
        nF[t] = b->n_src[k];
        if (nF[t] > INT32_MAX)
          return fail(HG_EUNSUPPORTED, "hop %d: more than 2^31-1 vertices of type %d", h - 1, t);
      }
    }
    // pair layout of this hop (the device computed the same from the sizes)
    std::vector<int64_t> pb(R + 1, 0);
    for (int32_t i = 0; i < R; ++i) pb[i + 1] = pb[i] + nF[g->et[i].dst];
    P = hs[kSlotPairs];
    if (P != pb[R]) return fail(HG_EDEVICE, "hop %d: pair count mismatch", h);
    const int64_t S = hs[kSlotEdges];
    const int64_t n_hubs = hs[kSlotHubs], n_chunks = hs[kSlotChunks], n_wave = hs[kSlotWaves];
    std::vector<int64_t> eb(hs + kSlotNew + T, hs + kSlotNew + T + R + 1);

    // ---- outputs of the hop ------------------------------------------------
    std::vector<int64_t> in_by_type(T, 0);
    for (int32_t i = 0; i < R; ++i) in_by_type[g->et[i].src] += eb[i + 1] - eb[i];
    Carve oc;
    int64_t *indptr_all, *eid_all;
    int32_t *srcl_all, *dstl_all;
    std::vector<int64_t *> src_out(T, nullptr);
    std::vector<int64_t> bound(T);
    oc.add(&indptr_all, P + R);
    oc.add(&eid_all, S);
    oc.add(&srcl_all, S);
    oc.add(&dstl_all, S);
    // candidates of a type: its sources outside the frontier (a layer-wise
    // hop keeps at most its draws of them)
    std::vector<int64_t> cbound(T);
    for (int32_t t = 0; t < T; ++t) {
      cbound[t] = std::min(g->nt[t].num_nodes - nF[t], in_by_type[t]);
      int64_t gain = cbound[t];
      if (layer_sizes && layer_sizes[size_t(h) * T + t] >= 0)
        gain = std::min<int64_t>(gain, layer_sizes[size_t(h) * T + t]);
      bound[t] = nF[t] + gain;
      oc.add(&src_out[t], bound[t]);
    }
    void *ob = oc.allocate(g, stream);
    if (!ob) return fail(HG_ENOMEM, "hop %d: block arrays", h);
    b->mem->ptrs.push_back(ob);
    last_src = src_out;
    last_bound = bound;
    // the sampler's scratch (a layer-wise hop launches no sampler)
    int64_t *gid_tmp = nullptr;
    uint64_t *cand = nullptr;
    if (!layer_sizes) {
      Carve ec;
      ec.add(&gid_tmp, S);
      Carve cc;
      cc.add(&cand, n_hubs * kCandCap);
      if (!ec.in_scratch(ws->edges, stream) || !cc.in_scratch(ws->cand, stream))
        return fail(HG_ENOMEM, "hop %d: edge scratch", h);
    }

    // this hop's source lists (also the next hop's frontier): written by the
    // sampler launch itself for a few types, else by their own launches
    int64_t **src_slot = reinterpret_cast<int64_t **>(dreg(h) + lay.src_out);
    const bool inline_ptrs = T <= kInlineSrcOut;
    if (!inline_ptrs &&
        (e = launch_store_ptrs(reinterpret_cast<void **>(src_slot),
                               reinterpret_cast<void *const *>(src_out.data()), T, stream)) !=
            hipSuccess)
      return fail_device(e, "tables");

    if (layer_sizes) {
      if ((st = layer_hop(h, hv, nv, pa, P, S, nF, cbound, indptr_all, eid_all, srcl_all,
                          dstl_all, src_slot, src_out, inline_ptrs)) != HG_OK)
        return st;
      for (int32_t t = 0; t < T; ++t) {
        const size_t k = size_t(h) * T + t;
        b->n_dst[k] = nF[t];
        b->src_gid[k] = src_out[t];
      }
      for (int32_t i = 0; i < R; ++i) b->indptr[size_t(h) * R + i] = indptr_all + pb[i] + i;
      int64_t next_pairs = 0;
      for (int32_t i = 0; i < R; ++i) next_pairs += bound[g->et[i].dst];
      n_items = next_pairs + 1;
      continue;
    }

    // ---- 2-4. sample (and mark), compact, relabel ----------------------------
    reached_dirty = true;
    int64_t copy_total = 0;
    for (int64_t n : nF) copy_total += n;
    // bit mode when the call's vertices far outnumber the hop's kept edges
    const bool bit_mode = g->map_off[T] > kBitModeRatio * std::max<int64_t>(S, 1);
    // blocks ordered per XCD when each XCD's share is whole mini-batches
    // (pairs and kept edges are in mini-batch order)
    const bool xcd_order = g->R / std::max(g->key_R, 1) >= kXcds;
    if ((e = launch_sample(hv, ws->d_es, R, T, P, n_wave, n_chunks, n_hubs, pa, cand, ws->dsmall,
                           dsigmas(), g->key_R, h, key_bits, gid_tmp, eid_all, dstl_all,
                           indptr_all,
                           src_slot, src_out.data(), inline_ptrs ? T : 0, X, stream,
                           stage_ev(h, HG_STAGE_SAMPLE), stage_ev(h, HG_STAGE_SELECT),
                           bit_mode, xcd_order)) != hipSuccess)
      return fail_device(e, "sample");
    int64_t ticketed = 0;
    if ((e = next_epoch(&epoch)) != hipSuccess ||
        (e = launch_compact(hv, ws->d_ts, T, ws->reached, ws->fbits, g->d_tile_base, g->n_tiles,
                            copy_total,
                            ws->tile_sums, epoch, ticket_base, ws->dsmall, &ticketed,
                            stream, false, stage_ev(h, HG_STAGE_COMPACT),
                            bit_mode ? ws->rbits : nullptr)) != hipSuccess)
      return fail_device(e, "compact");
    ticket_base += uint64_t(ticketed);
    reached_dirty = false;
    if ((e = launch_relabel(hv, nv, ws->d_es, g->d_tile_base, ws->dsmall, T, R, S, gid_tmp,
                            srcl_all, stream, stage_ev(h, HG_STAGE_RELABEL),
                            xcd_order)) != hipSuccess)
      return fail_device(e, "relabel");
    // the map now holds the source lists of this hop, which are region h+1's
    // frontier; the relabel pass wrote their sizes into that region

    for (int32_t t = 0; t < T; ++t) {
      const size_t k = size_t(h) * T + t;
      b->n_dst[k] = nF[t];
      b->src_gid[k] = src_out[t];
    }
    for (int32_t i = 0; i < R; ++i) {
      const size_t k = size_t(h) * R + i;
      b->n_edges[k] = eb[i + 1] - eb[i];
      b->indptr[k] = indptr_all + pb[i] + i;
      b->src_local[k] = srcl_all + eb[i];
      b->dst_local[k] = dstl_all + eb[i];
      b->eid[k] = eid_all + eb[i];
    }
    // the next counting pass covers at most this many pair slots
    int64_t next_pairs = 0;
    for (int32_t i = 0; i < R; ++i) next_pairs += bound[g->et[i].dst];
    n_items = next_pairs + 1;
  }

  // final wait: new-vertex counts of the last hop.  The feature gather goes
  // in behind the readback, so the device is busy with it during the wait.
  uint64_t seq;
  if ((e = publish(true, &seq)) != hipSuccess) return fail_device(e, "sync");
  if (n_gather > 0) {
    hg_status gs = early_gather(last_src, last_bound);
    if (gs != HG_OK) {
      (void)wait_published(seq);
      return gs;
    }
  }
  if ((e = wait_published(seq)) != hipSuccess) return fail_device(e, "sync");
  hg_status st = check_flags("compact");
  if (st != HG_OK) return st;
  if ((st = close_layer_edges()) != HG_OK) return st;
  for (int32_t t = 0; t < T; ++t) {
    const size_t k = size_t(H - 1) * T + t;
    b->n_src[k] = b->n_dst[k] + ws->hsmall[kSlotNew + t];
    nF[t] = b->n_src[k];
    if (nF[t] > INT32_MAX)
      return fail(HG_EUNSUPPORTED, "hop %d: more than 2^31-1 vertices of type %d", H - 1, t);
    b->in_n[t] = nF[t];
    b->in_gid[t] = b->src_gid[k];
  }
  return HG_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI

namespace {

// Node types with many incoming edge types get a per-vertex mask of the edge
// types that have in-edges there, so that the counting pass skips the indptr
// reads of empty (vertex, edge type) pairs.  Built once; a type whose mask
// cannot be allocated goes without one.
hipError_t build_nonempty_masks(hg_graph *g, hipStream_t stream) {
  for (int32_t t = 0; t < g->T; ++t) {
    std::vector<int32_t> ets;
    for (int32_t i = 0; i < g->R; ++i)
      if (g->et[i].dst == t) ets.push_back(i);
    const int64_t n = g->nt[t].num_nodes;
    if (int32_t(ets.size()) < kNzMaskMinEtypes || n <= 0) continue;
    const int32_t words = int32_t((ets.size() + 31) / 32);
    uint32_t *mask = nullptr;
    const int64_t **ptrs = nullptr;
    if (hipMalloc(&mask, sizeof(uint32_t) * size_t(n) * size_t(words)) != hipSuccess) {
      (void)hipGetLastError();
      continue;
    }
    g->nz_masks.push_back(mask);
    std::vector<const int64_t *> h(ets.size());
    for (size_t k = 0; k < ets.size(); ++k) h[k] = g->et[ets[k]].indptr;
    hipError_t e = hipMalloc(&ptrs, sizeof(int64_t *) * h.size());
    if (e == hipSuccess)
      e = hipMemcpy(ptrs, h.data(), sizeof(int64_t *) * h.size(), hipMemcpyHostToDevice);
    if (e == hipSuccess)
      e = launch_nonempty_mask(ptrs, int32_t(ets.size()), words, n, mask, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    (void)hipFree(ptrs);
    if (e != hipSuccess) return e;
    for (size_t k = 0; k < ets.size(); ++k) {
      ETypeInfo &E = g->et[ets[k]];
      E.nz_mask = mask;
      E.nz_words = words;
      E.nz_slot = int32_t(k);
    }
  }
  return hipSuccess;
}

}  // namespace

extern "C" {

const char *hg_last_error(void) { return g_last_error.c_str(); }

hg_status hg_create(const hg_ntype_desc *ntypes, int32_t n_ntypes,
                    const hg_etype_desc *etypes, int32_t n_etypes,
                    const hg_allocator *allocator, hipStream_t stream,
                    hg_graph **out) {
  if (!out) return fail(HG_EINVAL, "hg_create: out is NULL");
  *out = nullptr;
  clear_pending_error();
  if (n_ntypes < 1 || !ntypes) return fail(HG_EINVAL, "hg_create: need at least one node type");
  if (n_etypes < 0 || (n_etypes > 0 && !etypes))
    return fail(HG_EINVAL, "hg_create: bad edge-type array");
  if (allocator && (!allocator->alloc || !allocator->free))
    return fail(HG_EINVAL, "hg_create: allocator needs alloc and free");
  for (int32_t t = 0; t < n_ntypes; ++t) {
    const hg_ntype_desc &d = ntypes[t];
    if (d.num_nodes < 0) return fail(HG_EINVAL, "node type %d: negative num_nodes", t);
    if (d.dtype < HG_DT_NONE || d.dtype > HG_DT_BF16)
      return fail(HG_EINVAL, "node type %d: unknown dtype %d", t, d.dtype);
    if (d.dtype != HG_DT_NONE) {
      if (d.dim <= 0) return fail(HG_EINVAL, "node type %d: feature dim must be > 0", t);
      if (d.num_nodes > 0 && !d.feat) return fail(HG_EINVAL, "node type %d: feature table is NULL", t);
    }
  }
  for (int32_t i = 0; i < n_etypes; ++i) {
    const hg_etype_desc &d = etypes[i];
    if (d.src_type < 0 || d.src_type >= n_ntypes || d.dst_type < 0 || d.dst_type >= n_ntypes)
      return fail(HG_EINVAL, "edge type %d: node type out of range", i);
    if (d.nnz < 0 || !d.indptr || (d.nnz > 0 && !d.indices))
      return fail(HG_EINVAL, "edge type %d: bad CSC arrays", i);
    if (d.nnz >= (int64_t(1) << 32))
      return fail(HG_EUNSUPPORTED, "edge type %d: nnz must be below 2^32", i);
  }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail_hip(hipGetLastError(), "hipGetDevice");

  hg_graph *g = new (std::nothrow) hg_graph();
  if (!g) return fail(HG_ENOMEM, "hg_create: out of host memory");
  g->device = dev;
  g->T = n_ntypes;
  g->R = n_etypes;
  if (allocator) {
    g->has_alloc = true;
    g->alloc = *allocator;
  }
  g->key_R = n_etypes;
  for (int32_t t = 0; t < n_ntypes; ++t) {
    const hg_ntype_desc &d = ntypes[t];
    const void *addr = d.feat;
    bool host = false;
    if (d.dtype != HG_DT_NONE && d.num_nodes > 0) {
      hg_status st = feature_address(t, d.feat, &addr, &host);
      if (st != HG_OK) {
        delete g;
        return st;
      }
    }
    g->nt.push_back({d.num_nodes, addr, d.dtype, d.dim, dtype_size(d.dtype) * int64_t(d.dim), host});
  }
  layout_types(g);
  for (int32_t i = 0; i < n_etypes; ++i) {
    const hg_etype_desc &d = etypes[i];
    g->et.push_back({d.src_type, d.dst_type, d.nnz, d.indptr, d.indices});
    g->total_nnz += d.nnz;
  }
  if (!allocator) {
    // keep freed blocks in the stream-ordered pool between calls
    hipMemPool_t pool;
    if (hipDeviceGetDefaultMemPool(&pool, dev) == hipSuccess) {
      uint64_t thr = UINT64_MAX;
      (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &thr);
    }
    (void)hipGetLastError();
  }

  // device copy of the tile table, and the array checks
  int32_t *d_err = nullptr;
  int32_t h_err = 0;
  hipError_t e = hipMalloc(&g->d_tile_base, sizeof(int64_t) * size_t(n_ntypes + 1));
  if (e == hipSuccess) e = hipMalloc(&d_err, sizeof(int32_t));
  if (e == hipSuccess)
    e = hipMemcpyAsync(g->d_tile_base, g->tile_base.data(), sizeof(int64_t) * size_t(n_ntypes + 1),
                       hipMemcpyHostToDevice, stream);
  if (e == hipSuccess) e = launch_fill_i32(d_err, 1, 0, stream);
  for (int32_t i = 0; i < n_etypes && e == hipSuccess; ++i) {
    const ETypeInfo &E = g->et[i];
    e = launch_check_etype(E.indptr, g->nt[E.dst].num_nodes, E.indices, E.nnz,
                           g->nt[E.src].num_nodes, d_err, stream);
  }
  if (e == hipSuccess)
    e = hipMemcpyAsync(&h_err, d_err, sizeof(int32_t), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  (void)hipFree(d_err);
  if (e != hipSuccess) {
    hg_status st = fail_hip(e, "hg_create");
    (void)hipFree(g->d_tile_base);
    delete g;
    return st;
  }
  if (h_err) {
    (void)hipFree(g->d_tile_base);
    delete g;
    return fail(HG_EINVAL, "hg_create: CSC arrays are invalid (indptr not starting at 0, "
                           "decreasing, not ending at nnz, or an index out of range)");
  }
  if ((e = build_nonempty_masks(g, stream)) != hipSuccess) {
    hg_status st = fail_hip(e, "hg_create: non-empty masks");
    free_graph(g);
    return st;
  }
  // set-up of the allocation-free entry point on this device (current here):
  // the device's address of its static scratch array, looked up once
  if ((e = noalloc_scratch_init(dev)) != hipSuccess) {
    hg_status st = fail_hip(e, "hg_create: scratch address");
    free_graph(g);
    return st;
  }
  *out = g;
  return HG_OK;
}

void hg_destroy(hg_graph *g) {
  if (!g) return;
  {
    DeviceGuard dg(g->device);
    free_graph(g);
  }
  clear_pending_error();
}

hg_status hg_retire_stream(hg_graph *g, hipStream_t stream) {
  if (!g) return fail(HG_EINVAL, "hg_retire_stream: graph is NULL");
  {
    DeviceGuard dg(g->device);
    retire_stream(g, stream);
  }
  clear_pending_error();
  return HG_OK;
}

}  // extern "C"

namespace {

// The input-frontier rows of node types gtypes[0..n_gather) into one new
// allocation owned by the blocks handle, gathered on `stream`.
hg_status gather_into_blocks(hg_graph *g, hg_blocks *b, const int32_t *gtypes,
                             int32_t n_gather, hipEvent_t start, hipEvent_t stop,
                             hipStream_t stream) {
  Carve c;
  std::vector<uint8_t *> dst(g->T, nullptr);
  for (int32_t k = 0; k < n_gather; ++k) {
    const int32_t t = gtypes[k];
    c.add(&dst[t], b->in_n[t] * g->nt[t].row_bytes);
  }
  void *base = c.allocate(g, stream);
  if (!base) return fail(HG_ENOMEM, "hg_sample_blocks_gather: feature arrays");
  b->mem->ptrs.push_back(base);
  std::vector<GatherJob> jobs;
  for (int32_t k = 0; k < n_gather; ++k) {
    const int32_t t = gtypes[k];
    const NTypeInfo &N = g->nt[t];
    b->feat[t] = dst[t];
    jobs.push_back(
        GatherJob{N.feat, N.num_nodes, N.row_bytes, b->in_gid[t], b->in_n[t], dst[t], nullptr});
  }
  hipError_t e = launch_gather_multi(jobs.data(), int32_t(jobs.size()), stream, start, stop);
  if (e != hipSuccess) return fail_hip(e, "gather");
  return HG_OK;
}

// Argument checks of one mini-batch on graph g (real).
hg_status check_batch(const hg_graph *g, const int64_t *const *seeds, const int64_t *n_seeds,
                      int32_t n_hops, const int32_t *fanouts, int32_t key_bits,
                      const int32_t *gtypes, int32_t n_gather) {
  if (n_hops < 0) return fail(HG_EINVAL, "hg_sample_blocks: n_hops < 0");
  if (key_bits < 1 || key_bits > 32) return fail(HG_EINVAL, "hg_sample_blocks: key_bits not in 1..32");
  if (!n_seeds) return fail(HG_EINVAL, "hg_sample_blocks: n_seeds is NULL");
  if (n_hops > 0 && g->R > 0 && !fanouts) return fail(HG_EINVAL, "hg_sample_blocks: fanouts is NULL");
  for (int64_t i = 0; i < int64_t(n_hops) * g->R; ++i)
    if (fanouts[i] < -1) return fail(HG_EINVAL, "hg_sample_blocks: fanout %d < -1", fanouts[i]);
  for (int32_t t = 0; t < g->T; ++t) {
    if (n_seeds[t] < 0) return fail(HG_EINVAL, "seeds of type %d: negative count", t);
    if (n_seeds[t] > 0 && (!seeds || !seeds[t]))
      return fail(HG_EINVAL, "seeds of type %d: NULL pointer", t);
    if (n_seeds[t] > g->nt[t].num_nodes)
      return fail(HG_EINVAL, "seeds of type %d: more seeds than vertices", t);
  }
  if (n_gather < 0 || (n_gather > 0 && !gtypes))
    return fail(HG_EINVAL, "hg_sample_blocks_gather: bad node type list");
  std::vector<char> seen(g->T, 0);
  for (int32_t k = 0; k < n_gather; ++k) {
    const int32_t t = gtypes[k];
    if (t < 0 || t >= g->T)
      return fail(HG_EINVAL, "hg_sample_blocks_gather: node type %d out of range", t);
    if (g->nt[t].dtype == HG_DT_NONE || g->nt[t].row_bytes <= 0)
      return fail(HG_EINVAL, "hg_sample_blocks_gather: node type %d has no features", t);
    if (seen[t]) return fail(HG_EINVAL, "hg_sample_blocks_gather: node type %d twice", t);
    seen[t] = 1;
  }
  return HG_OK;
}

// One sampling run on g (a graph or the virtual graph of a bundle, already
// checked), then the gather of node types gtypes into the handle.
// Stage events with only the gather's pair set (NULL when both are NULL).
struct GatherEvents {
  hg_stage_events ev{};
  const hg_stage_events *ptr = nullptr;
  GatherEvents(hipEvent_t start, hipEvent_t stop) {
    if (start || stop) {
      ev.gather_start = start;
      ev.gather_stop = stop;
      ptr = &ev;
    }
  }
};

hg_status run_sampling(hg_graph *g, const int64_t *const *seeds, const int64_t *n_seeds,
                       int32_t n_hops, const int32_t *fanouts, const uint64_t *sigmas,
                       int32_t n_sig, int32_t key_bits, const int32_t *gtypes, int32_t n_gather,
                       const hg_stage_events *sev, hipStream_t stream, hg_blocks **out) {
  DeviceGuard dg(g->device);
  SampleRun run(g, stream, n_hops, fanouts, sigmas, n_sig, key_bits);
  run.gtypes = gtypes;
  run.n_gather = n_gather;
  run.sev = sev;
  run.g_start = sev ? sev->gather_start : nullptr;
  run.g_stop = sev ? sev->gather_stop : nullptr;
  hg_status st = acquire_workspace(g, run.table_bytes(), stream, &run.ws);
  if (st != HG_OK) return st;
  run.b = new (std::nothrow) hg_blocks();
  if (!run.b) {
    run.finish(false);
    return fail(HG_ENOMEM, "hg_sample_blocks: out of host memory");
  }
  try {
    st = run.run(seeds, n_seeds);
    // the gather goes first: the map reset of finish() can wait behind it
    // (the hop loop launched it already unless there were no hops)
    if (st == HG_OK && n_gather > 0 && !run.gathered)
      st = gather_into_blocks(g, run.b, gtypes, n_gather, run.g_start, run.g_stop, stream);
  } catch (const std::bad_alloc &) {
    st = fail(HG_ENOMEM, "hg_sample_blocks: out of host memory");
  }
  if (st != HG_OK) {
    run.finish(false);
    return st;
  }
  hg_blocks *b = run.b;
  run.finish(true);
  *out = b;
  return HG_OK;
}

// An edge-seeded mini-batch (checked), then the gather.
hg_status run_edge_sampling(hg_graph *g, const hg_edge_batch *eb, int32_t n_hops,
                            const int32_t *fanouts, const uint64_t *sigmas, int32_t n_sig,
                            const int32_t *gtypes, int32_t n_gather, hipStream_t stream,
                            hg_blocks **out) {
  DeviceGuard dg(g->device);
  SampleRun run(g, stream, n_hops, fanouts, sigmas, n_sig, 32);
  run.gtypes = gtypes;
  run.n_gather = n_gather;
  run.eb = eb;
  run.edge_tab = align_up(sizeof(int64_t) * size_t(g->R + 1)) +
                 align_up(sizeof(EdgeEtype) * size_t(std::max(g->R, 1)));
  hg_status st = acquire_workspace(g, run.table_bytes(), stream, &run.ws);
  if (st != HG_OK) return st;
  run.b = new (std::nothrow) hg_blocks();
  if (!run.b) {
    run.finish(false);
    return fail(HG_ENOMEM, "hg_sample_edge_blocks: out of host memory");
  }
  try {
    st = run.run_edges();
    if (st == HG_OK && n_gather > 0 && !run.gathered)
      st = gather_into_blocks(g, run.b, gtypes, n_gather, nullptr, nullptr, stream);
  } catch (const std::bad_alloc &) {
    st = fail(HG_ENOMEM, "hg_sample_edge_blocks: out of host memory");
  }
  if (st != HG_OK) {
    run.finish(false);
    return st;
  }
  hg_blocks *b = run.b;
  run.finish(true);
  *out = b;
  return HG_OK;
}

// A layer-wise mini-batch (checked), then the gather.
hg_status run_layer_sampling(hg_graph *g, const int64_t *const *seeds, const int64_t *n_seeds,
                             int32_t n_hops, const int32_t *layer_sizes, const uint64_t *sigmas,
                             int32_t n_sig, const int32_t *gtypes, int32_t n_gather,
                             hipStream_t stream, hg_blocks **out) {
  DeviceGuard dg(g->device);
  SampleRun run(g, stream, n_hops, nullptr, sigmas, n_sig, 32);
  run.gtypes = gtypes;
  run.n_gather = n_gather;
  run.layer_sizes = layer_sizes;
  run.edge_tab = size_t(std::max(n_hops, 0)) * align_up(layer_table_bytes(g->T));
  hg_status st = acquire_workspace(g, run.table_bytes(), stream, &run.ws);
  if (st != HG_OK) return st;
  run.b = new (std::nothrow) hg_blocks();
  if (!run.b) {
    run.finish(false);
    return fail(HG_ENOMEM, "hg_sample_layers: out of host memory");
  }
  try {
    st = run.run_layers(seeds, n_seeds);
    if (st == HG_OK && n_gather > 0 && !run.gathered)
      st = gather_into_blocks(g, run.b, gtypes, n_gather, nullptr, nullptr, stream);
  } catch (const std::bad_alloc &) {
    st = fail(HG_ENOMEM, "hg_sample_layers: out of host memory");
  }
  if (st != HG_OK) {
    run.finish(false);
    return st;
  }
  hg_blocks *b = run.b;
  run.finish(true);
  *out = b;
  return HG_OK;
}

hg_status check_edge_batch(const hg_graph *g, const hg_edge_batch *eb) {
  if (!eb || !eb->n_eids) return fail(HG_EINVAL, "hg_sample_edge_blocks: no batch");
  if (eb->n_neg < 0 || eb->n_neg > HG_MAX_NEG)
    return fail(HG_EINVAL, "hg_sample_edge_blocks: n_neg not in 0..%d", HG_MAX_NEG);
  if (eb->exclude < HG_EXCLUDE_NONE || eb->exclude > HG_EXCLUDE_REVERSE)
    return fail(HG_EINVAL, "hg_sample_edge_blocks: unknown exclusion %d", eb->exclude);
  if (eb->exclude == HG_EXCLUDE_REVERSE && (!eb->rev_etype || !eb->rev_eid))
    return fail(HG_EINVAL, "hg_sample_edge_blocks: reverse exclusion without a reverse map");
  int64_t total = 0;
  for (int32_t i = 0; i < g->R; ++i) {
    const int64_t n = eb->n_eids[i];
    if (n < 0) return fail(HG_EINVAL, "targets of edge type %d: negative count", i);
    if (n > 0 && (!eb->eids || !eb->eids[i]))
      return fail(HG_EINVAL, "targets of edge type %d: NULL pointer", i);
    total += n;
    if (total > (int64_t(1) << 30)) return fail(HG_EUNSUPPORTED, "too many target edges");
    if (eb->exclude != HG_EXCLUDE_REVERSE || n == 0) continue;
    const int32_t r = eb->rev_etype[i];
    if (r < 0) continue;
    if (r >= g->R || g->et[r].src != g->et[i].dst || g->et[r].dst != g->et[i].src)
      return fail(HG_EINVAL, "edge type %d: reverse type %d does not run the other way", i, r);
    if (!eb->rev_eid[i]) return fail(HG_EINVAL, "edge type %d: NULL reverse map", i);
  }
  return HG_OK;
}

hg_status sample_impl(hg_graph *g, const int64_t *const *seeds, const int64_t *n_seeds,
                      int32_t n_hops, const int32_t *fanouts, uint64_t rng_seed,
                      int32_t key_bits, const int32_t *gtypes, int32_t n_gather,
                      hipEvent_t start, hipEvent_t stop, hipStream_t stream,
                      hg_blocks **out) {
  if (!out) return fail(HG_EINVAL, "hg_sample_blocks: out is NULL");
  *out = nullptr;
  clear_pending_error();
  if (!g) return fail(HG_EINVAL, "hg_sample_blocks: graph is NULL");
  hg_status st = check_batch(g, seeds, n_seeds, n_hops, fanouts, key_bits, gtypes, n_gather);
  if (st != HG_OK) return st;
  const GatherEvents ge(start, stop);
  return run_sampling(g, seeds, n_seeds, n_hops, fanouts, &rng_seed, 1, key_bits, gtypes,
                      n_gather, ge.ptr, stream, out);
}

// Map and bitmap layout of a graph's node types.
void layout_types(hg_graph *g) {
  g->map_off.assign(g->T + 1, 0);
  g->tile_base.assign(g->T + 1, 0);
  for (int32_t t = 0; t < g->T; ++t) {
    g->map_off[t + 1] = g->map_off[t] + g->nt[t].num_nodes;
    const int64_t words = (g->nt[t].num_nodes + 31) / 32;
    g->tile_base[t + 1] = g->tile_base[t] + (words + kTile - 1) / kTile;
  }
  g->n_tiles = g->tile_base[g->T];
}

void free_graph(hg_graph *g) {
  for (auto &kv : g->bundles) free_graph(kv.second);
  for (auto *w : g->ws) free_workspace(w);
  for (uint32_t *m : g->nz_masks) (void)hipFree(m);
  (void)hipFree(g->d_tile_base);
  delete g;
}

// The virtual graph of B copies of g (made once, kept until hg_destroy).
hg_status bundle_graph(hg_graph *g, int32_t B, hg_graph **out) {
  std::lock_guard<std::mutex> lk(g->mu);
  auto it = g->bundles.find(B);
  if (it != g->bundles.end()) {
    *out = it->second;
    return HG_OK;
  }
  hg_graph *v = new (std::nothrow) hg_graph();
  if (!v) return fail(HG_ENOMEM, "bundle: out of host memory");
  v->device = g->device;
  v->T = B * g->T;
  v->R = B * g->R;
  v->key_R = g->R;
  v->has_alloc = g->has_alloc;
  v->alloc = g->alloc;
  for (int32_t b = 0; b < B; ++b) {
    for (int32_t t = 0; t < g->T; ++t) v->nt.push_back(g->nt[t]);
    for (int32_t e = 0; e < g->R; ++e) {
      ETypeInfo E = g->et[e];
      E.src += b * g->T;
      E.dst += b * g->T;
      v->et.push_back(E);
    }
  }
  v->total_nnz = int64_t(B) * g->total_nnz;
  layout_types(v);
  DeviceGuard dg(g->device);
  hipError_t e = hipMalloc(&v->d_tile_base, sizeof(int64_t) * size_t(v->T + 1));
  if (e == hipSuccess)
    e = hipMemcpy(v->d_tile_base, v->tile_base.data(), sizeof(int64_t) * size_t(v->T + 1),
                  hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    (void)hipFree(v->d_tile_base);
    delete v;
    return fail(HG_ENOMEM, "bundle: device table: %s", hipGetErrorString(e));
  }
  g->bundles[B] = v;
  *out = v;
  return HG_OK;
}

// Handle of copy b of a bundle's virtual blocks, as a mini-batch of the real
// graph g; shares the arrays.
hg_blocks *split_blocks(hg_graph *g, const hg_blocks *v, int32_t b) {
  hg_blocks *o = new (std::nothrow) hg_blocks();
  if (!o) return nullptr;
  const int32_t T = g->T, R = g->R, H = v->H;
  o->g = g;
  o->stream = v->stream;
  o->H = H;
  o->T = T;
  o->R = R;
  o->n_dst.resize(size_t(H) * T);
  o->n_src.resize(size_t(H) * T);
  o->src_gid.resize(size_t(H) * T);
  o->n_edges.resize(size_t(H) * R);
  o->indptr.resize(size_t(H) * R);
  o->src_local.resize(size_t(H) * R);
  o->dst_local.resize(size_t(H) * R);
  o->eid.resize(size_t(H) * R);
  o->keys = v->keys;
  for (int32_t h = 0; h < H; ++h) {
    for (int32_t t = 0; t < T; ++t) {
      const size_t k = size_t(h) * T + t, kv = size_t(h) * v->T + size_t(b) * T + t;
      o->n_dst[k] = v->n_dst[kv];
      o->n_src[k] = v->n_src[kv];
      o->src_gid[k] = v->src_gid[kv];
    }
    for (int32_t e = 0; e < R; ++e) {
      const size_t k = size_t(h) * R + e, kv = size_t(h) * v->R + size_t(b) * R + e;
      o->n_edges[k] = v->n_edges[kv];
      o->indptr[k] = v->indptr[kv];
      o->src_local[k] = v->src_local[kv];
      o->dst_local[k] = v->dst_local[kv];
      o->eid[k] = v->eid[kv];
    }
  }
  for (int32_t t = 0; t < T; ++t) {
    o->in_n.push_back(v->in_n[size_t(b) * T + t]);
    o->in_gid.push_back(v->in_gid[size_t(b) * T + t]);
    o->feat.push_back(v->feat[size_t(b) * T + t]);
  }
  if (v->edge_seeded) {
    o->edge_seeded = true;
    o->n_neg = v->n_neg;
    for (int32_t t = 0; t < T; ++t) {
      o->seed_n.push_back(v->seed_n[size_t(b) * T + t]);
      o->seed_gid.push_back(v->seed_gid[size_t(b) * T + t]);
    }
    for (int32_t e = 0; e < R; ++e) {
      const size_t kv = size_t(b) * R + e;
      o->pair_n.push_back(v->pair_n[kv]);
      o->pos_src.push_back(v->pos_src[kv]);
      o->pos_dst.push_back(v->pos_dst[kv]);
      o->neg_dst.push_back(v->neg_dst[kv]);
    }
  }
  o->mem = v->mem;
  return o;
}

}  // namespace

extern "C" {

hg_status hg_sample_blocks_ex(hg_graph *g, const int64_t *const *seeds,
                              const int64_t *n_seeds, int32_t n_hops,
                              const int32_t *fanouts, uint64_t rng_seed,
                              int32_t key_bits, hipStream_t stream,
                              hg_blocks **out) {
  return sample_impl(g, seeds, n_seeds, n_hops, fanouts, rng_seed, key_bits, nullptr, 0,
                     nullptr, nullptr, stream, out);
}

hg_status hg_sample_blocks_gather(hg_graph *g, const int64_t *const *seeds,
                                  const int64_t *n_seeds, int32_t n_hops,
                                  const int32_t *fanouts, uint64_t rng_seed,
                                  const int32_t *gather_ntypes, int32_t n_gather,
                                  hipEvent_t start, hipEvent_t stop, hipStream_t stream,
                                  hg_blocks **out) {
  return sample_impl(g, seeds, n_seeds, n_hops, fanouts, rng_seed, 32, gather_ntypes, n_gather,
                     start, stop, stream, out);
}

static hg_status bundle_impl(hg_graph *g, int32_t n_batches, const int64_t *const *seeds,
                      const int64_t *n_seeds, int32_t n_hops, const int32_t *fanouts,
                      const uint64_t *rng_seeds, const int32_t *gather_ntypes, int32_t n_gather,
                      const hg_stage_events *sev, hipStream_t stream, hg_blocks **out) {
  if (!out) return fail(HG_EINVAL, "hg_sample_blocks_bundle: out is NULL");
  clear_pending_error();
  if (!g) return fail(HG_EINVAL, "hg_sample_blocks_bundle: graph is NULL");
  if (n_batches < 1 || n_batches > kMaxBundle)
    return fail(HG_EINVAL, "hg_sample_blocks_bundle: n_batches not in 1..%d", kMaxBundle);
  for (int32_t b = 0; b < n_batches; ++b) out[b] = nullptr;
  if (!rng_seeds || !n_seeds) return fail(HG_EINVAL, "hg_sample_blocks_bundle: NULL array");
  const int32_t T = g->T, R = g->R;
  for (int32_t b = 0; b < n_batches; ++b) {
    hg_status st = check_batch(g, seeds ? seeds + size_t(b) * T : nullptr,
                               n_seeds + size_t(b) * T, n_hops, fanouts, 32, gather_ntypes,
                               n_gather);
    if (st != HG_OK) return st;
  }
  if (n_batches == 1)
    return run_sampling(g, seeds, n_seeds, n_hops, fanouts, rng_seeds, 1, 32, gather_ntypes,
                        n_gather, sev, stream, out);
  hg_graph *v = nullptr;
  hg_status st = bundle_graph(g, n_batches, &v);
  if (st != HG_OK) return st;
  std::vector<const int64_t *> vseeds(size_t(n_batches) * T, nullptr);
  if (seeds) vseeds.assign(seeds, seeds + size_t(n_batches) * T);
  std::vector<int32_t> vfan(size_t(n_hops) * v->R);
  for (int32_t h = 0; h < n_hops; ++h)
    for (int32_t b = 0; b < n_batches; ++b)
      for (int32_t e = 0; e < R; ++e)
        vfan[size_t(h) * v->R + size_t(b) * R + e] = fanouts[size_t(h) * R + e];
  std::vector<int32_t> vg;
  for (int32_t b = 0; b < n_batches; ++b)
    for (int32_t k = 0; k < n_gather; ++k) vg.push_back(b * T + gather_ntypes[k]);
  hg_blocks *vb = nullptr;
  st = run_sampling(v, vseeds.data(), n_seeds, n_hops, vfan.empty() ? nullptr : vfan.data(),
                    rng_seeds, n_batches, 32, vg.empty() ? nullptr : vg.data(),
                    int32_t(vg.size()), sev, stream, &vb);
  if (st != HG_OK) return st;
  for (int32_t b = 0; b < n_batches; ++b) {
    out[b] = split_blocks(g, vb, b);
    if (!out[b]) {
      for (int32_t c = 0; c < b; ++c) {
        delete out[c];
        out[c] = nullptr;
      }
      delete vb;
      return fail(HG_ENOMEM, "hg_sample_blocks_bundle: out of host memory");
    }
  }
  delete vb;  // the split handles keep the arrays
  return HG_OK;
}

hg_status hg_sample_blocks_bundle(hg_graph *g, int32_t n_batches, const int64_t *const *seeds,
                                  const int64_t *n_seeds, int32_t n_hops,
                                  const int32_t *fanouts, const uint64_t *rng_seeds,
                                  const int32_t *gather_ntypes, int32_t n_gather,
                                  hipEvent_t start, hipEvent_t stop, hipStream_t stream,
                                  hg_blocks **out) {
  const GatherEvents ge(start, stop);
  return bundle_impl(g, n_batches, seeds, n_seeds, n_hops, fanouts, rng_seeds, gather_ntypes,
                     n_gather, ge.ptr, stream, out);
}

hg_status hg_sample_blocks_bundle_timed(hg_graph *g, int32_t n_batches,
                                        const int64_t *const *seeds, const int64_t *n_seeds,
                                        int32_t n_hops, const int32_t *fanouts,
                                        const uint64_t *rng_seeds, const int32_t *gather_ntypes,
                                        int32_t n_gather, const hg_stage_events *events,
                                        hipStream_t stream, hg_blocks **out) {
  return bundle_impl(g, n_batches, seeds, n_seeds, n_hops, fanouts, rng_seeds, gather_ntypes,
                     n_gather, events, stream, out);
}

hg_status hg_sample_edge_blocks(hg_graph *g, const hg_edge_batch *batch, int32_t n_hops,
                                const int32_t *fanouts, uint64_t rng_seed,
                                const int32_t *gather_ntypes, int32_t n_gather,
                                hipStream_t stream, hg_blocks **out) {
  if (!out) return fail(HG_EINVAL, "hg_sample_edge_blocks: out is NULL");
  *out = nullptr;
  clear_pending_error();
  if (!g) return fail(HG_EINVAL, "hg_sample_edge_blocks: graph is NULL");
  std::vector<int64_t> zero(g->T, 0);
  hg_status st = check_batch(g, nullptr, zero.data(), n_hops, fanouts, 32, gather_ntypes,
                             n_gather);
  if (st != HG_OK) return st;
  st = check_edge_batch(g, batch);
  if (st != HG_OK) return st;
  return run_edge_sampling(g, batch, n_hops, fanouts, &rng_seed, 1, gather_ntypes, n_gather,
                           stream, out);
}

hg_status hg_sample_layers(hg_graph *g, const int64_t *const *seeds, const int64_t *n_seeds,
                           int32_t n_hops, const int32_t *layer_sizes, uint64_t rng_seed,
                           const int32_t *gather_ntypes, int32_t n_gather, hipStream_t stream,
                           hg_blocks **out) {
  if (!out) return fail(HG_EINVAL, "hg_sample_layers: out is NULL");
  *out = nullptr;
  clear_pending_error();
  if (!g) return fail(HG_EINVAL, "hg_sample_layers: graph is NULL");
  if (n_hops > 0 && !layer_sizes) return fail(HG_EINVAL, "hg_sample_layers: layer_sizes is NULL");
  for (int64_t i = 0; i < int64_t(std::max(n_hops, 0)) * g->T; ++i)
    if (layer_sizes[i] < -1)
      return fail(HG_EINVAL, "hg_sample_layers: layer size %d < -1", layer_sizes[i]);
  std::vector<int32_t> every(size_t(std::max(n_hops, 0)) * g->R + 1, -1);
  hg_status st = check_batch(g, seeds, n_seeds, n_hops, every.data(), 32, gather_ntypes,
                             n_gather);
  if (st != HG_OK) return st;
  return run_layer_sampling(g, seeds, n_seeds, n_hops, layer_sizes, &rng_seed, 1, gather_ntypes,
                            n_gather, stream, out);
}

hg_status hg_sample_layers_bundle(hg_graph *g, int32_t n_batches, const int64_t *const *seeds,
                                  const int64_t *n_seeds, int32_t n_hops,
                                  const int32_t *layer_sizes, const uint64_t *rng_seeds,
                                  const int32_t *gather_ntypes, int32_t n_gather,
                                  hipStream_t stream, hg_blocks **out) {
  if (!out) return fail(HG_EINVAL, "hg_sample_layers_bundle: out is NULL");
  clear_pending_error();
  if (!g) return fail(HG_EINVAL, "hg_sample_layers_bundle: graph is NULL");
  if (n_batches < 1 || n_batches > kMaxBundle)
    return fail(HG_EINVAL, "hg_sample_layers_bundle: n_batches not in 1..%d", kMaxBundle);
  for (int32_t b = 0; b < n_batches; ++b) out[b] = nullptr;
  if (!rng_seeds || !n_seeds) return fail(HG_EINVAL, "hg_sample_layers_bundle: NULL array");
  if (n_hops > 0 && !layer_sizes)
    return fail(HG_EINVAL, "hg_sample_layers_bundle: layer_sizes is NULL");
  const int32_t T = g->T;
  for (int64_t i = 0; i < int64_t(std::max(n_hops, 0)) * T; ++i)
    if (layer_sizes[i] < -1)
      return fail(HG_EINVAL, "hg_sample_layers_bundle: layer size %d < -1", layer_sizes[i]);
  std::vector<int32_t> every(size_t(std::max(n_hops, 0)) * g->R + 1, -1);
  for (int32_t b = 0; b < n_batches; ++b) {
    hg_status st = check_batch(g, seeds ? seeds + size_t(b) * T : nullptr,
                               n_seeds + size_t(b) * T, n_hops, every.data(), 32, gather_ntypes,
                               n_gather);
    if (st != HG_OK) return st;
  }
  if (n_batches == 1)
    return run_layer_sampling(g, seeds, n_seeds, n_hops, layer_sizes, rng_seeds, 1,
                              gather_ntypes, n_gather, stream, out);
  hg_graph *v = nullptr;
  hg_status st = bundle_graph(g, n_batches, &v);
  if (st != HG_OK) return st;
  std::vector<const int64_t *> vseeds(size_t(n_batches) * T, nullptr);
  if (seeds) vseeds.assign(seeds, seeds + size_t(n_batches) * T);
  // every copy draws the same layer sizes for its own node types
  std::vector<int32_t> vsizes(size_t(std::max(n_hops, 0)) * v->T);
  for (int32_t h = 0; h < n_hops; ++h)
    for (int32_t b = 0; b < n_batches; ++b)
      for (int32_t t = 0; t < T; ++t)
        vsizes[size_t(h) * v->T + size_t(b) * T + t] = layer_sizes[size_t(h) * T + t];
  std::vector<int32_t> vg;
  for (int32_t b = 0; b < n_batches; ++b)
    for (int32_t k = 0; k < n_gather; ++k) vg.push_back(b * T + gather_ntypes[k]);
  hg_blocks *vb = nullptr;
  st = run_layer_sampling(v, vseeds.data(), n_seeds, n_hops,
                          vsizes.empty() ? nullptr : vsizes.data(), rng_seeds, n_batches,
                          vg.empty() ? nullptr : vg.data(), int32_t(vg.size()), stream, &vb);
  if (st != HG_OK) return st;
  for (int32_t b = 0; b < n_batches; ++b) {
    out[b] = split_blocks(g, vb, b);
    if (!out[b]) {
      for (int32_t c = 0; c < b; ++c) {
        delete out[c];
        out[c] = nullptr;
      }
      delete vb;
      return fail(HG_ENOMEM, "hg_sample_layers_bundle: out of host memory");
    }
  }
  delete vb;  // the split handles keep the arrays
  return HG_OK;
}

hg_status hg_sample_edge_blocks_bundle(hg_graph *g, int32_t n_batches,
                                       const hg_edge_batch *batches, int32_t n_hops,
                                       const int32_t *fanouts, const uint64_t *rng_seeds,
                                       const int32_t *gather_ntypes, int32_t n_gather,
                                       hipStream_t stream, hg_blocks **out) {
  if (!out) return fail(HG_EINVAL, "hg_sample_edge_blocks_bundle: out is NULL");
  clear_pending_error();
  if (!g) return fail(HG_EINVAL, "hg_sample_edge_blocks_bundle: graph is NULL");
  if (n_batches < 1 || n_batches > kMaxBundle)
    return fail(HG_EINVAL, "hg_sample_edge_blocks_bundle: n_batches not in 1..%d", kMaxBundle);
  for (int32_t b = 0; b < n_batches; ++b) out[b] = nullptr;
  if (!batches || !rng_seeds) return fail(HG_EINVAL, "hg_sample_edge_blocks_bundle: NULL array");
  const int32_t T = g->T, R = g->R;
  std::vector<int64_t> zero(T, 0);
  hg_status st = check_batch(g, nullptr, zero.data(), n_hops, fanouts, 32, gather_ntypes, n_gather);
  if (st != HG_OK) return st;
  for (int32_t b = 0; b < n_batches; ++b) {
    if ((st = check_edge_batch(g, &batches[b])) != HG_OK) return st;
    if (batches[b].n_neg != batches[0].n_neg || batches[b].exclude != batches[0].exclude)
      return fail(HG_EINVAL, "hg_sample_edge_blocks_bundle: batches differ in n_neg or exclude");
  }
  if (n_batches == 1)
    return run_edge_sampling(g, &batches[0], n_hops, fanouts, rng_seeds, 1, gather_ntypes,
                             n_gather, stream, out);
  hg_graph *v = nullptr;
  if ((st = bundle_graph(g, n_batches, &v)) != HG_OK) return st;
  // the batches as one batch of the virtual graph: copy b's edge type e is b * R + e
  const int32_t X = batches[0].exclude;
  const size_t VR = size_t(n_batches) * R;
  std::vector<const int64_t *> eids(VR, nullptr), rev_eid(VR, nullptr);
  std::vector<int64_t> n_eids(VR, 0);
  std::vector<int32_t> rev_et(VR, -1);
  for (int32_t b = 0; b < n_batches; ++b)
    for (int32_t e = 0; e < R; ++e) {
      const hg_edge_batch &B = batches[b];
      const size_t k = size_t(b) * R + e;
      n_eids[k] = B.n_eids[e];
      eids[k] = B.n_eids[e] > 0 ? B.eids[e] : nullptr;
      if (X == HG_EXCLUDE_REVERSE && B.rev_etype[e] >= 0) {
        rev_et[k] = b * R + B.rev_etype[e];
        rev_eid[k] = B.rev_eid[e];
      }
    }
  const hg_edge_batch vb{eids.data(), n_eids.data(), batches[0].n_neg, X,
                         X == HG_EXCLUDE_REVERSE ? rev_et.data() : nullptr,
                         X == HG_EXCLUDE_REVERSE ? rev_eid.data() : nullptr};
  std::vector<int32_t> vfan(size_t(n_hops) * VR);
  for (int32_t h = 0; h < n_hops; ++h)
    for (int32_t b = 0; b < n_batches; ++b)
      for (int32_t e = 0; e < R; ++e)
        vfan[size_t(h) * VR + size_t(b) * R + e] = fanouts[size_t(h) * R + e];
  std::vector<int32_t> vg;
  for (int32_t b = 0; b < n_batches; ++b)
    for (int32_t k = 0; k < n_gather; ++k) vg.push_back(b * T + gather_ntypes[k]);
  hg_blocks *vbk = nullptr;
  st = run_edge_sampling(v, &vb, n_hops, vfan.empty() ? nullptr : vfan.data(), rng_seeds,
                         n_batches, vg.empty() ? nullptr : vg.data(), int32_t(vg.size()), stream,
                         &vbk);
  if (st != HG_OK) return st;
  for (int32_t b = 0; b < n_batches; ++b) {
    out[b] = split_blocks(g, vbk, b);
    if (!out[b]) {
      for (int32_t c = 0; c < b; ++c) {
        delete out[c];
        out[c] = nullptr;
      }
      delete vbk;
      return fail(HG_ENOMEM, "hg_sample_edge_blocks_bundle: out of host memory");
    }
  }
  delete vbk;  // the split handles keep the arrays
  return HG_OK;
}

hg_status hg_blocks_seeds(const hg_blocks *b, int32_t ntype, int64_t *n, const int64_t **gid) {
  if (!b) return fail(HG_EINVAL, "hg_blocks_seeds: blocks is NULL");
  if (ntype < 0 || ntype >= b->T)
    return fail(HG_EINVAL, "hg_blocks_seeds: node type %d out of range", ntype);
  int64_t cnt;
  const int64_t *p;
  if (b->edge_seeded) {
    cnt = b->seed_n[ntype];
    p = b->seed_gid[ntype];
  } else if (b->H > 0) {  // the frontier of hop 0, the head of its source list
    cnt = b->n_dst[ntype];
    p = b->src_gid[ntype];
  } else {
    cnt = b->in_n[ntype];
    p = b->in_gid[ntype];
  }
  if (n) *n = cnt;
  if (gid) *gid = p;
  return HG_OK;
}

hg_status hg_blocks_edge_pairs(const hg_blocks *b, int32_t etype, int64_t *n_pos,
                               const int32_t **pos_src, const int32_t **pos_dst,
                               int64_t *n_negs, const int32_t **neg_dst) {
  if (!b) return fail(HG_EINVAL, "hg_blocks_edge_pairs: blocks is NULL");
  if (!b->edge_seeded) return fail(HG_EINVAL, "hg_blocks_edge_pairs: not an edge-seeded batch");
  if (etype < 0 || etype >= b->R)
    return fail(HG_EINVAL, "hg_blocks_edge_pairs: edge type %d out of range", etype);
  if (n_pos) *n_pos = b->pair_n[etype];
  if (pos_src) *pos_src = b->pos_src[etype];
  if (pos_dst) *pos_dst = b->pos_dst[etype];
  if (n_negs) *n_negs = b->pair_n[etype] * b->n_neg;
  if (neg_dst) *neg_dst = b->neg_dst[etype];
  return HG_OK;
}

hg_status hg_blocks_features(const hg_blocks *b, int32_t ntype, int64_t *rows,
                             const void **feat) {
  if (!b) return fail(HG_EINVAL, "hg_blocks_features: blocks is NULL");
  if (ntype < 0 || ntype >= b->T)
    return fail(HG_EINVAL, "hg_blocks_features: node type %d out of range", ntype);
  const bool have = b->feat[ntype] != nullptr;
  if (rows) *rows = have ? b->in_n[ntype] : 0;
  if (feat) *feat = b->feat[ntype];
  return HG_OK;
}

hg_status hg_sample_blocks(hg_graph *g, const int64_t *const *seeds,
                           const int64_t *n_seeds, int32_t n_hops,
                           const int32_t *fanouts, uint64_t rng_seed,
                           hipStream_t stream, hg_blocks **out) {
  return hg_sample_blocks_ex(g, seeds, n_seeds, n_hops, fanouts, rng_seed, 32,
                             stream, out);
}

hg_status hg_graph_types(const hg_graph *g, int32_t *n_ntypes, int32_t *n_etypes) {
  if (!g) return fail(HG_EINVAL, "hg_graph_types: graph is NULL");
  if (n_ntypes) *n_ntypes = g->T;
  if (n_etypes) *n_etypes = g->R;
  return HG_OK;
}

int32_t hg_blocks_num_hops(const hg_blocks *b) { return b ? b->H : -1; }

hg_status hg_blocks_edge_counts(const hg_blocks *b, int64_t *counts) {
  if (!b || !counts) return fail(HG_EINVAL, "hg_blocks_edge_counts: NULL argument");
  for (size_t k = 0; k < b->n_edges.size(); ++k) counts[k] = b->n_edges[k];
  return HG_OK;
}

hg_status hg_blocks_counts(const hg_blocks *b, int64_t *n_dst, int64_t *n_src, int64_t *keys) {
  if (!b) return fail(HG_EINVAL, "hg_blocks_counts: blocks is NULL");
  for (size_t k = 0; k < b->n_dst.size(); ++k) {
    if (n_dst) n_dst[k] = b->n_dst[k];
    if (n_src) n_src[k] = b->n_src[k];
  }
  if (keys)
    for (size_t h = 0; h < b->keys.size(); ++h) keys[h] = b->keys[h];
  return HG_OK;
}

hg_status hg_blocks_nodes(const hg_blocks *b, int32_t hop, int32_t ntype,
                          int64_t *n_dst, int64_t *n_src,
                          const int64_t **src_gid) {
  if (!b) return fail(HG_EINVAL, "hg_blocks_nodes: blocks is NULL");
  if (hop < 0 || hop >= b->H || ntype < 0 || ntype >= b->T)
    return fail(HG_EINVAL, "hg_blocks_nodes: hop %d / node type %d out of range", hop, ntype);
  const size_t k = size_t(hop) * b->T + ntype;
  if (n_dst) *n_dst = b->n_dst[k];
  if (n_src) *n_src = b->n_src[k];
  if (src_gid) *src_gid = b->src_gid[k];
  return HG_OK;
}

hg_status hg_blocks_edges(const hg_blocks *b, int32_t hop, int32_t etype,
                          int64_t *n_edges, const int64_t **indptr,
                          const int32_t **src_local, const int32_t **dst_local,
                          const int64_t **eid) {
  if (!b) return fail(HG_EINVAL, "hg_blocks_edges: blocks is NULL");
  if (hop < 0 || hop >= b->H || etype < 0 || etype >= b->R)
    return fail(HG_EINVAL, "hg_blocks_edges: hop %d / edge type %d out of range", hop, etype);
  const size_t k = size_t(hop) * b->R + etype;
  if (n_edges) *n_edges = b->n_edges[k];
  if (indptr) *indptr = b->indptr[k];
  if (src_local) *src_local = b->src_local[k];
  if (dst_local) *dst_local = b->dst_local[k];
  if (eid) *eid = b->eid[k];
  return HG_OK;
}

hg_status hg_blocks_input_nodes(const hg_blocks *b, int32_t ntype, int64_t *n,
                                const int64_t **gid) {
  if (!b) return fail(HG_EINVAL, "hg_blocks_input_nodes: blocks is NULL");
  if (ntype < 0 || ntype >= b->T)
    return fail(HG_EINVAL, "hg_blocks_input_nodes: node type %d out of range", ntype);
  if (n) *n = b->in_n[ntype];
  if (gid) *gid = b->in_gid[ntype];
  return HG_OK;
}

hg_status hg_gather_rows(hg_graph *g, int32_t ntype, const int64_t *ids,
                         int64_t n, void *out, hipStream_t stream) {
  if (!g) return fail(HG_EINVAL, "hg_gather_rows: graph is NULL");
  if (ntype < 0 || ntype >= g->T)
    return fail(HG_EINVAL, "hg_gather_rows: node type %d out of range", ntype);
  const NTypeInfo &N = g->nt[ntype];
  if (N.dtype == HG_DT_NONE || N.row_bytes <= 0)
    return fail(HG_EINVAL, "hg_gather_rows: node type %d has no features", ntype);
  if (n < 0) return fail(HG_EINVAL, "hg_gather_rows: n < 0");
  if (n == 0) return HG_OK;
  if (!ids || !out) return fail(HG_EINVAL, "hg_gather_rows: NULL ids or out");
  DeviceGuard dg(g->device);
  clear_pending_error();
  // a workspace lends its readback slots: the kernel flags an ID out of range
  // in the error slot, which is read back once the gather has run
  Workspace *w = nullptr;
  hg_status st = acquire_workspace(g, 0, stream, &w);
  if (st != HG_OK) return st;
  int64_t *err_slot = w->dsmall + kSlotErr;
  const uint64_t seq = ++w->publish_seq;
  hipError_t e = launch_gather(N.feat, N.num_nodes, N.row_bytes, ids, n, out, stream, nullptr,
                               reinterpret_cast<unsigned long long *>(err_slot));
  if (e == hipSuccess)
    e = launch_publish(w->dsmall, w->hsmall, int32_t(small_slots(g)), seq, true, stream);
  if (e == hipSuccess) e = wait_flag(g, w, seq, stream);
  if (e != hipSuccess) {
    w->poisoned = true;
    release_workspace(g, w, stream);
    return fail_hip(e, "gather");
  }
  const int64_t bad = w->hsmall[kSlotErr];
  release_workspace(g, w, stream);
  if (bad)
    return fail(HG_EINVAL, "hg_gather_rows: %lld IDs are outside [0, %lld) of node type %d",
                static_cast<long long>(bad), static_cast<long long>(N.num_nodes), ntype);
  return HG_OK;
}

hg_status hg_gather_rows_noalloc(hg_graph *g, int32_t ntype, const int64_t *ids, int64_t n,
                                 void *out, hipStream_t stream) {
  if (!g) return fail(HG_EINVAL, "hg_gather_rows_noalloc: graph is NULL");
  if (ntype < 0 || ntype >= g->T)
    return fail(HG_EINVAL, "hg_gather_rows_noalloc: node type %d out of range", ntype);
  const NTypeInfo &N = g->nt[ntype];
  if (N.dtype == HG_DT_NONE || N.row_bytes <= 0)
    return fail(HG_EINVAL, "hg_gather_rows_noalloc: node type %d has no features", ntype);
  if (n < 0) return fail(HG_EINVAL, "hg_gather_rows_noalloc: n < 0");
  if (n == 0) return HG_OK;
  if (!ids || !out) return fail(HG_EINVAL, "hg_gather_rows_noalloc: NULL ids or out");
  DeviceGuard dg(g->device);
  clear_pending_error();
  // the GPU's copy of the static scratch array, looked up by hg_create
  unsigned long long *bad = noalloc_scratch(g->device);
  if (!bad) return fail(HG_EDEVICE, "hg_gather_rows_noalloc: no scratch address for the device");
  // the count starts at zero (a kernel, not a memset, clears it)
  hipError_t e = launch_fill_u32(reinterpret_cast<uint32_t *>(bad), 2, 0u, stream);
  if (e == hipSuccess)
    e = launch_gather(N.feat, N.num_nodes, N.row_bytes, ids, n, out, stream, nullptr, bad);
  unsigned long long host_bad = 0;
  if (e == hipSuccess)
    e = hipMemcpyAsync(&host_bad, bad, sizeof(host_bad), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return fail_hip(e, "hg_gather_rows_noalloc");
  if (host_bad)
    return fail(HG_EINVAL,
                "hg_gather_rows_noalloc: %llu IDs are outside [0, %lld) of node type %d",
                host_bad, static_cast<long long>(N.num_nodes), ntype);
  return HG_OK;
}

hg_status hg_gather_features(hg_graph *g, const hg_blocks *b, int32_t ntype,
                             void *out, hipStream_t stream) {
  if (!g || !b) return fail(HG_EINVAL, "hg_gather_features: NULL graph or blocks");
  if (b->g != g) return fail(HG_EINVAL, "hg_gather_features: blocks come from another graph");
  if (ntype < 0 || ntype >= g->T)
    return fail(HG_EINVAL, "hg_gather_features: node type %d out of range", ntype);
  const NTypeInfo &N = g->nt[ntype];
  if (N.dtype == HG_DT_NONE || N.row_bytes <= 0)
    return fail(HG_EINVAL, "hg_gather_features: node type %d has no features", ntype);
  const int64_t n = b->in_n[ntype];
  if (n == 0) return HG_OK;
  if (!out) return fail(HG_EINVAL, "hg_gather_features: out is NULL");
  // the input frontier holds valid IDs of the type by construction: no check
  DeviceGuard dg(g->device);
  clear_pending_error();
  hipError_t e = launch_gather(N.feat, N.num_nodes, N.row_bytes, b->in_gid[ntype], n, out, stream);
  if (e != hipSuccess) return fail_hip(e, "gather");
  return HG_OK;
}

hg_status hg_gather_features_multi(hg_graph *g, const hg_blocks *b,
                                   const int32_t *ntypes, void *const *outs,
                                   int32_t n, hipStream_t stream) {
  return hg_gather_features_multi_timed(g, b, ntypes, outs, n, stream, nullptr, nullptr);
}

hg_status hg_gather_features_multi_timed(hg_graph *g, const hg_blocks *b,
                                         const int32_t *ntypes, void *const *outs,
                                         int32_t n, hipStream_t stream, hipEvent_t start,
                                         hipEvent_t stop) {
  if (!g || !b) return fail(HG_EINVAL, "hg_gather_features_multi: NULL graph or blocks");
  if (b->g != g) return fail(HG_EINVAL, "hg_gather_features_multi: blocks come from another graph");
  if (n < 0 || (n > 0 && (!ntypes || !outs)))
    return fail(HG_EINVAL, "hg_gather_features_multi: bad type or output arrays");
  std::vector<GatherJob> jobs;
  for (int32_t k = 0; k < n; ++k) {
    const int32_t t = ntypes[k];
    if (t < 0 || t >= g->T)
      return fail(HG_EINVAL, "hg_gather_features_multi: node type %d out of range", t);
    const NTypeInfo &N = g->nt[t];
    if (N.dtype == HG_DT_NONE || N.row_bytes <= 0)
      return fail(HG_EINVAL, "hg_gather_features_multi: node type %d has no features", t);
    if (b->in_n[t] > 0 && !outs[k])
      return fail(HG_EINVAL, "hg_gather_features_multi: output %d is NULL", k);
    jobs.push_back(
        GatherJob{N.feat, N.num_nodes, N.row_bytes, b->in_gid[t], b->in_n[t], outs[k], nullptr});
  }
  DeviceGuard dg(g->device);
  clear_pending_error();
  hipError_t e = launch_gather_multi(jobs.data(), int32_t(jobs.size()), stream, start, stop);
  if (e != hipSuccess) return fail_hip(e, "gather");
  return HG_OK;
}

}  // extern "C"

namespace hg {

hg_status set_error(hg_status st, const char *msg) {
  g_last_error = msg;
  return st;
}

void blocks_detach_stream(hg_blocks *b) {
  b->stream = nullptr;
  if (b->mem) b->mem->stream = nullptr;
}

int graph_device(const hg_graph *g) { return g->device; }

}  // namespace hg

extern "C" {

void hg_blocks_free(hg_blocks *b) {
  delete b;  // the arrays go with the last handle that shares them
  clear_pending_error();
}

hg_status hg_bench_philox(uint64_t rng_seed, int32_t hop, int32_t etype, int64_t n_groups,
                          uint32_t lim, uint64_t *count, hipEvent_t start, hipEvent_t stop,
                          hipStream_t stream) {
  if (n_groups <= 0 || n_groups % 64 != 0 || n_groups > (int64_t(1) << 32) || !count ||
      hop < 0 || etype < 0)
    return fail(HG_EINVAL, "hg_bench_philox: bad arguments");
  clear_pending_error();
  hipError_t e = launch_philox_rate(rng_seed, hop, etype, n_groups, lim, count, start, stop,
                                    stream);
  if (e != hipSuccess) return fail_hip(e, "philox rate");
  return HG_OK;
}

hg_status hg_debug_philox(const uint32_t *ctr, uint64_t key, int64_t n,
                          uint32_t *out, hipStream_t stream) {
  if (n < 0 || (n > 0 && (!ctr || !out))) return fail(HG_EINVAL, "hg_debug_philox: bad arguments");
  clear_pending_error();
  hipError_t e = launch_philox(ctr, key, n, out, stream);
  if (e != hipSuccess) return fail_hip(e, "philox");
  return HG_OK;
}

}  // extern "C"
