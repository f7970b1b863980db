// Host runtime of the C ABI in include/hg.h: argument checks, device
// workspaces, per-hop orchestration of the gfx950 kernels, and error state.
//
// One mini-batch (DistDGLv2, arXiv 2112.15345, Sec. 3.2 and Sec. 4.2.2) runs
// hop by hop.  Per hop:
//   1. count + scan   : kept-edge count of every (frontier vertex, etype)
//                       pair and its output offset;      -> wait #1 (sizes)
//   2. sample + mark  : the kept edges; new sources set a bitmap bit;
//      block CSC, popcount scan of the bitmap;           -> wait #2 (sizes)
//   3. assign + relabel: new vertices get local IDs in ascending ID order,
//                       edges get local source IDs.
// The source list of hop h is the frontier of hop h+1.
#include "hg.h"

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
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
  const void *feat;
  int32_t dtype;
  int32_t dim;
  int64_t row_bytes;
};

struct ETypeInfo {
  int32_t src, dst;
  int64_t nnz;
  const int64_t *indptr;
  const int64_t *indices;
};

// Per-call device state.  One call uses a workspace at a time; between calls
// the map is all -1 and the bitmap all 0.
struct Workspace {
  int32_t *map = nullptr;        // sum of num_nodes
  uint32_t *bitmap = nullptr;    // n_tiles * kTile words
  int64_t *tile_cnt = nullptr;   // n_tiles + 1
  int64_t *dsmall = nullptr;     // err | n_new[T] | ebase[R+1]
  int64_t *hsmall = nullptr;     // pinned mirror of dsmall
  char *dtab = nullptr;          // per-hop tables (device)
  char *htab = nullptr;          // per-hop tables (pinned host)
  size_t tab_cap = 0;
  hipEvent_t done = nullptr;
  bool busy = false;
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
  std::vector<int64_t> tile_base;  // [T+1]
  int64_t n_tiles = 0;
  int64_t *d_tile_base = nullptr;  // device copy of tile_base
  std::mutex mu;
  std::vector<Workspace *> ws;
};

struct hg_blocks {
  hg_graph *g = nullptr;
  hipStream_t stream = nullptr;
  int32_t H = 0, T = 0, R = 0;
  std::vector<int64_t> n_dst, n_src;  // [H*T]
  std::vector<int64_t *> src_gid;     // [H*T]
  std::vector<int64_t> n_edges;       // [H*R]
  std::vector<int64_t *> indptr;
  std::vector<int32_t *> src_local, dst_local;
  std::vector<int64_t *> eid;
  std::vector<int64_t> in_n;          // [T]
  std::vector<const int64_t *> in_gid;
  std::vector<void *> allocs;
};

// ---------------------------------------------------------------------------
// Device memory

namespace {

void *dev_alloc(hg_graph *g, size_t bytes, hipStream_t s) {
  bytes = align_up(bytes ? bytes : 1);
  if (g->has_alloc) return g->alloc.alloc(g->alloc.ctx, bytes, s);
  void *p = nullptr;
  if (hipMallocAsync(&p, bytes, s) != hipSuccess) {
    (void)hipGetLastError();
    return nullptr;
  }
  return p;
}

void dev_free(hg_graph *g, void *p, hipStream_t s) {
  if (!p) return;
  if (g->has_alloc)
    g->alloc.free(g->alloc.ctx, p, s);
  else
    (void)hipFreeAsync(p, s);
}

// Several arrays carved out of one allocation.
struct Arena {
  struct Req {
    void **slot;
    size_t bytes;
  };
  std::vector<Req> reqs;
  void *base = nullptr;
  template <typename T>
  void add(T **slot, int64_t n) {
    reqs.push_back({reinterpret_cast<void **>(slot),
                    align_up(size_t(std::max<int64_t>(n, 1)) * sizeof(T))});
  }
  bool allocate(hg_graph *g, hipStream_t s) {
    size_t total = 0;
    for (auto &r : reqs) total += r.bytes;
    base = dev_alloc(g, total, s);
    if (!base) return false;
    size_t off = 0;
    for (auto &r : reqs) {
      *r.slot = static_cast<char *>(base) + off;
      off += r.bytes;
    }
    return true;
  }
};

// Table layout of one region (one hop, or the seed/final steps).
struct RegionLayout {
  size_t etype_off, pbase_off, ntype_off, tbase_off, size;
  RegionLayout(int32_t T, int32_t R) {
    etype_off = 0;
    pbase_off = etype_off + align_up(sizeof(HopEtype) * size_t(std::max(R, 1)));
    ntype_off = pbase_off + align_up(sizeof(int64_t) * size_t(R + 1));
    tbase_off = ntype_off + align_up(sizeof(HopNtype) * size_t(T));
    size = tbase_off + align_up(sizeof(int64_t) * size_t(T + 1));
  }
};

void free_workspace(Workspace *w) {
  if (w->done) {
    (void)hipEventSynchronize(w->done);
    (void)hipEventDestroy(w->done);
  }
  (void)hipFree(w->map);
  (void)hipFree(w->bitmap);
  (void)hipFree(w->tile_cnt);
  (void)hipFree(w->dsmall);
  (void)hipFree(w->dtab);
  if (w->hsmall) (void)hipHostFree(w->hsmall);
  if (w->htab) (void)hipHostFree(w->htab);
  delete w;
}

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
    const size_t small_n = size_t(1 + g->T + g->R + 1);
    hipError_t e = hipSuccess;
    if (e == hipSuccess) e = hipMalloc(&w->map, sizeof(int32_t) * size_t(std::max<int64_t>(map_n, 1)));
    if (e == hipSuccess)
      e = hipMalloc(&w->bitmap, sizeof(uint32_t) * size_t(std::max<int64_t>(g->n_tiles * kTile, 1)));
    if (e == hipSuccess) e = hipMalloc(&w->tile_cnt, sizeof(int64_t) * size_t(g->n_tiles + 1));
    if (e == hipSuccess) e = hipMalloc(&w->dsmall, sizeof(int64_t) * small_n);
    if (e == hipSuccess) e = hipHostMalloc(reinterpret_cast<void **>(&w->hsmall), sizeof(int64_t) * small_n, 0);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&w->done, hipEventDisableTiming);
    if (e == hipSuccess) e = launch_fill_i32(w->map, map_n, -1, stream);
    if (e == hipSuccess) e = launch_fill_u32(w->bitmap, g->n_tiles * kTile, 0u, stream);
    if (e != hipSuccess) {
      free_workspace(w);
      return fail(HG_ENOMEM, "workspace allocation failed: %s", hipGetErrorString(e));
    }
    w->busy = true;
  } else {
    // the previous user may have run on another stream
    if (hipStreamWaitEvent(stream, w->done, 0) != hipSuccess) {
      std::lock_guard<std::mutex> lk(g->mu);
      w->busy = false;
      return fail_hip(hipGetLastError(), "hipStreamWaitEvent");
    }
  }
  if (w->tab_cap < tab_bytes) {
    // the tables of any earlier call were consumed before that call returned
    (void)hipFree(w->dtab);
    if (w->htab) (void)hipHostFree(w->htab);
    w->dtab = nullptr;
    w->htab = nullptr;
    w->tab_cap = 0;
    if (hipMalloc(&w->dtab, tab_bytes) != hipSuccess ||
        hipHostMalloc(reinterpret_cast<void **>(&w->htab), tab_bytes, 0) != hipSuccess) {
      (void)hipGetLastError();
      if (fresh) {
        free_workspace(w);
      } else {
        std::lock_guard<std::mutex> lk(g->mu);
        w->busy = false;
      }
      return fail(HG_ENOMEM, "workspace tables: allocation failed");
    }
    w->tab_cap = tab_bytes;
  }
  if (fresh) {
    std::lock_guard<std::mutex> lk(g->mu);
    g->ws.push_back(w);
  }
  *out = w;
  return HG_OK;
}

void release_workspace(hg_graph *g, Workspace *w, hipStream_t stream) {
  (void)hipEventRecord(w->done, stream);
  std::lock_guard<std::mutex> lk(g->mu);
  w->busy = false;
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
  uint64_t sigma;
  int32_t key_bits;
  const int32_t *fanouts;
  RegionLayout lay;

  std::vector<const int64_t *> F;   // current frontier per type
  std::vector<int64_t> nF;
  std::vector<void *> scratch;      // per-call temporaries
  // vertex lists that cover every map entry set so far
  std::vector<const int64_t *> map_lists;
  std::vector<int64_t> map_list_n;
  bool bitmap_dirty = false;

  SampleRun(hg_graph *g_, hipStream_t s, int32_t H_, const int32_t *fo,
            uint64_t sig, int32_t kb)
      : g(g_), stream(s), T(g_->T), R(g_->R), H(H_), sigma(sig), key_bits(kb),
        fanouts(fo), lay(g_->T, g_->R) {}

  char *htab(int region) { return ws->htab + size_t(region) * lay.size; }
  char *dtab(int region) { return ws->dtab + size_t(region) * lay.size; }

  hipError_t upload(int region, size_t off, size_t bytes) {
    return hipMemcpyAsync(dtab(region) + off, htab(region) + off, bytes,
                          hipMemcpyHostToDevice, stream);
  }

  // Writes the per-type table of `region` for `lists` and uploads it.
  hipError_t put_ntypes(int region, const std::vector<const int64_t *> &lists,
                        const std::vector<int64_t> &n,
                        const std::vector<int64_t *> &src_out, int64_t *total) {
    HopNtype *ht = reinterpret_cast<HopNtype *>(htab(region) + lay.ntype_off);
    int64_t *tb = reinterpret_cast<int64_t *>(htab(region) + lay.tbase_off);
    int64_t acc = 0;
    for (int32_t t = 0; t < T; ++t) {
      ht[t].frontier = lists[t];
      ht[t].n_frontier = n[t];
      ht[t].num_nodes = g->nt[t].num_nodes;
      ht[t].map = ws->map + g->map_off[t];
      ht[t].src_out = src_out.empty() ? nullptr : src_out[t];
      ht[t].new_base = 0;
      tb[t] = acc;
      acc += n[t];
    }
    tb[T] = acc;
    *total = acc;
    return upload(region, lay.ntype_off, lay.size - lay.ntype_off);
  }

  hipError_t sync_small(size_t first, size_t count) {
    hipError_t e = hipMemcpyAsync(ws->hsmall + first, ws->dsmall + first,
                                  sizeof(int64_t) * count, hipMemcpyDeviceToHost,
                                  stream);
    if (e != hipSuccess) return e;
    return hipStreamSynchronize(stream);
  }

  void *alloc_scratch(size_t bytes) {
    void *p = dev_alloc(g, bytes, stream);
    if (p) scratch.push_back(p);
    return p;
  }

  // Undoes the map and bitmap state; frees what the call took.
  void cleanup(bool keep_blocks) {
    if (bitmap_dirty) (void)launch_fill_u32(ws->bitmap, g->n_tiles * kTile, 0u, stream);
    int64_t total = 0;
    if (!map_lists.empty() &&
        put_ntypes(H + 1, map_lists, map_list_n, {}, &total) == hipSuccess) {
      (void)launch_reset_map(reinterpret_cast<const HopNtype *>(dtab(H + 1) + lay.ntype_off),
                             reinterpret_cast<const int64_t *>(dtab(H + 1) + lay.tbase_off),
                             T, total, stream);
    }
    for (void *p : scratch) dev_free(g, p, stream);
    scratch.clear();
    if (!keep_blocks && b) {
      for (void *p : b->allocs) dev_free(g, p, stream);
      delete b;
      b = nullptr;
    }
    release_workspace(g, ws, stream);
    ws = nullptr;
  }

  hg_status run(const int64_t *const *seeds, const int64_t *n_seeds);
};

hg_status SampleRun::run(const int64_t *const *seeds, const int64_t *n_seeds) {
  hipError_t e;
  b->g = g;
  b->stream = stream;
  b->H = H;
  b->T = T;
  b->R = R;
  b->n_dst.assign(size_t(H) * T, 0);
  b->n_src.assign(size_t(H) * T, 0);
  b->src_gid.assign(size_t(H) * T, nullptr);
  b->n_edges.assign(size_t(H) * R, 0);
  b->indptr.assign(size_t(H) * R, nullptr);
  b->src_local.assign(size_t(H) * R, nullptr);
  b->dst_local.assign(size_t(H) * R, nullptr);
  b->eid.assign(size_t(H) * R, nullptr);
  b->in_n.assign(T, 0);
  b->in_gid.assign(T, nullptr);

  F.assign(T, nullptr);
  nF.assign(T, 0);
  for (int32_t t = 0; t < T; ++t) {
    F[t] = n_seeds[t] > 0 ? seeds[t] : nullptr;
    nF[t] = n_seeds[t];
  }

  // ---- hop 0 frontier: insert the seeds into the map (checks them) -------
  int32_t *err = reinterpret_cast<int32_t *>(ws->dsmall);
  if ((e = launch_fill_i32(err, 2, 0, stream)) != hipSuccess) return fail_hip(e, "fill");
  int64_t total = 0;
  if ((e = put_ntypes(H, F, nF, {}, &total)) != hipSuccess) return fail_hip(e, "upload");
  map_lists = F;
  map_list_n = nF;
  if ((e = launch_insert_frontier(
           reinterpret_cast<const HopNtype *>(dtab(H) + lay.ntype_off),
           reinterpret_cast<const int64_t *>(dtab(H) + lay.tbase_off), T, total,
           err, stream)) != hipSuccess)
    return fail_hip(e, "insert seeds");
  if (H == 0) {
    if ((e = sync_small(0, 1)) != hipSuccess) return fail_hip(e, "sync");
    if (int32_t(ws->hsmall[0]) != 0)
      return fail(HG_EINVAL, "seeds: out of range or repeated within a node type");
  }

  const size_t o_new = 1, o_ebase = 1 + size_t(T);
  for (int32_t h = 0; h < H; ++h) {
    // ---- 1. pair table, count, scan -----------------------------------
    HopEtype *het = reinterpret_cast<HopEtype *>(htab(h) + lay.etype_off);
    int64_t *pb = reinterpret_cast<int64_t *>(htab(h) + lay.pbase_off);
    int64_t P = 0;
    for (int32_t ei = 0; ei < R; ++ei) {
      const ETypeInfo &E = g->et[ei];
      het[ei].frontier = F[E.dst];
      het[ei].indptr = E.indptr;
      het[ei].indices = E.indices;
      het[ei].src_map = ws->map + g->map_off[E.src];
      het[ei].src_bitmap = ws->bitmap + g->tile_base[E.src] * kTile;
      het[ei].pair_base = P;
      het[ei].n_pairs = nF[E.dst];
      het[ei].n_dst_nodes = g->nt[E.dst].num_nodes;
      het[ei].fanout = fanouts[size_t(h) * R + ei];
      het[ei].src_type = E.src;
      pb[ei] = P;
      P += nF[E.dst];
    }
    pb[R] = P;
    if ((e = upload(h, 0, lay.ntype_off)) != hipSuccess) return fail_hip(e, "upload");
    const HopEtype *d_et = reinterpret_cast<const HopEtype *>(dtab(h) + lay.etype_off);
    const int64_t *d_pb = reinterpret_cast<const int64_t *>(dtab(h) + lay.pbase_off);

    Arena sa;
    int64_t *cnt, *plo, *pdeg, *off, *scan_tmp;
    sa.add(&cnt, P);
    sa.add(&plo, P);
    sa.add(&pdeg, P);
    sa.add(&off, P + 1);
    sa.add(&scan_tmp, scan_scratch_elems(P));
    if (!sa.allocate(g, stream)) return fail(HG_ENOMEM, "hop %d: pair scratch", h);
    scratch.push_back(sa.base);
    int64_t *d_ebase = ws->dsmall + o_ebase;
    if ((e = launch_count(d_et, d_pb, R, P, cnt, plo, pdeg, err, stream)) != hipSuccess ||
        (e = launch_scan_i64(cnt, P, off, scan_tmp, stream)) != hipSuccess ||
        (e = launch_edge_bases(d_pb, off, R, d_ebase, stream)) != hipSuccess)
      return fail_hip(e, "count/scan");
    // wait #1: error flag and per-etype edge counts
    if ((e = sync_small(0, 1 + size_t(T) + size_t(R) + 1)) != hipSuccess)
      return fail_hip(e, "sync");
    if (int32_t(ws->hsmall[0]) != 0)
      return fail(HG_EINVAL, "seeds: out of range or repeated within a node type");
    const int64_t *ebase = ws->hsmall + o_ebase;
    std::vector<int64_t> eb(ebase, ebase + R + 1);
    const int64_t S = eb[R];

    // ---- 2. outputs of the hop, sampler, bitmap scan -------------------
    std::vector<int64_t> in_by_type(T, 0);
    for (int32_t ei = 0; ei < R; ++ei) in_by_type[g->et[ei].src] += eb[ei + 1] - eb[ei];
    Arena out;
    int64_t *indptr_all, *eid_all;
    int32_t *srcl_all, *dstl_all;
    std::vector<int64_t *> src_out(T, nullptr);
    out.add(&indptr_all, P + R);
    out.add(&eid_all, S);
    out.add(&srcl_all, S);
    out.add(&dstl_all, S);
    for (int32_t t = 0; t < T; ++t) {
      const int64_t bound = nF[t] + std::min(g->nt[t].num_nodes - nF[t], in_by_type[t]);
      out.add(&src_out[t], bound);
    }
    if (!out.allocate(g, stream)) return fail(HG_ENOMEM, "hop %d: block arrays", h);
    b->allocs.push_back(out.base);
    int64_t *gid_tmp = static_cast<int64_t *>(alloc_scratch(sizeof(int64_t) * size_t(std::max<int64_t>(S, 1))));
    if (!gid_tmp) return fail(HG_ENOMEM, "hop %d: edge scratch", h);

    bitmap_dirty = true;
    int64_t *d_new = ws->dsmall + o_new;
    if ((e = launch_sample(d_et, d_pb, R, P, cnt, plo, pdeg, off, sigma, h, key_bits,
                           gid_tmp, eid_all, dstl_all, stream)) != hipSuccess ||
        (e = launch_block_indptr(d_pb, off, R, P, indptr_all, stream)) != hipSuccess ||
        (e = launch_bitmap_tile_counts(ws->bitmap, g->n_tiles, ws->tile_cnt, stream)) != hipSuccess ||
        (e = launch_bitmap_scan(ws->tile_cnt, g->d_tile_base, T, d_new, stream)) != hipSuccess)
      return fail_hip(e, "sample");
    // wait #2: new-vertex counts
    if ((e = sync_small(o_new, size_t(T))) != hipSuccess) return fail_hip(e, "sync");
    std::vector<int64_t> U(ws->hsmall + o_new, ws->hsmall + o_new + T);
    for (int32_t t = 0; t < T; ++t)
      if (nF[t] + U[t] > INT32_MAX)
        return fail(HG_EUNSUPPORTED, "hop %d: more than 2^31-1 vertices of type %d", h, t);

    // ---- 3. local IDs of new vertices, destination prefix, relabel ------
    if ((e = put_ntypes(h, F, nF, src_out, &total)) != hipSuccess) return fail_hip(e, "upload");
    const HopNtype *d_nt = reinterpret_cast<const HopNtype *>(dtab(h) + lay.ntype_off);
    const int64_t *d_tb = reinterpret_cast<const int64_t *>(dtab(h) + lay.tbase_off);
    if ((e = launch_bitmap_assign(ws->bitmap, g->n_tiles, ws->tile_cnt, g->d_tile_base,
                                  d_nt, T, stream)) != hipSuccess)
      return fail_hip(e, "assign");
    bitmap_dirty = false;
    if ((e = launch_copy_frontier(d_nt, d_tb, T, total, stream)) != hipSuccess ||
        (e = launch_relabel(d_et, d_ebase, R, S, gid_tmp, srcl_all, stream)) != hipSuccess)
      return fail_hip(e, "relabel");

    for (int32_t t = 0; t < T; ++t) {
      const size_t k = size_t(h) * T + t;
      b->n_dst[k] = nF[t];
      b->n_src[k] = nF[t] + U[t];
      b->src_gid[k] = src_out[t];
      F[t] = src_out[t];
      nF[t] += U[t];
    }
    map_lists = F;
    map_list_n = nF;
    for (int32_t ei = 0; ei < R; ++ei) {
      const size_t k = size_t(h) * R + ei;
      b->n_edges[k] = eb[ei + 1] - eb[ei];
      b->indptr[k] = indptr_all + pb[ei] + ei;
      b->src_local[k] = srcl_all + eb[ei];
      b->dst_local[k] = dstl_all + eb[ei];
      b->eid[k] = eid_all + eb[ei];
    }
    for (void *p : scratch) dev_free(g, p, stream);
    scratch.clear();
  }

  // ---- input frontier ---------------------------------------------------
  if (H == 0) {
    Arena a;
    std::vector<int64_t *> cp(T, nullptr);
    for (int32_t t = 0; t < T; ++t) a.add(&cp[t], nF[t]);
    if (!a.allocate(g, stream)) return fail(HG_ENOMEM, "seed copy");
    b->allocs.push_back(a.base);
    for (int32_t t = 0; t < T; ++t) {
      if (nF[t] > 0 &&
          (e = hipMemcpyAsync(cp[t], F[t], sizeof(int64_t) * size_t(nF[t]),
                              hipMemcpyDeviceToDevice, stream)) != hipSuccess)
        return fail_hip(e, "seed copy");
      F[t] = cp[t];
    }
  }
  for (int32_t t = 0; t < T; ++t) {
    b->in_n[t] = nF[t];
    b->in_gid[t] = F[t];
  }
  return HG_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI

extern "C" {

const char *hg_last_error(void) { return g_last_error.c_str(); }

hg_status hg_create(const hg_ntype_desc *ntypes, int32_t n_ntypes,
                    const hg_etype_desc *etypes, int32_t n_etypes,
                    const hg_allocator *allocator, hipStream_t stream,
                    hg_graph **out) {
  if (!out) return fail(HG_EINVAL, "hg_create: out is NULL");
  *out = nullptr;
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
  g->map_off.assign(n_ntypes + 1, 0);
  g->tile_base.assign(n_ntypes + 1, 0);
  for (int32_t t = 0; t < n_ntypes; ++t) {
    const hg_ntype_desc &d = ntypes[t];
    g->nt.push_back({d.num_nodes, d.feat, d.dtype, d.dim, dtype_size(d.dtype) * int64_t(d.dim)});
    g->map_off[t + 1] = g->map_off[t] + d.num_nodes;
    const int64_t words = (d.num_nodes + 31) / 32;
    g->tile_base[t + 1] = g->tile_base[t] + (words + kTile - 1) / kTile;
  }
  g->n_tiles = g->tile_base[n_ntypes];
  for (int32_t i = 0; i < n_etypes; ++i) {
    const hg_etype_desc &d = etypes[i];
    g->et.push_back({d.src_type, d.dst_type, d.nnz, d.indptr, d.indices});
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
  *out = g;
  return HG_OK;
}

void hg_destroy(hg_graph *g) {
  if (!g) return;
  DeviceGuard dg(g->device);
  for (auto *w : g->ws) free_workspace(w);
  (void)hipFree(g->d_tile_base);
  delete g;
}

hg_status hg_sample_blocks_ex(hg_graph *g, const int64_t *const *seeds,
                              const int64_t *n_seeds, int32_t n_hops,
                              const int32_t *fanouts, uint64_t rng_seed,
                              int32_t key_bits, hipStream_t stream,
                              hg_blocks **out) {
  if (!out) return fail(HG_EINVAL, "hg_sample_blocks: out is NULL");
  *out = nullptr;
  if (!g) return fail(HG_EINVAL, "hg_sample_blocks: graph is NULL");
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
  DeviceGuard dg(g->device);
  SampleRun run(g, stream, n_hops, fanouts, rng_seed, key_bits);
  hg_status st = acquire_workspace(g, run.lay.size * size_t(n_hops + 2), stream, &run.ws);
  if (st != HG_OK) return st;
  run.b = new (std::nothrow) hg_blocks();
  if (!run.b) {
    run.cleanup(false);
    return fail(HG_ENOMEM, "hg_sample_blocks: out of host memory");
  }
  try {
    st = run.run(seeds, n_seeds);
  } catch (const std::bad_alloc &) {
    st = fail(HG_ENOMEM, "hg_sample_blocks: out of host memory");
  }
  if (st != HG_OK) {
    run.cleanup(false);
    return st;
  }
  hg_blocks *b = run.b;
  run.cleanup(true);
  *out = b;
  return HG_OK;
}

hg_status hg_sample_blocks(hg_graph *g, const int64_t *const *seeds,
                           const int64_t *n_seeds, int32_t n_hops,
                           const int32_t *fanouts, uint64_t rng_seed,
                           hipStream_t stream, hg_blocks **out) {
  return hg_sample_blocks_ex(g, seeds, n_seeds, n_hops, fanouts, rng_seed, 32,
                             stream, out);
}

int32_t hg_blocks_num_hops(const hg_blocks *b) { return b ? b->H : -1; }

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
  hipError_t e = launch_gather(N.feat, N.num_nodes, N.row_bytes, ids, n, out, stream);
  if (e != hipSuccess) return fail_hip(e, "gather");
  return HG_OK;
}

hg_status hg_gather_features(hg_graph *g, const hg_blocks *b, int32_t ntype,
                             void *out, hipStream_t stream) {
  if (!g || !b) return fail(HG_EINVAL, "hg_gather_features: NULL graph or blocks");
  if (b->g != g) return fail(HG_EINVAL, "hg_gather_features: blocks come from another graph");
  if (ntype < 0 || ntype >= g->T)
    return fail(HG_EINVAL, "hg_gather_features: node type %d out of range", ntype);
  return hg_gather_rows(g, ntype, b->in_gid[ntype], b->in_n[ntype], out, stream);
}

void hg_blocks_free(hg_blocks *b) {
  if (!b) return;
  DeviceGuard dg(b->g->device);
  for (void *p : b->allocs) dev_free(b->g, p, b->stream);
  delete b;
}

hg_status hg_debug_philox(const uint32_t *ctr, uint64_t key, int64_t n,
                          uint32_t *out, hipStream_t stream) {
  if (n < 0 || (n > 0 && (!ctr || !out))) return fail(HG_EINVAL, "hg_debug_philox: bad arguments");
  hipError_t e = launch_philox(ctr, key, n, out, stream);
  if (e != hipSuccess) return fail_hip(e, "philox");
  return HG_OK;
}

}  // extern "C"
