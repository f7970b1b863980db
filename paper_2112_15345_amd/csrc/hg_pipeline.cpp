// Mini-batch pipeline of the C ABI in include/hg.h (DistDGLv2, arXiv
// 2112.15345, Sec. 4.2.1: mini-batches are generated ahead of their use by
// concurrent stages with bounded queues between them).
//
// Worker threads, each with its own HIP stream (and so its own workspace of the
// graph handle), take submitted mini-batches (single or bundled) in order and
// run them with hg_sample_blocks_bundle, or for layer-wise and edge-seeded
// submissions with hg_sample_layers_bundle and hg_sample_edge_blocks_bundle.
// While one worker waits on its stream (the per-hop size readbacks), the others
// keep the GPU busy, so the waits and the host's launch work of one mini-batch
// overlap the kernels of the next.  Results are handed back in submission
// order.
#include <condition_variable>
#include <deque>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "hg.h"
#include "hg_internal.hpp"

struct hg_pipeline {
  enum Kind { kVertex, kLayers, kEdges };
  // n mini-batches (a bundle when n > 1) with sequence numbers seq .. seq+n-1
  struct Job {
    Kind kind = kVertex;
    uint64_t seq = 0;
    int32_t n = 0;
    std::vector<const int64_t *> seeds;  // [n * T] (vertex, layers)
    std::vector<int64_t> n_seeds;        // [n * T]
    int32_t n_hops = 0;
    std::vector<int32_t> fanouts;        // [n_hops * R] fanouts, or [n_hops * T] layer sizes
    std::vector<uint64_t> sigmas;        // [n]
    hipEvent_t start = nullptr, stop = nullptr;
    bool timed = false;       // the stage events below apply
    hg_stage_events ev{};
    // edge-seeded batches: the host arrays of each hg_edge_batch, copied
    // ([n * R] each; the rev_* arrays only where the batch gives them)
    std::vector<const int64_t *> eids, rev_eid;
    std::vector<int64_t> n_eids;
    std::vector<int32_t> rev_etype;
    std::vector<int32_t> n_neg, exclude;        // [n]
    std::vector<uint8_t> has_rev_etype, has_rev_eid;  // [n]
  };
  struct Result {
    hg_blocks *b = nullptr;
    hg_status st = HG_OK;
    std::string err;
    hipEvent_t done = nullptr;
  };

  hg_graph *g = nullptr;
  int device = 0;
  int32_t T = 0, R = 0;
  int32_t capacity = 1;
  std::vector<int32_t> gather;
  std::vector<hipStream_t> streams;
  std::vector<std::thread> workers;

  std::mutex mu;
  std::condition_variable cv_job, cv_result, cv_space;
  std::deque<Job> jobs;
  std::map<uint64_t, Result> results;
  std::vector<hipEvent_t> free_events;
  uint64_t submitted = 0, returned = 0;
  bool stopping = false;

  void work(int k);
  hg_status run(Job &j, hipStream_t s, hg_blocks **out);
  hg_status enqueue(Job &&j);
};

hg_status hg_pipeline::run(Job &j, hipStream_t s, hg_blocks **out) {
  const int32_t *gt = gather.empty() ? nullptr : gather.data();
  const int32_t ng = int32_t(gather.size());
  const int32_t *fo = j.fanouts.empty() ? nullptr : j.fanouts.data();
  if (j.kind == kLayers)
    return hg_sample_layers_bundle(g, j.n, j.seeds.data(), j.n_seeds.data(), j.n_hops, fo,
                                   j.sigmas.data(), gt, ng, s, out);
  if (j.kind == kEdges) {
    std::vector<hg_edge_batch> eb(size_t(j.n));
    for (int32_t b = 0; b < j.n; ++b) {
      const size_t o = size_t(b) * size_t(R);
      eb[size_t(b)] = hg_edge_batch{j.eids.data() + o, j.n_eids.data() + o, j.n_neg[size_t(b)],
                                    j.exclude[size_t(b)],
                                    j.has_rev_etype[size_t(b)] ? j.rev_etype.data() + o : nullptr,
                                    j.has_rev_eid[size_t(b)] ? j.rev_eid.data() + o : nullptr};
    }
    return hg_sample_edge_blocks_bundle(g, j.n, eb.data(), j.n_hops, fo, j.sigmas.data(), gt, ng,
                                        s, out);
  }
  if (j.timed)
    return hg_sample_blocks_bundle_timed(g, j.n, j.seeds.data(), j.n_seeds.data(), j.n_hops, fo,
                                         j.sigmas.data(), gt, ng, &j.ev, s, out);
  return hg_sample_blocks_bundle(g, j.n, j.seeds.data(), j.n_seeds.data(), j.n_hops, fo,
                                 j.sigmas.data(), gt, ng, j.start, j.stop, s, out);
}

// Waits while the outstanding mini-batches would exceed the capacity, then
// queues the job under the next sequence numbers.
hg_status hg_pipeline::enqueue(Job &&j) {
  {
    std::unique_lock<std::mutex> lk(mu);
    cv_space.wait(lk, [&] { return submitted + uint64_t(j.n) - returned <= uint64_t(capacity); });
    j.seq = submitted;
    submitted += uint64_t(j.n);
    jobs.push_back(std::move(j));
  }
  cv_job.notify_one();
  return HG_OK;
}

void hg_pipeline::work(int k) {
  (void)hipSetDevice(device);
  hipStream_t s = streams[size_t(k)];
  for (;;) {
    Job j;
    {
      std::unique_lock<std::mutex> lk(mu);
      cv_job.wait(lk, [&] { return stopping || !jobs.empty(); });
      if (jobs.empty()) return;
      j = std::move(jobs.front());
      jobs.pop_front();
    }
    std::vector<hg_blocks *> out(size_t(j.n), nullptr);
    hg_status st = run(j, s, out.data());
    std::string err = st != HG_OK ? std::string(hg_last_error()) : std::string();
    std::vector<Result> rs(size_t(j.n));
    for (int32_t i = 0; i < j.n; ++i) {
      Result &r = rs[size_t(i)];
      r.st = st;
      r.err = err;
      r.b = out[size_t(i)];
      if (st != HG_OK) continue;
      {
        std::lock_guard<std::mutex> lk(mu);
        if (!free_events.empty()) {
          r.done = free_events.back();
          free_events.pop_back();
        }
      }
      hipError_t e = r.done ? hipSuccess : hipEventCreateWithFlags(&r.done, hipEventDisableTiming);
      if (e == hipSuccess) e = hipEventRecord(r.done, s);
      if (e != hipSuccess) {
        (void)hipGetLastError();
        r.err = std::string("pipeline: event: ") + hipGetErrorString(e);
        r.st = HG_EDEVICE;
      }
    }
    {
      std::lock_guard<std::mutex> lk(mu);
      for (int32_t i = 0; i < j.n; ++i) results.emplace(j.seq + uint64_t(i), std::move(rs[size_t(i)]));
    }
    cv_result.notify_all();
  }
}

extern "C" {

hg_status hg_pipeline_create(hg_graph *g, int32_t n_workers, int32_t capacity,
                             const int32_t *gather_ntypes, int32_t n_gather,
                             hg_pipeline **out) {
  if (!out) return hg::set_error(HG_EINVAL, "hg_pipeline_create: out is NULL");
  *out = nullptr;
  if (!g) return hg::set_error(HG_EINVAL, "hg_pipeline_create: graph is NULL");
  if (n_workers < 1 || n_workers > 16)
    return hg::set_error(HG_EINVAL, "hg_pipeline_create: n_workers not in 1..16");
  if (capacity < 1) return hg::set_error(HG_EINVAL, "hg_pipeline_create: capacity < 1");
  if (n_gather < 0 || (n_gather > 0 && !gather_ntypes))
    return hg::set_error(HG_EINVAL, "hg_pipeline_create: bad node type list");
  auto *p = new (std::nothrow) hg_pipeline();
  if (!p) return hg::set_error(HG_ENOMEM, "hg_pipeline_create: out of host memory");
  p->g = g;
  p->device = hg::graph_device(g);
  if (hg_graph_types(g, &p->T, &p->R) != HG_OK) {
    delete p;
    return HG_EINVAL;
  }
  p->capacity = capacity;
  p->gather.assign(gather_ntypes, gather_ntypes + n_gather);
  int prev = 0;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(p->device);
  for (int32_t k = 0; k < n_workers; ++k) {
    hipStream_t s = nullptr;
    if (hipStreamCreateWithFlags(&s, hipStreamNonBlocking) != hipSuccess) {
      (void)hipGetLastError();
      for (hipStream_t x : p->streams) (void)hipStreamDestroy(x);
      (void)hipSetDevice(prev);
      delete p;
      return hg::set_error(HG_EDEVICE, "hg_pipeline_create: stream creation failed");
    }
    p->streams.push_back(s);
  }
  (void)hipSetDevice(prev);
  try {
    for (int32_t k = 0; k < n_workers; ++k) p->workers.emplace_back(&hg_pipeline::work, p, k);
  } catch (...) {
    {
      std::lock_guard<std::mutex> lk(p->mu);
      p->stopping = true;
    }
    p->cv_job.notify_all();
    for (auto &t : p->workers) t.join();
    for (hipStream_t x : p->streams) (void)hipStreamDestroy(x);
    delete p;
    return hg::set_error(HG_ENOMEM, "hg_pipeline_create: cannot start worker threads");
  }
  *out = p;
  return HG_OK;
}

static hg_status submit_impl(hg_pipeline *p, int32_t n_batches, const int64_t *const *seeds,
                             const int64_t *n_seeds, int32_t n_hops,
                             const int32_t *fanouts, const uint64_t *rng_seeds,
                             hipEvent_t start, hipEvent_t stop, const hg_stage_events *ev) {
  if (!p) return hg::set_error(HG_EINVAL, "hg_pipeline_submit: pipeline is NULL");
  if (n_batches < 1 || n_batches > p->capacity)
    return hg::set_error(HG_EINVAL, "hg_pipeline_submit: n_batches not in 1..capacity");
  if (!n_seeds || !rng_seeds)
    return hg::set_error(HG_EINVAL, "hg_pipeline_submit: NULL n_seeds or rng_seeds");
  if (n_hops < 0) return hg::set_error(HG_EINVAL, "hg_pipeline_submit: n_hops < 0");
  int32_t T = 0, R = 0;
  if (hg_graph_types(p->g, &T, &R) != HG_OK) return HG_EINVAL;
  if (n_hops > 0 && R > 0 && !fanouts)
    return hg::set_error(HG_EINVAL, "hg_pipeline_submit: fanouts is NULL");
  const size_t nt = size_t(n_batches) * size_t(T);
  hg_pipeline::Job j;
  try {
    j.seeds.assign(nt, nullptr);
    if (seeds) j.seeds.assign(seeds, seeds + nt);
    j.n_seeds.assign(n_seeds, n_seeds + nt);
    if (fanouts) j.fanouts.assign(fanouts, fanouts + size_t(n_hops) * size_t(R));
    j.sigmas.assign(rng_seeds, rng_seeds + n_batches);
  } catch (const std::bad_alloc &) {
    return hg::set_error(HG_ENOMEM, "hg_pipeline_submit: out of host memory");
  }
  j.n = n_batches;
  j.n_hops = n_hops;
  j.start = start;
  j.stop = stop;
  if (ev) {
    j.timed = true;
    j.ev = *ev;
  }
  return p->enqueue(std::move(j));
}

hg_status hg_pipeline_submit(hg_pipeline *p, int32_t n_batches, const int64_t *const *seeds,
                             const int64_t *n_seeds, int32_t n_hops,
                             const int32_t *fanouts, const uint64_t *rng_seeds,
                             hipEvent_t start, hipEvent_t stop) {
  return submit_impl(p, n_batches, seeds, n_seeds, n_hops, fanouts, rng_seeds, start, stop,
                     nullptr);
}

hg_status hg_pipeline_submit_timed(hg_pipeline *p, int32_t n_batches,
                                   const int64_t *const *seeds, const int64_t *n_seeds,
                                   int32_t n_hops, const int32_t *fanouts,
                                   const uint64_t *rng_seeds, const hg_stage_events *events) {
  return submit_impl(p, n_batches, seeds, n_seeds, n_hops, fanouts, rng_seeds, nullptr, nullptr,
                     events);
}

hg_status hg_pipeline_submit_layers(hg_pipeline *p, int32_t n_batches,
                                    const int64_t *const *seeds, const int64_t *n_seeds,
                                    int32_t n_hops, const int32_t *layer_sizes,
                                    const uint64_t *rng_seeds) {
  if (!p) return hg::set_error(HG_EINVAL, "hg_pipeline_submit_layers: pipeline is NULL");
  if (n_batches < 1 || n_batches > p->capacity)
    return hg::set_error(HG_EINVAL, "hg_pipeline_submit_layers: n_batches not in 1..capacity");
  if (!n_seeds || !rng_seeds)
    return hg::set_error(HG_EINVAL, "hg_pipeline_submit_layers: NULL n_seeds or rng_seeds");
  if (n_hops < 0) return hg::set_error(HG_EINVAL, "hg_pipeline_submit_layers: n_hops < 0");
  if (n_hops > 0 && p->T > 0 && !layer_sizes)
    return hg::set_error(HG_EINVAL, "hg_pipeline_submit_layers: layer_sizes is NULL");
  const size_t nt = size_t(n_batches) * size_t(p->T);
  hg_pipeline::Job j;
  try {
    j.seeds.assign(nt, nullptr);
    if (seeds) j.seeds.assign(seeds, seeds + nt);
    j.n_seeds.assign(n_seeds, n_seeds + nt);
    if (layer_sizes) j.fanouts.assign(layer_sizes, layer_sizes + size_t(n_hops) * size_t(p->T));
    j.sigmas.assign(rng_seeds, rng_seeds + n_batches);
  } catch (const std::bad_alloc &) {
    return hg::set_error(HG_ENOMEM, "hg_pipeline_submit_layers: out of host memory");
  }
  j.kind = hg_pipeline::kLayers;
  j.n = n_batches;
  j.n_hops = n_hops;
  return p->enqueue(std::move(j));
}

hg_status hg_pipeline_submit_edges(hg_pipeline *p, int32_t n_batches,
                                   const hg_edge_batch *batches, int32_t n_hops,
                                   const int32_t *fanouts, const uint64_t *rng_seeds) {
  if (!p) return hg::set_error(HG_EINVAL, "hg_pipeline_submit_edges: pipeline is NULL");
  if (n_batches < 1 || n_batches > p->capacity)
    return hg::set_error(HG_EINVAL, "hg_pipeline_submit_edges: n_batches not in 1..capacity");
  if (!batches || !rng_seeds)
    return hg::set_error(HG_EINVAL, "hg_pipeline_submit_edges: NULL batches or rng_seeds");
  if (n_hops < 0) return hg::set_error(HG_EINVAL, "hg_pipeline_submit_edges: n_hops < 0");
  if (n_hops > 0 && p->R > 0 && !fanouts)
    return hg::set_error(HG_EINVAL, "hg_pipeline_submit_edges: fanouts is NULL");
  const size_t R = size_t(p->R);
  for (int32_t b = 0; b < n_batches; ++b)
    if (R > 0 && !batches[b].n_eids)
      return hg::set_error(HG_EINVAL, "hg_pipeline_submit_edges: a batch has no n_eids");
  hg_pipeline::Job j;
  try {
    const size_t nr = size_t(n_batches) * R;
    j.eids.assign(nr, nullptr);
    j.n_eids.assign(nr, 0);
    j.rev_etype.assign(nr, -1);
    j.rev_eid.assign(nr, nullptr);
    for (int32_t b = 0; b < n_batches; ++b) {
      const hg_edge_batch &x = batches[b];
      const size_t o = size_t(b) * R;
      for (size_t e = 0; e < R; ++e) {
        if (x.eids) j.eids[o + e] = x.eids[e];
        j.n_eids[o + e] = x.n_eids[e];
        if (x.rev_etype) j.rev_etype[o + e] = x.rev_etype[e];
        if (x.rev_eid) j.rev_eid[o + e] = x.rev_eid[e];
      }
      j.n_neg.push_back(x.n_neg);
      j.exclude.push_back(x.exclude);
      j.has_rev_etype.push_back(x.rev_etype ? 1 : 0);
      j.has_rev_eid.push_back(x.rev_eid ? 1 : 0);
    }
    if (fanouts) j.fanouts.assign(fanouts, fanouts + size_t(n_hops) * R);
    j.sigmas.assign(rng_seeds, rng_seeds + n_batches);
  } catch (const std::bad_alloc &) {
    return hg::set_error(HG_ENOMEM, "hg_pipeline_submit_edges: out of host memory");
  }
  j.kind = hg_pipeline::kEdges;
  j.n = n_batches;
  j.n_hops = n_hops;
  return p->enqueue(std::move(j));
}

hg_status hg_pipeline_next(hg_pipeline *p, hg_blocks **out) {
  if (!out) return hg::set_error(HG_EINVAL, "hg_pipeline_next: out is NULL");
  *out = nullptr;
  if (!p) return hg::set_error(HG_EINVAL, "hg_pipeline_next: pipeline is NULL");
  hg_pipeline::Result r;
  {
    std::unique_lock<std::mutex> lk(p->mu);
    if (p->returned == p->submitted)
      return hg::set_error(HG_EINVAL, "hg_pipeline_next: no mini-batch outstanding");
    const uint64_t seq = p->returned;
    p->cv_result.wait(lk, [&] { return p->results.count(seq) != 0; });
    auto it = p->results.find(seq);
    r = std::move(it->second);
    p->results.erase(it);
    p->returned++;
  }
  p->cv_space.notify_all();
  if (r.st != HG_OK) return hg::set_error(r.st, r.err.c_str());
  const hipError_t e = hipEventSynchronize(r.done);
  {
    std::lock_guard<std::mutex> lk(p->mu);
    p->free_events.push_back(r.done);
  }
  if (e != hipSuccess) {
    (void)hipGetLastError();
    hg_blocks_free(r.b);
    return hg::set_error(HG_EDEVICE, "hg_pipeline_next: device work of the mini-batch failed");
  }
  hg::blocks_detach_stream(r.b);
  *out = r.b;
  return HG_OK;
}

void hg_pipeline_destroy(hg_pipeline *p) {
  if (!p) return;
  {
    std::lock_guard<std::mutex> lk(p->mu);
    p->stopping = true;
  }
  p->cv_job.notify_all();
  for (auto &t : p->workers) t.join();
  int prev = 0;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(p->device);
  for (hipStream_t s : p->streams) (void)hipStreamSynchronize(s);
  for (auto &kv : p->results) {
    if (kv.second.b) {
      hg::blocks_detach_stream(kv.second.b);
      hg_blocks_free(kv.second.b);
    }
    if (kv.second.done) (void)hipEventDestroy(kv.second.done);
  }
  for (hipEvent_t e : p->free_events) (void)hipEventDestroy(e);
  // the graph's workspaces (and its bundle graphs') last used by the workers
  // hold events recorded on the worker streams: detach them before the
  // streams go away
  for (hipStream_t s : p->streams) (void)hg_retire_stream(p->g, s);
  for (hipStream_t s : p->streams) (void)hipStreamDestroy(s);
  (void)hipSetDevice(prev);
  (void)hipGetLastError();
  delete p;
}

}  // extern "C"
