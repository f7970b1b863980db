/*
 * hg.h -- C ABI of the MI355X (gfx950) heterogeneous mini-batch generator.
 *
 * One mini-batch of DistDGLv2's vertex-wise neighbour sampling on a
 * heterogeneous graph (arXiv 2112.15345): multi-hop, per-edge-type fanout
 * sampling of the seeds' in-neighbourhoods over CSC adjacency (Sec. 3.2,
 * Sec. 4.2.2), compaction of every hop into a relabelled bipartite block
 * (Sec. 4.2.1 pipeline stages, Sec. 4.2.2), and the gather of the input
 * frontier's feature rows (Sec. 4.2.1, the feature-copy stage, here a copy
 * inside HBM).  Vertex and edge IDs are type-specific (Sec. 4.1.4).
 *
 * Conventions shared by every call:
 *  - Pointers marked "device" are HIP device addresses on the current device;
 *    "host" pointers are read before the call returns.
 *  - All device work goes on the caller's `stream`.  hg_sample_blocks waits on
 *    that stream once per hop and once at the end, to size its outputs; the
 *    gathers of blocks' input frontiers are fully asynchronous, and
 *    hg_gather_rows waits once, to report IDs out of range.
 *  - Functions return hg_status; no C++ exception crosses this boundary.
 *    After a failure, hg_last_error() describes it (thread-local text, valid
 *    until the next call on the same thread).
 *  - Node types and edge types are the positions in the arrays given to
 *    hg_create; these indices enter the random key.
 */
#ifndef HG_H
#define HG_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum hg_status {
  HG_OK = 0,
  HG_EINVAL = -1,       /* an argument or an input value is invalid */
  HG_ENOMEM = -2,       /* an allocation failed */
  HG_EDEVICE = -3,      /* a HIP runtime call failed */
  HG_EUNSUPPORTED = -4  /* a size exceeds what the library supports */
} hg_status;

/* Element type of a feature table.  The gather copies bytes; the type only
 * fixes the element size (4, 2, 2 bytes). */
typedef enum hg_dtype {
  HG_DT_NONE = 0,
  HG_DT_F32 = 1,
  HG_DT_F16 = 2,
  HG_DT_BF16 = 3
} hg_dtype;

/* One node type (Sec. 4.1.4: features are stored per node type, in an ID
 * space of that type).  feat: row-major [num_nodes, dim] of `dtype`, rows
 * contiguous, in device memory or in pinned host memory (hipHostMalloc; the
 * paper keeps features in CPU memory, Sec. 4.1): the gathers read a pinned
 * table through its device mapping, over the host link, with no staging copy.
 * Pageable host memory is refused (HG_EINVAL).  NULL with dtype HG_DT_NONE for
 * a featureless type.  Borrowed: it must stay valid until hg_destroy. */
typedef struct hg_ntype_desc {
  int64_t num_nodes;
  const void *feat;
  int32_t dtype; /* hg_dtype */
  int32_t dim;
} hg_ntype_desc;

/* One edge type src_type -> dst_type as CSC keyed by destination: the
 * in-edges of destination v are slots indptr[v] .. indptr[v+1]-1 and
 * indices[slot] is the source vertex.  The slot number is the edge's ID.
 * Messages flow from in-neighbours to a vertex (Sec. 3.1, Eq. 1), so a
 * destination samples among its in-edges.
 * indptr: device int64 [num_nodes(dst_type) + 1]; indices: device int64 [nnz].
 * Borrowed until hg_destroy.  nnz must be below 2^32. */
typedef struct hg_etype_desc {
  int32_t src_type;
  int32_t dst_type;
  int64_t nnz;
  const int64_t *indptr;
  const int64_t *indices;
} hg_etype_desc;

/* Optional device allocator for the output arrays of hg_sample_blocks.
 * alloc returns NULL on failure (hg_sample_blocks then returns HG_ENOMEM and
 * releases what it took).  A NULL allocator means stream-ordered
 * allocations (hipMallocFromPoolAsync / hipFreeAsync) from the library's own
 * pool on the device, which keeps memory freed into it reserved until the
 * process ends.  Working memory (a per-vertex map and bitmap, per-pair and
 * per-edge scratch) belongs to the graph handle: it comes from that pool,
 * grows to the largest call and is returned to the pool by hg_destroy;
 * concurrent calls each get their own. */
typedef struct hg_allocator {
  void *ctx;
  void *(*alloc)(void *ctx, size_t bytes, hipStream_t stream);
  void (*free)(void *ctx, void *ptr, hipStream_t stream);
} hg_allocator;

typedef struct hg_graph hg_graph;
typedef struct hg_blocks hg_blocks;
typedef struct hg_pipeline hg_pipeline;

/* Creates an immutable graph handle over borrowed device arrays.
 * Checks the descriptors on the host and the arrays on the device (indptr
 * starts at 0, never decreases and ends at nnz; every index is a valid
 * source), synchronising `stream` once.  Returns HG_EINVAL on a bad
 * descriptor or array.  A node type with 16 or more incoming edge types gets
 * a graph-owned mask of ceil(k / 32) 32-bit words per vertex (k = its
 * incoming edge types) saying which of them have in-edges there; it lets the
 * sampler skip empty (vertex, edge type) pairs and is freed by hg_destroy.
 * The handle may be used from several threads and streams at once (the
 * graph is read-only, Sec. 4.2.1 ahead-of-time work on immutable data). */
hg_status hg_create(const hg_ntype_desc *ntypes, int32_t n_ntypes,
                    const hg_etype_desc *etypes, int32_t n_etypes,
                    const hg_allocator *allocator, hipStream_t stream,
                    hg_graph **out);

/* Releases the handle and its workspaces: waits for the handle's outstanding
 * work, frees its device memory, and leaves no HIP error pending on the
 * calling thread.  Every stream that calls on the handle used must still
 * exist, or have been passed to hg_retire_stream before it was destroyed. */
void hg_destroy(hg_graph *graph);

/* Detaches the graph's internal state from `stream` before the caller
 * destroys that stream.  A call leaves a marker of its working memory on
 * the stream it ran on, which the next call on another stream (or
 * hg_destroy) waits for; a marker on a destroyed stream must not be waited
 * for.  This waits for the graph's work on `stream` and drops those markers.
 * No call on this graph may be running on `stream` meanwhile.  Leaves no HIP
 * error pending.  HG_EINVAL for a NULL graph.  hg_pipeline_destroy does this
 * for its own worker streams. */
hg_status hg_retire_stream(hg_graph *graph, hipStream_t stream);

/* Number of node types and edge types of a graph handle (either output may
 * be NULL). */
hg_status hg_graph_types(const hg_graph *graph, int32_t *n_ntypes, int32_t *n_etypes);

/* One mini-batch (Sec. 3.2, Sec. 4.2.2).
 * seeds: host array of n_ntypes device pointers; seeds[t] holds n_seeds[t]
 *   int64 vertex IDs of type t, which must be unique and in range
 *   (HG_EINVAL otherwise); seeds[t] may be NULL when n_seeds[t] == 0.
 * n_seeds: host int64 [n_ntypes].
 * fanouts: host int32 [n_hops * n_etypes], hop-major; hop 0 starts from the
 *   seeds.  -1 keeps every in-edge, 0 none, K keeps min(deg, K).
 * rng_seed: sigma of the random key.  The kept in-edges of a destination are
 *   the K with the smallest (key, edge ID), key = output word (eid & 3) of
 *   Philox4x32-10 at counter (g lo32, g hi32, hop, etype), g = eid >> 2,
 *   with key (sigma lo32, sigma hi32).
 * Block h: per node type, the destination list is the hop's frontier and the
 *   source list is that frontier followed by the newly reached vertices in
 *   ascending ID; per edge type, the edges grouped by destination in frontier
 *   order and by ascending edge ID within a destination.  The source list of
 *   block h is the frontier of hop h+1 (Sec. 4.2.2).
 * On success *out owns every output array until hg_blocks_free.  On failure
 *   nothing is returned and every intermediate is released. */
hg_status hg_sample_blocks(hg_graph *graph, const int64_t *const *seeds,
                           const int64_t *n_seeds, int32_t n_hops,
                           const int32_t *fanouts, uint64_t rng_seed,
                           hipStream_t stream, hg_blocks **out);

/* hg_sample_blocks with only the top `key_bits` (1..32) bits of each key
 * compared, ties still broken by edge ID.  key_bits = 32 is hg_sample_blocks.
 * Small values make equal keys common; tests use it to exercise ties. */
hg_status hg_sample_blocks_ex(hg_graph *graph, const int64_t *const *seeds,
                              const int64_t *n_seeds, int32_t n_hops,
                              const int32_t *fanouts, uint64_t rng_seed,
                              int32_t key_bits, hipStream_t stream,
                              hg_blocks **out);

/* Number of hops of a blocks handle (-1 for NULL). */
int32_t hg_blocks_num_hops(const hg_blocks *blocks);

/* Kept edges of every block in one call: counts[hop * n_etypes + etype] for
 * every hop and edge type (host int64 [n_hops * n_etypes], caller-owned), as
 * hg_blocks_edges reports them one at a time.  HG_EINVAL for NULL arguments. */
hg_status hg_blocks_edge_counts(const hg_blocks *blocks, int64_t *counts);

/* Sizes of every block in one call (any output may be NULL; all host,
 * caller-owned): n_dst and n_src [n_hops * n_ntypes], hop-major, as
 * hg_blocks_nodes reports them one at a time; keys [n_hops], the random keys
 * the sampler evaluated in each hop (the in-degrees summed over every
 * (vertex, edge type) pair that chose K of more than K available in-edges:
 * Sec. 3.2 random choice, every candidate edge keyed once).  A handle of a
 * bundle reports the bundle's key totals.  HG_EINVAL for a NULL handle. */
hg_status hg_blocks_counts(const hg_blocks *blocks, int64_t *n_dst, int64_t *n_src,
                           int64_t *keys);

/* Vertices of node type `ntype` in block `hop` (Sec. 4.2.2: the frontier of
 * a hop is the unique set of vertices its sampled edges reach, and it seeds
 * the next hop; Sec. 4.2.1: compaction relabels the vertices of the
 * sampled subgraph): n_dst frontier vertices and n_src source vertices;
 * *src_gid: device int64 [n_src] whose first n_dst entries are the frontier
 * (local ID = position), followed by the newly reached vertices in ascending
 * ID.  Owned by the handle.  HG_EINVAL for a NULL handle, a hop outside
 * [0, n_hops) or a node type out of range; any output pointer may be NULL. */
hg_status hg_blocks_nodes(const hg_blocks *blocks, int32_t hop, int32_t ntype,
                          int64_t *n_dst, int64_t *n_src,
                          const int64_t **src_gid);

/* Edges of edge type `etype` in block `hop` (Sec. 3.2: at most K sampled
 * in-neighbours per destination; Sec. 4.2.1: compaction remaps the vertex
 * IDs and edge IDs of the sampled subgraph), all device, owned by the handle:
 * indptr int64 [n_dst(dst_type) + 1] (block CSC by destination local ID),
 * src_local / dst_local int32 [n_edges] (COO with local IDs), eid int64
 * [n_edges] (edge IDs of the input graph, type-specific as in Sec. 4.1.4).
 * HG_EINVAL for a NULL handle, a hop outside [0, n_hops) or an edge type out
 * of range.  Any output pointer may be NULL. */
hg_status hg_blocks_edges(const hg_blocks *blocks, int32_t hop, int32_t etype,
                          int64_t *n_edges, const int64_t **indptr,
                          const int32_t **src_local, const int32_t **dst_local,
                          const int64_t **eid);

/* The input frontier of node type `ntype`: the source list of the last hop,
 * or the seeds when n_hops == 0 (device int64 [n], owned by the handle).
 * These are the rows the feature copy needs (Sec. 4.2.1). */
hg_status hg_blocks_input_nodes(const hg_blocks *blocks, int32_t ntype,
                                int64_t *n, const int64_t **gid);

/* The feature copy of one node type (Sec. 4.2.1: the feature-copy stage
 * needs the frontier of the input layer; Sec. 4.1.4: features are stored per
 * node type): out[i, :] = feat_ntype[input_frontier[i], :], bits copied
 * unchanged.  out: device, caller-owned, [n_input(ntype), dim] of the type's
 * dtype.  HG_EINVAL for NULL arguments, blocks of another graph, a node type
 * out of range or a featureless type.  Asynchronous on `stream`. */
hg_status hg_gather_features(hg_graph *graph, const hg_blocks *blocks,
                             int32_t ntype, void *out, hipStream_t stream);

/* hg_gather_features for several node types at once, in as few launches as
 * possible: for k < n, outs[k] (device, caller-owned) receives the input
 * frontier rows of node type ntypes[k].  ntypes: host int32 [n]; outs: host
 * array of n device pointers.  HG_EINVAL if any type is featureless.
 * Asynchronous on `stream`. */
hg_status hg_gather_features_multi(hg_graph *graph, const hg_blocks *blocks,
                                   const int32_t *ntypes, void *const *outs,
                                   int32_t n, hipStream_t stream);

/* hg_gather_features_multi, with the 16-byte-vector gather launches
 * carrying `start` (first launch) and `stop` (last launch) as their own
 * timestamps (either may be NULL), so that hipEventElapsedTime(start, stop)
 * is the device time of those kernels.  For benchmarks. */
hg_status hg_gather_features_multi_timed(hg_graph *graph, const hg_blocks *blocks,
                                         const int32_t *ntypes, void *const *outs,
                                         int32_t n, hipStream_t stream,
                                         hipEvent_t start, hipEvent_t stop);

/* One mini-batch together with its input features (Sec. 4.2.1: a mini-batch
 * is the sampled blocks plus the features of the input frontier).  Samples as
 * hg_sample_blocks does, then gathers the input-frontier rows of every node
 * type in gather_ntypes (host int32 [n_gather], each featured and listed at
 * most once) into device arrays that the blocks handle owns; read them with
 * hg_blocks_features.  The outputs come from the graph's allocator like the
 * block arrays.  start / stop (either may be NULL) are carried by the gather
 * launches as in hg_gather_features_multi_timed.  HG_EINVAL for a bad type
 * list; otherwise as hg_sample_blocks.  The gather is asynchronous on
 * `stream` when the call returns. */
hg_status hg_sample_blocks_gather(hg_graph *graph, const int64_t *const *seeds,
                                  const int64_t *n_seeds, int32_t n_hops,
                                  const int32_t *fanouts, uint64_t rng_seed,
                                  const int32_t *gather_ntypes, int32_t n_gather,
                                  hipEvent_t start, hipEvent_t stop, hipStream_t stream,
                                  hg_blocks **out);

/* n_batches (1..32) mini-batches in one launch sequence (Sec. 4.2.2: the
 * sampling of several mini-batches is bundled so that it runs in parallel).
 * Batch b has seeds seeds[b * n_ntypes + t] with counts n_seeds[b * n_ntypes
 * + t] (host arrays) and sampling seed rng_seeds[b]; all share n_hops and
 * fanouts.  out: host array of n_batches handles, one per batch, each the
 * same mini-batch (blocks and gathered features) as
 * hg_sample_blocks_gather with that batch's arguments would give, each freed
 * by hg_blocks_free (the arrays of a bundle are released with its last
 * handle).  The batches are sampled together: each has its own frontier map
 * and compaction, every pass covers all of them, and the stream waits once
 * per hop for the whole bundle.  Working memory grows with n_batches.
 * All-or-nothing: an invalid batch fails the call. */
hg_status hg_sample_blocks_bundle(hg_graph *graph, int32_t n_batches,
                                  const int64_t *const *seeds, const int64_t *n_seeds,
                                  int32_t n_hops, const int32_t *fanouts,
                                  const uint64_t *rng_seeds, const int32_t *gather_ntypes,
                                  int32_t n_gather, hipEvent_t start, hipEvent_t stop,
                                  hipStream_t stream, hg_blocks **out);

/* Device timestamps of the stages of a sampling call, for benchmarks.  For
 * hop h < HG_MAX_TIMED_HOPS and stage s, start[h][s] / stop[h][s] (either may
 * be NULL) are carried by the first and the last kernel launch of that stage
 * (hipExtLaunchKernelGGL), so hipEventElapsedTime(start, stop) is the device
 * time of the stage's own kernels; a stage that launches nothing records both
 * events back to back.  The stages of one hop, in order: HG_STAGE_COUNT the
 * counting pass (kept edges per (vertex, edge type) pair and their offsets;
 * Sec. 3.2 at most K per pair), HG_STAGE_SAMPLE the sampler (the random choice
 * among in-edges and the emission of kept edges), HG_STAGE_SELECT the
 * selection of the K smallest keys of pairs with more candidate edges than
 * one wavefront holds, HG_STAGE_COMPACT the new frontier (the unique set of
 * reached vertices, Sec. 4.2.2) and HG_STAGE_RELABEL the local IDs of the
 * kept edges (Sec. 4.2.1 compaction).  gather_start / gather_stop are carried
 * by the feature gather launches.  The events belong to the caller, who
 * creates them (with timing) and keeps them until they have completed. */
#define HG_MAX_TIMED_HOPS 8
#define HG_STAGE_COUNT 0
#define HG_STAGE_SAMPLE 1
#define HG_STAGE_SELECT 2
#define HG_STAGE_COMPACT 3
#define HG_STAGE_RELABEL 4
#define HG_NUM_STAGES 5
typedef struct hg_stage_events {
  hipEvent_t start[HG_MAX_TIMED_HOPS][HG_NUM_STAGES];
  hipEvent_t stop[HG_MAX_TIMED_HOPS][HG_NUM_STAGES];
  hipEvent_t gather_start, gather_stop;
} hg_stage_events;

/* hg_sample_blocks_bundle with the stages' device timestamps (events may be
 * NULL: then it is hg_sample_blocks_bundle without gather events).  For a
 * bundle the stages cover all its mini-batches at once.  For benchmarks. */
hg_status hg_sample_blocks_bundle_timed(hg_graph *graph, int32_t n_batches,
                                        const int64_t *const *seeds, const int64_t *n_seeds,
                                        int32_t n_hops, const int32_t *fanouts,
                                        const uint64_t *rng_seeds, const int32_t *gather_ntypes,
                                        int32_t n_gather, const hg_stage_events *events,
                                        hipStream_t stream, hg_blocks **out);

/* The rows gathered for node type `ntype` by hg_sample_blocks_gather:
 * *rows = n_input(ntype) and *feat = device [rows, dim] of the type's dtype,
 * owned by the handle; *rows = 0 and *feat = NULL when the type was not
 * gathered.  Either output pointer may be NULL. */
hg_status hg_blocks_features(const hg_blocks *blocks, int32_t ntype, int64_t *rows,
                             const void **feat);

/* A pull of feature rows by vertex ID (Sec. 3.3: the KVStore's pull of
 * vertex features; Sec. 4.1.4: IDs are type-specific):
 * out[i, :] = feat_ntype[ids[i], :] for i < n.  ids: device int64 [n];
 * out: device, caller-owned, [n, dim] of the type's dtype.  Waits for
 * `stream` once (the kernel checks every ID on the device and the call reads
 * the result back): HG_EINVAL when an ID lies outside [0, num_nodes) of the
 * type (out then holds zero rows for those IDs and the other rows as
 * gathered), for a featureless or out-of-range type, NULL pointers or n < 0.
 * Concurrent calls on several streams are allowed. */
hg_status hg_gather_rows(hg_graph *graph, int32_t ntype, const int64_t *ids,
                         int64_t n, void *out, hipStream_t stream);

/* hg_gather_rows for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation.
 * Same arguments, output and errors as hg_gather_rows; it calls no hipMalloc,
 * hipFree or other allocating routine.  Its only scratch -- the count of IDs
 * out of range -- lives in a static device array of HG_NOALLOC_SCRATCH_BYTES
 * bytes that the library holds on every GPU it runs on until the process
 * ends (hg_create looks up that GPU's address of it).  The scratch does not
 * grow with n, so no size is refused for it.  Every call on a GPU shares that
 * GPU's array: the call clears the count with a kernel, gathers, copies the
 * count to the host and waits for `stream`; calls that overlap on one GPU
 * (from several threads or streams) race on the count and must be
 * serialised by the caller. */
#define HG_NOALLOC_SCRATCH_BYTES 256
hg_status hg_gather_rows_noalloc(hg_graph *graph, int32_t ntype, const int64_t *ids,
                                 int64_t n, void *out, hipStream_t stream);

/* Releases a blocks handle (stream-ordered on the stream it was made on;
 * on the null stream for handles returned by hg_pipeline_next), so that
 * stream must still exist.  A handle does not depend on its graph handle: it
 * may be released after hg_destroy (with a caller allocator, that allocator
 * must still work).  Leaves no HIP error pending. */
void hg_blocks_free(hg_blocks *blocks);

/* A mini-batch pipeline (Sec. 4.2.1: mini-batches are generated ahead of
 * their use by concurrent stages with bounded queues between them).
 * n_workers (1..16) host threads, each with its own HIP stream (created here,
 * default priority) and its own workspace of the graph, run submitted
 * mini-batches (single, or bundled as by hg_sample_blocks_bundle)
 * concurrently, so that the stream waits of one overlap the kernels of
 * another.  Mini-batches come back in
 * submission order; at most `capacity` (>= 1) are submitted and not yet
 * returned.  gather_ntypes (host int32 [n_gather], copied): the node types
 * whose input features every mini-batch gathers (may be empty).  The graph
 * must outlive the pipeline. */
hg_status hg_pipeline_create(hg_graph *graph, int32_t n_workers, int32_t capacity,
                             const int32_t *gather_ntypes, int32_t n_gather,
                             hg_pipeline **out);

/* Queues n_batches (1..capacity) mini-batches, sampled together as one
 * bundle when n_batches > 1: arguments as in hg_sample_blocks_bundle
 * (n_seeds, fanouts and rng_seeds are copied; the seed arrays are read on a
 * worker's stream and must stay valid until the mini-batches have been
 * returned by hg_pipeline_next).  start / stop: optional events carried by
 * the bundle's gather launches.  Each mini-batch is returned separately, in
 * submission order.  Waits while the outstanding mini-batches would exceed
 * `capacity`.  Argument errors found later (bad seeds, ...) fail the whole
 * bundle and are returned by hg_pipeline_next for each of its mini-batches. */
hg_status hg_pipeline_submit(hg_pipeline *pipe, int32_t n_batches,
                             const int64_t *const *seeds, const int64_t *n_seeds,
                             int32_t n_hops, const int32_t *fanouts,
                             const uint64_t *rng_seeds, hipEvent_t start, hipEvent_t stop);

/* hg_pipeline_submit with the stages' device timestamps of the bundle
 * (copied; see hg_sample_blocks_bundle_timed).  The events must stay valid
 * until the mini-batches have been returned. */
hg_status hg_pipeline_submit_timed(hg_pipeline *pipe, int32_t n_batches,
                                   const int64_t *const *seeds, const int64_t *n_seeds,
                                   int32_t n_hops, const int32_t *fanouts,
                                   const uint64_t *rng_seeds, const hg_stage_events *events);

/* Waits for the oldest outstanding mini-batch.  On success *out owns its
 * blocks and gathered features (hg_blocks_free) and all of its device work
 * has completed.  A mini-batch that failed returns its status (and
 * hg_last_error its text) with *out = NULL; later ones are unaffected.
 * HG_EINVAL when none is outstanding. */
hg_status hg_pipeline_next(hg_pipeline *pipe, hg_blocks **out);

/* Finishes the queued mini-batches, frees those not returned, stops the
 * workers, detaches the graph from their streams (hg_retire_stream) and
 * destroys them.  Leaves no HIP error pending. */
void hg_pipeline_destroy(hg_pipeline *pipe);

/* ---- Edge-seeded mini-batches (link prediction) ----------------------------
 * DistDGLv2's scheduler picks target vertices or target edges per mini-batch
 * (Sec. 4.2.1), and the same sampling decomposition runs from either (Sec.
 * 4.2.2).  From target edges:
 *  - a target is an edge ID (CSC slot) of an edge type; targets may repeat;
 *  - its endpoints are indices[eid] (source) and the destination v with
 *    indptr[v] <= eid < indptr[v+1];
 *  - n_neg negatives per target keep its source and take a destination
 *    uniform over the destination type: floor(u * n / 2^64), u = word0 |
 *    word1 << 32 of Philox4x32-10 at counter (eid lo32, eid hi32, 2^31 | k,
 *    etype) under key (rng_seed lo32, rng_seed hi32), k = 0 .. n_neg-1;
 *  - the seeds of a node type are its endpoints and negative destinations,
 *    each once, in ascending ID; the hops then run from them as in
 *    hg_sample_blocks;
 *  - exclusion removes edges from every hop's sampling: HG_EXCLUDE_SELF the
 *    targets, HG_EXCLUDE_REVERSE also each target's reverse edge
 *    rev_eid[e][eid] of type rev_etype[e] (which must run from the target's
 *    destination back to its source).  A pair keeps all its remaining
 *    in-edges when at most K remain, else the K remaining ones with the
 *    smallest (key, edge ID); keys are those of hg_sample_blocks. */
#define HG_MAX_NEG 64
#define HG_EXCLUDE_NONE 0
#define HG_EXCLUDE_SELF 1
#define HG_EXCLUDE_REVERSE 2

typedef struct hg_edge_batch {
  const int64_t *const *eids;    /* host array [n_etypes] of device int64 target IDs (NULL if none) */
  const int64_t *n_eids;         /* host int64 [n_etypes] */
  int32_t n_neg;                 /* negatives per target, 0 .. HG_MAX_NEG */
  int32_t exclude;               /* HG_EXCLUDE_* */
  const int32_t *rev_etype;      /* host int32 [n_etypes], -1 = no reverse (HG_EXCLUDE_REVERSE) */
  const int64_t *const *rev_eid; /* host array [n_etypes] of device int64 [nnz] (HG_EXCLUDE_REVERSE) */
} hg_edge_batch;

/* One edge-seeded mini-batch with its input features (gather_ntypes as in
 * hg_sample_blocks_gather).  HG_EINVAL for a bad argument, a target out of
 * range or a reverse edge that does not run back along its target; else as
 * hg_sample_blocks.  The target and reverse arrays are read on `stream`. */
hg_status hg_sample_edge_blocks(hg_graph *graph, const hg_edge_batch *batch, int32_t n_hops,
                                const int32_t *fanouts, uint64_t rng_seed,
                                const int32_t *gather_ntypes, int32_t n_gather,
                                hipStream_t stream, hg_blocks **out);

/* n_batches (1..32) edge-seeded mini-batches in one launch sequence, as
 * hg_sample_blocks_bundle does for vertex seeds: batch b is batches[b] with
 * seed rng_seeds[b] (host uint64 [n_batches]) and comes back in out[b], each
 * the mini-batch its own hg_sample_edge_blocks call would make.  All batches
 * share n_hops, fanouts, gather_ntypes and the batches' n_neg and exclude;
 * their target and reverse arrays may differ.  On failure no handle is
 * returned. */
hg_status hg_sample_edge_blocks_bundle(hg_graph *graph, int32_t n_batches,
                                       const hg_edge_batch *batches, int32_t n_hops,
                                       const int32_t *fanouts, const uint64_t *rng_seeds,
                                       const int32_t *gather_ntypes, int32_t n_gather,
                                       hipStream_t stream, hg_blocks **out);

/* The seeds of node type `ntype` (device int64 [n], owned by the handle): for
 * an edge-seeded batch its endpoints in ascending ID; otherwise the hop-0
 * frontier (the given seeds). */
hg_status hg_blocks_seeds(const hg_blocks *blocks, int32_t ntype, int64_t *n,
                          const int64_t **gid);

/* The pair graph of edge type `etype` of an edge-seeded batch, as local IDs
 * among the seeds (device int32, owned by the handle): target i joins
 * pos_src[i] -> pos_dst[i] (i < n_pos, in target order); negative
 * i * n_neg + k joins pos_src[i] -> neg_dst[i * n_neg + k] (n_negs = n_pos *
 * n_neg).  HG_EINVAL for a vertex-seeded batch. */
hg_status hg_blocks_edge_pairs(const hg_blocks *blocks, int32_t etype, int64_t *n_pos,
                               const int32_t **pos_src, const int32_t **pos_dst,
                               int64_t *n_negs, const int32_t **neg_dst);

/* ---- Layer-wise mini-batches (LADIES) ---------------------------------------
 * Sec. 4.2.2 names layer-wise sampling as fitting the same decomposition of
 * sampling, compaction and feature copy; the algorithm is LADIES (Zou et al.,
 * NeurIPS 2019, Algorithm 1).  Hop h, from its frontier (hop 0: the seeds):
 *  - the candidates of node type t are the sources of the frontier's in-edges
 *    (over every edge type whose source type is t) that are not in the
 *    frontier;
 *  - a candidate's importance is the sum over its edges u -> v into the
 *    frontier of floor(2^32 / deg_e(v)^2), deg_e(v) the in-degree of v in
 *    that edge type (an integer, so the sums are exact in any order);
 *  - layer_sizes[h * n_ntypes + t] = n draws n times with replacement among
 *    type t's candidates in ascending ID: draw k takes
 *    r = floor(x * total / 2^64), x = word0 | word1 << 32 of Philox4x32-10 at
 *    counter (k lo32, k hi32, 2^30 | h, t) under key (rng_seed lo32,
 *    rng_seed hi32), total = the candidates' importance sum, and picks the
 *    candidate whose interval [prefix, prefix + importance) holds r (none
 *    when total is 0); -1 takes every candidate, 0 none;
 *  - the hop's source vertices (the next frontier) are the frontier followed
 *    by the distinct drawn vertices in ascending ID;
 *  - its block keeps every in-edge of a frontier vertex whose source is in
 *    the next frontier, per destination in CSC slot order; local IDs as in
 *    hg_sample_blocks.
 * Seeds and the output handle are as for hg_sample_blocks (gather_ntypes as
 * in hg_sample_blocks_gather).  layer_sizes: host int32 [n_hops * n_ntypes],
 * each >= -1.  Errors as hg_sample_blocks. */
hg_status hg_sample_layers(hg_graph *graph, const int64_t *const *seeds, const int64_t *n_seeds,
                           int32_t n_hops, const int32_t *layer_sizes, uint64_t rng_seed,
                           const int32_t *gather_ntypes, int32_t n_gather, hipStream_t stream,
                           hg_blocks **out);

/* n_batches (1..32) layer-wise mini-batches in one launch sequence: batch b
 * takes seeds[b * n_ntypes + t] / n_seeds[b * n_ntypes + t] and seed
 * rng_seeds[b], shares n_hops and layer_sizes, and comes back in out[b] as
 * its own hg_sample_layers call would make it.  On failure no handle is
 * returned. */
hg_status hg_sample_layers_bundle(hg_graph *graph, int32_t n_batches,
                                  const int64_t *const *seeds, const int64_t *n_seeds,
                                  int32_t n_hops, const int32_t *layer_sizes,
                                  const uint64_t *rng_seeds, const int32_t *gather_ntypes,
                                  int32_t n_gather, hipStream_t stream, hg_blocks **out);

/* Pipeline submissions of layer-wise and edge-seeded mini-batches (Sec.
 * 4.2.1 and 4.2.2: the asynchronous pipeline serves every kind of sampling).
 * As hg_pipeline_submit, with the arguments of hg_sample_layers_bundle and
 * hg_sample_edge_blocks_bundle: a worker makes the n_batches (1..capacity;
 * more than 32 fail at the worker) mini-batches as one bundle, gathering the
 * pipeline's gather_ntypes, and hg_pipeline_next returns them one by one in
 * submission order.  Host arrays (n_seeds, layer_sizes, fanouts, rng_seeds,
 * each hg_edge_batch and the host arrays it points to) are copied; the device
 * arrays they point to (seeds, targets, reverse maps) are read on the
 * worker's stream and must stay valid until the mini-batches have been
 * returned.  HG_EINVAL here for a NULL or out-of-range argument; errors found
 * later fail the whole bundle at hg_pipeline_next. */
hg_status hg_pipeline_submit_layers(hg_pipeline *pipe, int32_t n_batches,
                                    const int64_t *const *seeds, const int64_t *n_seeds,
                                    int32_t n_hops, const int32_t *layer_sizes,
                                    const uint64_t *rng_seeds);
hg_status hg_pipeline_submit_edges(hg_pipeline *pipe, int32_t n_batches,
                                   const hg_edge_batch *batches, int32_t n_hops,
                                   const int32_t *fanouts, const uint64_t *rng_seeds);

/* Thread-local description of the last failure on this thread. */
const char *hg_last_error(void);

/* Philox4x32-10 on the device: out[4i..4i+3] = Philox4x32-10 of counter
 * ctr[4i..4i+3] under key (key lo32, key hi32), for i < n.
 * ctr, out: device uint32 [4n].  Asynchronous.  Exposes the generator the
 * sampler uses so that it can be checked on its own. */
hg_status hg_debug_philox(const uint32_t *ctr, uint64_t key, int64_t n,
                          uint32_t *out, hipStream_t stream);

/* The sampler's key loop on its own, for measuring its rate (the roof of the
 * selection among in-edges when keys must be computed for every candidate
 * edge, Sec. 3.2 random choice of at most K neighbours): evaluates the keys
 * of key groups g = 0 .. n_groups-1 of (rng_seed, hop, etype) -- the keys of
 * edge IDs 0 .. 4 * n_groups - 1, as hg_sample_blocks defines them -- with the
 * sampler's own code, and adds the number of keys <= lim to *count (device
 * uint64, caller-owned, not cleared).  n_groups: a positive multiple of 64,
 * at most 2^32.  start / stop (either may be NULL) are carried by the launch,
 * so hipEventElapsedTime(start, stop) is its device time.  Asynchronous. */
hg_status hg_bench_philox(uint64_t rng_seed, int32_t hop, int32_t etype, int64_t n_groups,
                          uint32_t lim, uint64_t *count, hipEvent_t start, hipEvent_t stop,
                          hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* HG_H */
