// Internal interface between the host runtime (hg_runtime.cpp) and the gfx950
// kernels (hg_sample.hip, hg_compact.hip, hg_gather.hip).  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>

#include "hg.h"

#include <cstddef>
#include <cstdint>

namespace hg {

// Bitmap tiles: 256 threads x 2 words.
constexpr int kTileThreads = 256;
constexpr int kTileItems = 2;
constexpr int64_t kTile = int64_t(kTileThreads) * kTileItems;  // 512 words

// Pair tiles of the counting pass: 256 threads x 2 pairs.
// Pairs per thread of the counting pass: few for small hops (more blocks in
// flight), more for large ones (fewer tiles, whose tickets serialize).
constexpr int kPairItemsSmall = 2;
constexpr int kPairItemsLarge = 8;
constexpr int64_t kPairLargeFrom = int64_t(kTileThreads) * kPairItemsSmall * 512;
inline int pair_items(int64_t n_items) {
  return n_items >= kPairLargeFrom ? kPairItemsLarge : kPairItemsSmall;
}

// Candidate capacity of one bottom-K selection (LDS entries per wavefront,
// and per hub in the global candidate lists).
constexpr int kCandCap = 512;

// Node types whose per-hop table entries travel inside a launch's arguments.
constexpr int kInlineTypes = 8;
// Node types whose source-list pointers the sampler launch stores into the
// hop's table itself (a bundle of 32 mini-batches of 4 node types is 128).
constexpr int kInlineSrcOut = 128;

// Pairs whose in-edges are all kept and number at most this many are copied
// 64 pairs per wavefront; larger ones by a wavefront each.
constexpr int64_t kThreadTakeAll = 32;

// Pairs that keep K < deg edges with deg > kHubChunk ("hubs") are sampled in
// chunks of kHubChunk edges, handed to wavefronts in runs of chunks.
constexpr int64_t kHubChunk = 2048;

// Pairs that keep K < deg edges with deg <= kLaneSelect (and nothing
// excluded) are sampled by one lane each, among the pairs of the take-all
// groups: all their keys fit in registers.
constexpr int64_t kLaneSelect = 16;

// Readback slots of the small device buffer (int64 each).
constexpr int kSlotErr = 0;     // error bits in the low int32
constexpr int kSlotTicket = 1;  // tile tickets of the single-pass scans
constexpr int kSlotKeys = 2;    // random keys the sampler evaluates, summed over the hops so far
constexpr int kSlotPairs = 3;   // pairs of the hop
constexpr int kSlotEdges = 4;   // kept edges of the hop
constexpr int kSlotHubs = 5;    // hub pairs
constexpr int kSlotChunks = 6;  // hub chunks
constexpr int kSlotWaves = 7;   // pairs sampled by one wavefront each
constexpr int kSlotNew = 8;     // n_new[T], then ebase[R+1], then kept ebase[R+1]

constexpr int32_t kErrSeedRange = 1;   // a frontier vertex out of range
constexpr int32_t kErrSeedRepeat = 2;  // a vertex twice in a frontier
constexpr int32_t kErrLookback = 4;    // a scan wait exceeded its bound
constexpr int32_t kErrBound = 8;       // more pairs or chunks than buffers were sized for
constexpr int32_t kErrTarget = 16;     // a target edge out of range, or a bad reverse edge

// The dense vertex -> local-ID map of a workspace holds one int32 per vertex.
// An entry is meaningful only while the vertex's frontier bit is set (see
// TypeStatic); the frontier bitmap is cleared after every call, so stale
// entries are never read and the map itself is never cleared.

// Static per edge type (per workspace).
struct EtypeStatic {
  const int64_t *indptr;
  const int64_t *indices;
  int32_t *src_map;       // vertex -> local-ID map of the source type
  uint8_t *src_reached;   // reached flags of the source type
  uint32_t *src_rbits;    // reached bits of the source type (hops in bit mode)
  int64_t n_dst_nodes;
  int32_t src_type;
  int32_t dst_type;
  // Graphs with many edge types into one node type: per destination vertex a
  // row of nz_words words whose bit nz_slot says whether this edge type has
  // an in-edge there (nullptr: no mask, read indptr).
  const uint32_t *nz_mask;
  int32_t nz_words, nz_slot;
};

// Node types with at least this many incoming edge types get the mask above.
constexpr int32_t kNzMaskMinEtypes = 16;

// Static per node type (per workspace).
// Per node type one flag byte and one frontier bit per vertex: the sampler
// stores 1 into the `reached` byte of every kept edge's source (a plain store,
// so that popular sources cost no atomics), and `fbits` holds the frontier.  A
// hop's new vertices are the reached vertices whose frontier bit is clear; the
// compaction adds them to fbits and clears the reached bytes.  Both are zero
// between calls.  The layouts follow the bitmap tiles: type t starts at tile
// tile_base[t], a tile covering kTile * 32 vertices.
struct TypeStatic {
  int32_t *map;
  uint8_t *reached;
  uint32_t *fbits;
  int64_t num_nodes;
  uint32_t *rbits;  // reached bits (hops in bit mode), laid out as fbits
};

// A hop marks its kept sources either with the byte flags above (plain
// stores: no atomics on popular sources) or, when the call's vertices far
// outnumber the hop's kept edges, with one reached bit per vertex (atomicOr
// without return), so that the compaction reads an eighth of the bytes.
// Bit mode is chosen when vertices > kBitModeRatio x kept edges.
constexpr int64_t kBitModeRatio = 16;
// The chip's XCDs, each with its own L2; workgroups are handed to them in turn.
// A call of at least kXcds mini-batches orders its sampler, hub selection and relabel blocks
// per XCD, so that each XCD runs whole mini-batches.
constexpr int kXcds = 8;

// One hop, as device arrays.  Host-written: frontier, src_out, fanout.
// nF and pair_base are written by the host for hop 0 and by the previous
// hop's relabel pass afterwards.
struct HopView {
  int64_t *nF;                  // [T] frontier sizes
  int64_t *pair_base;           // [R+1] pairs of etype e: [pair_base[e], pair_base[e+1])
  const int64_t *const *frontier;  // [T]
  int64_t *const *src_out;      // [T] source lists of this hop (frontier ++ new)
  const int32_t *fanout;        // [R]
};

// Words of a single-pass (decoupled look-back) scan of NV values: per tile
// NV 64-bit words, each epoch (20 bits) | state (2 bits) | value (42 bits);
// state 1 = aggregate, overwritten by state 2 = inclusive prefix.  Epochs run 1 .. 2^20-1;
// the words are zeroed before an epoch is reused.
struct Lookback {
  uint64_t *word;
};
constexpr uint32_t kEpochLimit = 1u << 20;

// Edges that no hop may sample (an edge-seeded mini-batch with exclusion), as
// two open-addressing hash tables with linear probing: the excluded edges,
// keyed (etype << 32 | eid), and per pair with excluded in-edges its count,
// keyed (etype << 32 | destination local ID).  Every excluded edge ends at a
// seed, and the seeds are the first local IDs of every hop's frontier, so
// only pairs whose destination local ID is below n_seed[etype] are looked up.
// edge_keys == nullptr: nothing is excluded.
constexpr uint64_t kHashEmpty = ~uint64_t(0);
struct ExclView {
  const uint64_t *edge_keys;  // [edge_mask + 1]
  const uint64_t *pair_keys;  // [pair_mask + 1]
  const int32_t *pair_cnt;    // [pair_mask + 1]
  const int64_t *n_seed;      // [R] seeds of each etype's destination type
  uint32_t edge_mask, pair_mask;
};

__host__ __device__ inline uint32_t hash_slot(uint64_t key, uint32_t mask) {
  return uint32_t((key * 0x9E3779B97F4A7C15ull) >> 32) & mask;
}

// Per-pair arrays of one hop (device), n_items entries each.
struct PairArrays {
  int64_t *plo;      // first in-edge slot
  int64_t *pdeg;     // in-degree
  int64_t *off;      // exclusive scan of kept edges
  int32_t *pet;      // edge type of the pair
  int64_t *wlist;    // the pair of each wavefront pair, in pair order
  int32_t *hub_cnt;  // per hub: candidates appended
  int64_t *hub_pair; // per hub: its pair
  int64_t *hub_choff; // per hub: its first chunk (strictly increasing)
};

// ---- runtime hooks (hg_runtime.cpp) for the pipeline ------------------------

// Sets this thread's hg_last_error text; returns st.
hg_status set_error(hg_status st, const char *msg);
// Later frees of the handle's arrays are ordered on the null stream (its own
// stream is going away; its work has completed).
void blocks_detach_stream(hg_blocks *b);
int graph_device(const hg_graph *g);

// ---- launchers (all asynchronous on `stream`) -------------------------------

// Device timestamps of one stage: `start` is carried by the stage's first
// kernel launch and `stop` by its last; a stage that launches nothing records
// both with hipEventRecord.  Null events: plain launches.
struct StageEv {
  hipEvent_t start = nullptr, stop = nullptr;
  bool any() const { return start || stop; }
};
// Records an empty stage's events (no kernel to carry them).
hipError_t record_empty_stage(const StageEv &ev, hipStream_t stream);

// The hop-0 frontier: the seed's frontier bit, map[seed] = position; flags
// range errors and repeats (a frontier bit already set).
hipError_t launch_insert_frontier(HopView hv, const TypeStatic *ts,
                                  int32_t n_types, int64_t total, int64_t *small,
                                  hipStream_t stream);

// Counting pass over n_items >= P + 1 pair slots (P = pair_base[R]): per pair
// its in-edge range; exclusive scans of kept edges, hub chunks, wavefront
// pairs and hub flags; per-etype edge starts (ebase) and the hop totals into
// `small`.  Single pass, tiles taken by ticket.
int64_t count_tiles(int64_t n_items);
hipError_t launch_count_scan(HopView hv, const EtypeStatic *es, int32_t n_etypes,
                             int32_t n_types, int64_t n_items, PairArrays pa,
                             Lookback lb, uint32_t epoch, uint64_t ticket_base,
                             ExclView X, int64_t *small, hipStream_t stream,
                             StageEv ev = {});

// The sampler, two launches.  First: block CSC entries and small take-all
// pairs (a wavefront per 64 pairs), wavefront pairs (one wavefront each) and
// hub chunks (one wavefront each, appending candidates to the hub's list).
// Then one wavefront per hub selects from its list.  Writes each pair's kept
// edges at off[p], grouped by pair, ascending edge ID: source vertex, edge
// ID, destination local ID.
// The sampler launches.  With n_src_out <= kInlineSrcOut the first one also
// stores src_out[0..n_src_out) into src_out_slot (the hop's table entries).
// Edge type e is keyed as type e % key_R with seed sigmas[e / key_R] (device).
hipError_t launch_sample(HopView hv, const EtypeStatic *es, int32_t n_etypes,
                         int32_t n_types, int64_t n_pairs, int64_t n_wave,
                         int64_t n_chunks, int64_t n_hubs, PairArrays pa,
                         uint64_t *cand, const int64_t *small, const uint64_t *sigmas,
                         int32_t key_R, int32_t hop, int32_t key_bits, int64_t *src_gid,
                         int64_t *eid, int32_t *dst_local, int64_t *indptr_all,
                         int64_t **src_out_slot, int64_t *const *src_out, int32_t n_src_out,
                         ExclView X, hipStream_t stream, StageEv ev_sample = {},
                         StageEv ev_select = {}, bool bit_mode = false, bool xcd_order = false);


// Compaction pass: per bitmap tile, ranks of the set bits within the node
// type -> local IDs n_frontier + rank, written to the map and the source
// list, bits cleared; each type's new-vertex count goes to small[kSlotNew + t];
// extra blocks copy the frontier into the head of the source lists.  Up to
// kSinglePassTiles tiles: one launch, a single-pass scan whose look-back words
// are tile_sums (ticketed blocks: *ticketed is their number).  Beyond: three
// launches (reduce, scan, rank) with no inter-block waits; *ticketed = 0.
// tile_sums: device scratch of 2 * n_tiles + 2 64-bit words.  With `collect`
// the ranked vertices are only listed (in the source lists of hv, from local
// 0) and their reached flags cleared: the map and the frontier bits are left
// as they are.
constexpr int64_t kSinglePassTiles = 256;
hipError_t launch_compact(HopView hv, const TypeStatic *ts, int32_t n_types,
                          uint8_t *reached, uint32_t *fbits, const int64_t *tile_base,
                          int64_t n_tiles, int64_t copy_total, int64_t *tile_sums,
                          uint32_t epoch, uint64_t ticket_base, int64_t *small,
                          int64_t *ticketed, hipStream_t stream, bool collect = false,
                          StageEv ev = {}, uint32_t *rbits = nullptr);

// ---- layer-wise (LADIES) sampling (hg_layers.hip) ----------------------------

// One hop of a layer-wise call.  The sampler has emitted every in-edge of the
// frontier (all_src / all_eid / all_dst_local, grouped by pair at pa.off);
// per node type t (at most kInlineTypes), wt[t] holds the importance of every
// vertex (zero between uses), cand[t] and prefix[t] the candidates and the
// exclusive prefix of their importance, scan tiles cand_tile[t] ..
// cand_tile[t+1] of the candidate scan, and draws[t] the draws of the hop.
// Values per tile of the layer-wise scans (256 threads, two values each).
constexpr int64_t kLayerTile = 512;

struct LayerArgs {
  HopView hv, next;
  const EtypeStatic *es;
  const TypeStatic *ts;
  const int64_t *tile_base;  // bitmap tiles per type (plans the next hop)
  int32_t n_types, n_etypes;
  PairArrays pa;
  int64_t n_pairs;
  // n_all in-edges of the frontier, numbered by the counting pass (pair p's
  // in-edges are positions off[p] .. off[p+1]-1, CSC slots plo[p] ..); they
  // are read from the CSC where they are needed, never written out
  int64_t n_all;
  int64_t *tile_pair;  // [n_keep_tiles + 1]: the last pair with off <= tile * kLayerTile
  // per node type, in a device table of the hop (see LayerTable)
  uint64_t *const *wt;        // [T] importance of every vertex of the type
  int64_t *const *cand;       // [T] the type's candidates, ascending
  uint64_t *const *prefix;    // [T] their importance prefix
  const int64_t *cand_tile;   // [T+1] first scan tile of each type's candidates
  const int64_t *draw_base;   // [T+1] threads of the draw launch per type
  const int32_t *draws;       // [T] draws (-1: every candidate)
  int64_t cand_tiles, draw_threads;  // cand_tile[T], draw_base[T] (host copies)
  int64_t *tile_sum;   // per scan tile
  int64_t *tile_pre;   // per scan tile: exclusive scan over all tiles, then the grand total
  int64_t n_keep_tiles;
  int64_t *pos;        // [n_all + 1] exclusive scan of the kept flags
  int64_t *out_eid;
  int32_t *out_src_local, *out_dst_local;
  int64_t *out_indptr;  // [P + R]
  // node type t is keyed as type t % key_T with seed sigmas[t / key_T] (a
  // bundle's copy; a single batch: key_T = n_types)
  const uint64_t *sigmas;
  int32_t key_T;
  int32_t hop;
  int64_t *small;
};

// The per-type arrays of one layer-wise hop, as laid out in the call's
// tables (8-byte words): wt [T], cand [T], prefix [T], cand_tile [T+1],
// draw_base [T+1], draws [T] (int32, rounded up to words).
inline size_t layer_table_bytes(int32_t T) {
  return sizeof(int64_t) * (3 * size_t(T) + 2 * (size_t(T) + 1) + (size_t(T) + 1) / 2);
}

// The first pair of every kLayerTile-position tile of the in-edges (tile_pair),
// then the importance of every candidate: for each in-edge u -> v of the
// frontier whose source is not in the frontier, u is marked reached and
// wt[type(u)][u] += floor(2^32 / deg(v)^2).
hipError_t launch_lw_weights(const LayerArgs &A, hipStream_t stream);
// Exclusive prefix of the candidates' importance per node type (three
// launches: tile sums, one scan of the tile sums, apply); zeroes the
// candidates' importance entries.
hipError_t launch_lw_prefix(const LayerArgs &A, hipStream_t stream);
// The draws of every node type: marks the drawn candidates reached.
hipError_t launch_lw_draw(const LayerArgs &A, hipStream_t stream);
// The kept in-edges (source in the next frontier): scan of their flags,
// emitted in order; then the block CSC, the kept edge starts per etype
// (small slots after ebase) and the next hop's plan.
hipError_t launch_lw_keep(const LayerArgs &A, hipStream_t stream);

// src_local[j] = map_{src_type(e)}[src_gid[j]] for the edges of etype e,
// which are [ebase[e], ebase[e+1]), ebase = small + kSlotNew + n_types.
// Block 0 also writes the next hop's frontier sizes (this hop's plus its new
// vertices) and pair layout into `next`.
hipError_t launch_relabel(HopView hv, HopView next, const EtypeStatic *es,
                          const int64_t *tile_base, const int64_t *small,
                          int32_t n_types, int32_t n_etypes, int64_t n_edges,
                          const int64_t *src_gid, int32_t *src_local,
                          hipStream_t stream, StageEv ev = {}, bool xcd_order = false);

// Fill helpers (kernels, so that they are safe under graph capture).
// One block copies small[0..n) to pinned host memory host[0..n) and then
// writes `seq` to host[n] (system scope, after the slots).  With `clear` it
// then zeroes small[0..n), ready for the next call.
hipError_t launch_publish(int64_t *small, int64_t *host, int32_t n, uint64_t seq, bool clear,
                          hipStream_t stream);
// dst[i] = vals[i] for i < n (device pointer table), stream-ordered, with the
// values passed in the launches.
hipError_t launch_store_ptrs(void **dst, void *const *vals, int32_t n, hipStream_t stream);
hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t stream);
hipError_t launch_fill_u32(uint32_t *p, int64_t n, uint32_t v, hipStream_t stream);
// dst[0..n) = src[0..n) by a kernel that reads src, pinned host memory, over
// the host link (no DMA copy on the stream); dst and src 8-byte aligned, else
// hipErrorInvalidValue.  The host must not rewrite src until the kernel ran.
hipError_t launch_upload(void *dst, const void *src, int64_t n, hipStream_t stream);

// The non-empty mask of one destination type: for v < n, bit k of row v
// (words per row) is set when indptrs[k][v + 1] > indptrs[k][v]; indptrs is a
// device array of n_etypes pointers.
hipError_t launch_nonempty_mask(const int64_t *const *indptrs, int32_t n_etypes, int32_t words,
                                int64_t n, uint32_t *mask, hipStream_t stream);

// Graph check of one edge type: indptr[0] == 0, non-decreasing,
// indptr[n_dst] == nnz, indices in [0, n_src).  Sets *err on a violation.
hipError_t launch_check_etype(const int64_t *indptr, int64_t n_dst,
                              const int64_t *indices, int64_t nnz,
                              int64_t n_src, int32_t *err, hipStream_t stream);

// Row gather: out[i] = table[ids[i]] (row_bytes bytes); a zero row when the
// ID is out of range, which also adds 1 to *bad (when bad is not NULL).  Picks the widest vector width that divides row_bytes and the
// alignment of both pointers.
// With n_dev, the rows are min(*n_dev, n) (read on the device; n bounds them
// and sizes the grid).
hipError_t launch_gather(const void *table, int64_t n_rows, int64_t row_bytes,
                         const int64_t *ids, int64_t n, void *out,
                         hipStream_t stream, const int64_t *n_dev = nullptr,
                         unsigned long long *bad = nullptr);

// The allocation-free row pull keeps its counters in a static device array
// of this many bytes per GPU.  noalloc_scratch_init (with `device` current)
// looks up that GPU's address of the array once; noalloc_scratch returns it
// (NULL before the lookup).
constexpr size_t kNoAllocScratchBytes = HG_NOALLOC_SCRATCH_BYTES;
hipError_t noalloc_scratch_init(int device);
unsigned long long *noalloc_scratch(int device);

// One row gather of launch_gather_multi.
struct GatherJob {
  const void *table;
  int64_t n_rows;
  int64_t row_bytes;
  const int64_t *ids;
  int64_t n;             // rows (or, with n_dev, their bound)
  void *out;
  const int64_t *n_dev;  // device row count, or nullptr
};
// Several row gathers, as few launches as possible.  `start` / `stop` (may be
// NULL) are recorded by the batched launches themselves.
hipError_t launch_gather_multi(const GatherJob *jobs, int32_t n_jobs, hipStream_t stream,
                               hipEvent_t start, hipEvent_t stop);

// ---- edge-seeded mini-batches (hg_edges.hip) --------------------------------

// Per edge type of an edge-seeded call (device table).
struct EdgeEtype {
  const int64_t *eids;     // target edge IDs
  const int64_t *rev_eid;  // reverse edge ID of every edge (exclusion 2), or NULL
  int64_t nnz;
  int32_t rev;             // reverse edge type, or -1
};

struct EdgeBatchArgs {
  const EtypeStatic *es;
  const TypeStatic *ts;
  const EdgeEtype *et;     // [n_etypes]
  const int64_t *tbase;    // [n_etypes + 1] prefix of target counts
  int32_t n_etypes, n_types;
  int64_t n_targets;
  int32_t n_neg, exclude;
  // edge type e belongs to copy e / key_R of a bundle (a single batch: key_R
  // = n_etypes), keyed as type e % key_R with seed sigmas[e / key_R] (device)
  const uint64_t *sigmas;
  int32_t key_R;
  int64_t *tsrc, *tdst;    // [n_targets] endpoints (-1 for an invalid target)
  int64_t *tneg;           // [n_targets * n_neg]
  int64_t *trev;           // [n_targets] reverse edge ID (exclusion 2), -1 when none
  int32_t *pos_src, *pos_dst, *neg_dst;  // pair graphs, target order
  uint64_t *edge_keys, *pair_keys;
  int32_t *pair_cnt;
  int64_t *n_seed;         // [n_etypes]
  uint32_t edge_mask, pair_mask;
  int64_t *small;
};

// Endpoints and negatives of every target; sets their bitmap bits (the seeds,
// ranked by the compaction pass); flags bad targets and reverse edges.
hipError_t launch_edge_targets(const EdgeBatchArgs &A, hipStream_t stream);
// After the compaction of the seeds: the pair graphs' local IDs, the
// exclusion tables, and hop 0's frontier sizes and pair layout (`first`).
hipError_t launch_edge_relabel(const EdgeBatchArgs &A, HopView first,
                               const int64_t *tile_base, hipStream_t stream);

// Philox4x32-10 on n counters.
hipError_t launch_philox(const uint32_t *ctr, uint64_t key, int64_t n,
                         uint32_t *out, hipStream_t stream);

// The sampler's key loop alone over key groups 0 .. n_groups-1 (a multiple of
// 64) of (key, hop, etype): adds the number of keys <= lim to *count (device
// uint64).  start / stop (may be NULL) are carried by the launch.
hipError_t launch_philox_rate(uint64_t key, int32_t hop, int32_t etype, int64_t n_groups,
                              uint32_t lim, uint64_t *count, hipEvent_t start,
                              hipEvent_t stop, hipStream_t stream);

}  // namespace hg
