/*
 * oracle.h -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow CPU reference for heterogeneous multi-hop
 * fanout neighbour sampling, per-hop compaction into relabelled bipartite
 * blocks, and the gather of input-frontier features, as DistDGLv2 describes
 * them (arXiv 2112.15345: Sec. 3.2 "Mini-batch training", Sec. 4.2.2
 * "Distributed hybrid CPU/GPU sampling", Sec. 4.1.4 type-specific IDs).
 *
 * It is single-threaded as built for the tests; the same source built with
 * OpenMP shares independent loops out among threads (see oracle_threads) and
 * gives the same results.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may call it.  It shares no code, header, table or helper with the GPU
 * library; the two agree only through the written definition of the method.
 *
 * Status codes are plain ints with the same meaning as the GPU library's:
 *   0 ok, -1 invalid argument, -2 out of memory, -4 unsupported size.
 */
#ifndef ORACLE_H
#define ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)
#define ORACLE_ENOMEM (-2)
#define ORACLE_EUNSUPPORTED (-4)

/* One node type: its vertex count and (optionally) a row-major feature table
 * of num_nodes rows of row_bytes bytes each.  feat == NULL or row_bytes == 0
 * means the type carries no features. */
typedef struct {
  int64_t num_nodes;
  const void *feat;
  int64_t row_bytes;
} oracle_ntype;

/* One edge type (src_type -> dst_type) stored as CSC keyed by destination:
 * the in-edges of destination v are slots indptr[v] .. indptr[v+1]-1, and
 * indices[slot] is the source vertex (a type-specific ID of src_type).
 * The slot number is the edge ID. */
typedef struct {
  int32_t src_type;
  int32_t dst_type;
  int64_t nnz;
  const int64_t *indptr;  /* num_nodes(dst_type) + 1 entries */
  const int64_t *indices; /* nnz entries */
} oracle_etype;

typedef struct oracle_blocks oracle_blocks;

/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11) on one 128-bit counter
 * and a 64-bit key; writes the four 32-bit output words. */
void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2],
                          uint32_t out[4]);

/* The random key of edge `eid` of edge type `etype` at hop `hop` under
 * sampling seed `sigma`, truncated to its top `key_bits` bits. */
uint32_t oracle_edge_key(uint64_t sigma, int32_t hop, int32_t etype,
                         int64_t eid, int32_t key_bits);

/* Sampling of one (destination, edge type) pair whose in-edges are slots
 * lo .. hi-1: writes the chosen edge IDs, ascending, to out_eids (capacity
 * at least hi-lo) and their count to *n_out. */
int oracle_select(uint64_t sigma, int32_t hop, int32_t etype, int64_t lo,
                  int64_t hi, int32_t fanout, int32_t key_bits,
                  int64_t *out_eids, int64_t *n_out);

/* Checks a graph (types in range, indptr starts at 0, is non-decreasing and
 * ends at nnz, indices in range). */
int oracle_check_graph(const oracle_ntype *ntypes, int32_t n_ntypes,
                       const oracle_etype *etypes, int32_t n_etypes);

/* Full multi-hop sampling + compaction.  seeds[t] holds n_seeds[t] unique
 * vertex IDs of type t (seeds[t] may be NULL when n_seeds[t] == 0);
 * fanouts is hop-major [n_hops * n_etypes], -1 meaning "all in-edges". */
int oracle_sample_blocks(const oracle_ntype *ntypes, int32_t n_ntypes,
                         const oracle_etype *etypes, int32_t n_etypes,
                         const int64_t *const *seeds, const int64_t *n_seeds,
                         int32_t n_hops, const int32_t *fanouts, uint64_t sigma,
                         int32_t key_bits, oracle_blocks **out);

void oracle_blocks_free(oracle_blocks *b);

int oracle_blocks_nodes(const oracle_blocks *b, int32_t hop, int32_t ntype,
                        int64_t *n_dst, int64_t *n_src,
                        const int64_t **src_gid);

int oracle_blocks_edges(const oracle_blocks *b, int32_t hop, int32_t etype,
                        int64_t *n_edges, const int64_t **indptr,
                        const int32_t **src_local, const int32_t **dst_local,
                        const int64_t **eid);

/* The input frontier of type t: the source list of the last hop (the seeds
 * when n_hops == 0). */
int oracle_blocks_input_nodes(const oracle_blocks *b, int32_t ntype,
                              int64_t *n, const int64_t **gid);

/* out[i] = bytes of row ids[i] of a table of n_rows rows of row_bytes. */
int oracle_gather_rows(const void *feat, int64_t n_rows, int64_t row_bytes,
                       const int64_t *ids, int64_t n, void *out);

/* Threads the sampling and gather loops use: 1 in the plain build; in the
 * OpenMP build (the same source compiled with -fopenmp, where the pairs of a
 * hop, the relabelled edges and the gathered rows are shared out among the
 * threads) the OpenMP thread count. */
int oracle_threads(void);


/* ---- Edge-seeded mini-batches (link prediction; Sec. 4.2.1: the scheduler
 * picks target vertices or target edges).  See oracle.c for the readings. */

#define ORACLE_MAX_NEG 64

typedef struct {
  const int64_t *const *eids; /* [n_etypes] target edge IDs per edge type (NULL when none) */
  const int64_t *n_eids;      /* [n_etypes] */
  int32_t n_neg;              /* negatives per target, 0..ORACLE_MAX_NEG */
  int32_t exclude;            /* 0 none, 1 the targets, 2 the targets and their reverses */
  const int32_t *rev_etype;   /* [n_etypes] reverse edge type or -1 (exclude == 2) */
  const int64_t *const *rev_eid; /* [n_etypes] reverse edge ID of every edge (exclude == 2) */
} oracle_edge_batch;

/* The destination of edge `eid` of a CSC: the v with indptr[v] <= eid < indptr[v+1]. */
int oracle_edge_dst(const int64_t *indptr, int64_t n_dst, int64_t eid, int64_t *dst);

/* Negative k of target edge `eid` of `etype`: a destination uniform on
 * [0, n_dst), floor(u * n_dst / 2^64) with u = word0 | word1 << 32 of
 * Philox4x32-10 at counter (eid lo32, eid hi32, 2^31 | k, etype), key sigma. */
int oracle_negative_dst(uint64_t sigma, int32_t etype, int64_t eid, int32_t k,
                        int64_t n_dst, int64_t *v);

int oracle_sample_edge_blocks(const oracle_ntype *ntypes, int32_t n_ntypes,
                              const oracle_etype *etypes, int32_t n_etypes,
                              const oracle_edge_batch *batch, int32_t n_hops,
                              const int32_t *fanouts, uint64_t sigma, int32_t key_bits,
                              oracle_blocks **out);

/* Seeds of an edge-seeded result: the endpoints of node type t, ascending. */
int oracle_blocks_seeds(const oracle_blocks *b, int32_t ntype, int64_t *n,
                        const int64_t **gid);

/* Pair graph of edge type e: target i joins seeds pos_src[i] -> pos_dst[i];
 * negative i * n_neg + k joins pos_src[i] -> neg_dst[i * n_neg + k]. */
int oracle_blocks_pairs(const oracle_blocks *b, int32_t etype, int64_t *n_pos,
                        const int32_t **pos_src, const int32_t **pos_dst,
                        int64_t *n_negs, const int32_t **neg_dst);

/* ---- Layer-wise sampling (LADIES; see oracle.c for the readings). ---- */

/* floor(2^32 / deg^2): one edge's share of its source's importance. */
uint64_t oracle_layer_weight(int64_t deg);

/* Draw k of hop h and node type t: floor(x * total / 2^64), x = word0 |
 * word1 << 32 of Philox4x32-10 at counter (k lo32, k hi32, 2^30 | h, t). */
uint64_t oracle_layer_draw(uint64_t sigma, int32_t hop, int32_t ntype, int64_t k,
                           uint64_t total);

/* Layer-wise mini-batch: layer_sizes is hop-major [n_hops * n_ntypes], the
 * draws per hop and node type (-1 every candidate).  Results as
 * oracle_sample_blocks. */
int oracle_sample_layers(const oracle_ntype *ntypes, int32_t n_ntypes,
                         const oracle_etype *etypes, int32_t n_etypes,
                         const int64_t *const *seeds, const int64_t *n_seeds, int32_t n_hops,
                         const int32_t *layer_sizes, uint64_t sigma, oracle_blocks **out);

#ifdef __cplusplus
}
#endif

#endif
