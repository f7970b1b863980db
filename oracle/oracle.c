/*
 * oracle.c -- TEST INFRASTRUCTURE ONLY (see oracle.h).
 *
 * Plain CPU reference of one mini-batch of DistDGLv2's vertex-wise neighbour
 * sampling on a heterogeneous graph, followed by per-hop compaction and the
 * gather of input-frontier features.  Everything here is written for a reader
 * checking it against the paper, not for speed: whole-array sorts, binary
 * searches and one Philox call per edge key.
 *
 * What the paper fixes:
 *  - A mini-batch starts from target ("seed") vertices; each target keeps at
 *    most K (the fanout) randomly chosen neighbours; this repeats recursively,
 *    one hop per GNN layer (Sec. 3.2).
 *  - Sampling goes one hop at a time; after a hop, the unique set of vertices
 *    (the frontier) seeds the next hop (Sec. 4.2.2).
 *  - Compaction removes empty vertices and relabels vertices and edges
 *    (Sec. 4.2.1 pipeline stages, Sec. 4.2.2).
 *  - Vertex and edge IDs are type-specific, unique only within their type
 *    (Sec. 4.1.4).
 *  - Messages flow from in-neighbours to a vertex (Sec. 3.1, Eq. 1), so a
 *    destination samples among its in-edges (CSC keyed by destination).
 *  - The input-layer frontier is what the feature copy needs (Sec. 4.2.1).
 *
 * Readings where the paper is silent (listed with their reasons in the design
 * notes of the repository):
 *  - "at most K randomly picked" is sampling without replacement: every
 *    in-edge is kept when deg <= K or K == -1; none when K == 0.
 *  - The random choice is made deterministic: the kept edges are the K with
 *    the smallest (key, edge ID), key = a 32-bit Philox4x32-10 output word of
 *    counter (g lo, g hi, hop, etype), g = eid >> 2, word eid & 3, under the
 *    64-bit key sigma; with key_bits < 32 only the top key_bits bits count
 *    (a test knob that makes ties common).
 *  - Fanouts are indexed by hop (hop 0 starts from the seeds) and edge type.
 *  - Edges of a block are grouped by destination in frontier order, and by
 *    ascending edge ID within one destination.
 *  - Source numbering of a block: the destination frontier first, in its
 *    given order, then the newly reached vertices in ascending vertex ID.
 *    Frontier vertices stay even when they sampled nothing.
 */
#include "oracle.h"

#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------ */
/* Philox4x32-10.  Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As
 * Easy as 1, 2, 3", SC'11, Sec. 3 (Philox): each round multiplies counter
 * words 0 and 2 by two fixed odd constants, xors the high halves of the
 * products with the other two counter words and the round key, and permutes
 * the words; the round key advances by a Weyl sequence (golden ratio and
 * sqrt(3)-1 constants) between rounds.  Ten rounds.                    */

static const uint32_t PHILOX_M0 = 0xD2511F53u;
static const uint32_t PHILOX_M1 = 0xCD9E8D57u;
static const uint32_t PHILOX_W0 = 0x9E3779B9u;
static const uint32_t PHILOX_W1 = 0xBB67AE85u;

void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2],
                          uint32_t out[4]) {
  uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += PHILOX_W0;
      k1 += PHILOX_W1;
    }
    uint64_t p0 = (uint64_t)PHILOX_M0 * (uint64_t)x0;
    uint64_t p1 = (uint64_t)PHILOX_M1 * (uint64_t)x2;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t y0 = hi1 ^ x1 ^ k0;
    uint32_t y1 = lo1;
    uint32_t y2 = hi0 ^ x3 ^ k1;
    uint32_t y3 = lo0;
    x0 = y0;
    x1 = y1;
    x2 = y2;
    x3 = y3;
  }
  out[0] = x0;
  out[1] = x1;
  out[2] = x2;
  out[3] = x3;
}

uint32_t oracle_edge_key(uint64_t sigma, int32_t hop, int32_t etype,
                         int64_t eid, int32_t key_bits) {
  uint64_t g = (uint64_t)eid >> 2;
  uint32_t ctr[4] = {(uint32_t)g, (uint32_t)(g >> 32), (uint32_t)hop,
                     (uint32_t)etype};
  uint32_t key[2] = {(uint32_t)sigma, (uint32_t)(sigma >> 32)};
  uint32_t out[4];
  oracle_philox4x32_10(ctr, key, out);
  uint32_t k = out[eid & 3];
  if (key_bits < 32) k >>= (32 - key_bits);
  return k;
}

/* ------------------------------------------------------------------ */
/* Choosing the neighbours of one (destination, edge type) pair.        */

typedef struct {
  uint32_t key;
  int64_t eid;
} keyed_edge;

static int cmp_keyed_edge(const void *a, const void *b) {
  const keyed_edge *x = (const keyed_edge *)a, *y = (const keyed_edge *)b;
  if (x->key != y->key) return x->key < y->key ? -1 : 1;
  if (x->eid != y->eid) return x->eid < y->eid ? -1 : 1;
  return 0;
}

static int cmp_i64(const void *a, const void *b) {
  int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
  return x < y ? -1 : (x > y ? 1 : 0);
}

/* index of x in the ascending array, or -1 */
static int64_t find_sorted(const int64_t *arr, int64_t n, int64_t x);

/* Sampling of one pair among its in-edges lo..hi-1 that are not in the
 * ascending list xs[0..nx) of excluded edge IDs: every remaining edge when
 * at most `fanout` remain (or fanout == -1), else the `fanout` remaining
 * edges with the smallest (key, eid); written in ascending edge ID. */
static int select_pair(uint64_t sigma, int32_t hop, int32_t etype, int64_t lo,
                       int64_t hi, int32_t fanout, int32_t key_bits,
                       const int64_t *xs, int64_t nx, int64_t *out_eids,
                       int64_t *n_out) {
  if (hi < lo || fanout < -1 || key_bits < 1 || key_bits > 32)
    return ORACLE_EINVAL;
  /* the in-edges that take part: every slot lo..hi-1 not excluded */
  int64_t deg = 0;
  for (int64_t j = lo; j < hi; ++j)
    if (nx == 0 || find_sorted(xs, nx, j) < 0) out_eids[deg++] = j;
  if (fanout < 0 || deg <= fanout) {
    /* keep every one of them, in slot order */
    *n_out = deg;
    return ORACLE_OK;
  }
  /* key every one, order by (key, eid), keep the first `fanout` */
  keyed_edge *all = (keyed_edge *)malloc(sizeof(keyed_edge) * (size_t)deg);
  if (!all) return ORACLE_ENOMEM;
  for (int64_t j = 0; j < deg; ++j) {
    all[j].eid = out_eids[j];
    all[j].key = oracle_edge_key(sigma, hop, etype, out_eids[j], key_bits);
  }
  qsort(all, (size_t)deg, sizeof(keyed_edge), cmp_keyed_edge);
  for (int64_t j = 0; j < fanout; ++j) out_eids[j] = all[j].eid;
  free(all);
  qsort(out_eids, (size_t)fanout, sizeof(int64_t), cmp_i64);
  *n_out = fanout;
  return ORACLE_OK;
}

int oracle_select(uint64_t sigma, int32_t hop, int32_t etype, int64_t lo,
                  int64_t hi, int32_t fanout, int32_t key_bits,
                  int64_t *out_eids, int64_t *n_out) {
  return select_pair(sigma, hop, etype, lo, hi, fanout, key_bits, NULL, 0,
                     out_eids, n_out);
}

/* ------------------------------------------------------------------ */
/* Input checks.                                                        */

int oracle_check_graph(const oracle_ntype *ntypes, int32_t n_ntypes,
                       const oracle_etype *etypes, int32_t n_etypes) {
  if (n_ntypes < 1 || n_etypes < 0 || !ntypes || (n_etypes > 0 && !etypes))
    return ORACLE_EINVAL;
  for (int32_t t = 0; t < n_ntypes; ++t) {
    if (ntypes[t].num_nodes < 0 || ntypes[t].row_bytes < 0)
      return ORACLE_EINVAL;
    if (ntypes[t].row_bytes > 0 && ntypes[t].num_nodes > 0 && !ntypes[t].feat)
      return ORACLE_EINVAL;
  }
  for (int32_t e = 0; e < n_etypes; ++e) {
    const oracle_etype *et = &etypes[e];
    if (et->src_type < 0 || et->src_type >= n_ntypes || et->dst_type < 0 ||
        et->dst_type >= n_ntypes || et->nnz < 0 || !et->indptr ||
        (et->nnz > 0 && !et->indices))
      return ORACLE_EINVAL;
    int64_t n_dst = ntypes[et->dst_type].num_nodes;
    int64_t n_src = ntypes[et->src_type].num_nodes;
    if (et->indptr[0] != 0 || et->indptr[n_dst] != et->nnz)
      return ORACLE_EINVAL;
    for (int64_t v = 0; v < n_dst; ++v)
      if (et->indptr[v + 1] < et->indptr[v]) return ORACLE_EINVAL;
    for (int64_t j = 0; j < et->nnz; ++j)
      if (et->indices[j] < 0 || et->indices[j] >= n_src)
        return ORACLE_EINVAL;
  }
  return ORACLE_OK;
}

/* ------------------------------------------------------------------ */
/* Result container.                                                    */

typedef struct {
  int64_t n_dst, n_src;
  int64_t *src_gid; /* n_src entries, the first n_dst being the frontier */
} onodes;

typedef struct {
  int64_t n_edges;
  int64_t *indptr; /* n_dst + 1 */
  int32_t *src_local;
  int32_t *dst_local;
  int64_t *eid;
} oedges;

struct oracle_blocks {
  int32_t n_hops, n_ntypes, n_etypes;
  onodes *nodes;   /* [n_hops * n_ntypes] */
  oedges *edges;   /* [n_hops * n_etypes] */
  int64_t *in_n;   /* [n_ntypes] */
  int64_t **in_gid;
  /* edge-seeded mini-batches only (NULL otherwise) */
  int64_t *seed_n;      /* [n_ntypes] */
  int64_t **seed_gid;   /* [n_ntypes] ascending */
  int32_t n_neg;
  int64_t *pair_n;      /* [n_etypes] target edges */
  int32_t **pos_src;    /* [n_etypes][pair_n] local IDs among the seeds */
  int32_t **pos_dst;
  int32_t **neg_dst;    /* [n_etypes][pair_n * n_neg] */
};

void oracle_blocks_free(oracle_blocks *b) {
  if (!b) return;
  if (b->nodes)
    for (int64_t i = 0; i < (int64_t)b->n_hops * b->n_ntypes; ++i)
      free(b->nodes[i].src_gid);
  if (b->edges)
    for (int64_t i = 0; i < (int64_t)b->n_hops * b->n_etypes; ++i) {
      free(b->edges[i].indptr);
      free(b->edges[i].src_local);
      free(b->edges[i].dst_local);
      free(b->edges[i].eid);
    }
  if (b->in_gid)
    for (int32_t t = 0; t < b->n_ntypes; ++t) free(b->in_gid[t]);
  if (b->seed_gid)
    for (int32_t t = 0; t < b->n_ntypes; ++t) free(b->seed_gid[t]);
  if (b->pos_src)
    for (int32_t e = 0; e < b->n_etypes; ++e) {
      free(b->pos_src[e]);
      free(b->pos_dst[e]);
      free(b->neg_dst[e]);
    }
  free(b->seed_n);
  free(b->seed_gid);
  free(b->pair_n);
  free(b->pos_src);
  free(b->pos_dst);
  free(b->neg_dst);
  free(b->nodes);
  free(b->edges);
  free(b->in_n);
  free(b->in_gid);
  free(b);
}

/* a vertex of the frontier with its position, for lookups by vertex ID */
typedef struct {
  int64_t gid;
  int64_t pos;
} gid_pos;

static int cmp_gid_pos(const void *a, const void *b) {
  const gid_pos *x = (const gid_pos *)a, *y = (const gid_pos *)b;
  return x->gid < y->gid ? -1 : (x->gid > y->gid ? 1 : 0);
}

/* position of gid in the sorted table, or -1 */
static int64_t find_gid_pos(const gid_pos *tab, int64_t n, int64_t gid) {
  int64_t a = 0, b = n;
  while (a < b) {
    int64_t m = a + (b - a) / 2;
    if (tab[m].gid < gid)
      a = m + 1;
    else
      b = m;
  }
  return (a < n && tab[a].gid == gid) ? tab[a].pos : -1;
}

/* index of gid in the ascending array, or -1 */
static int64_t find_sorted(const int64_t *arr, int64_t n, int64_t gid) {
  int64_t a = 0, b = n;
  while (a < b) {
    int64_t m = a + (b - a) / 2;
    if (arr[m] < gid)
      a = m + 1;
    else
      b = m;
  }
  return (a < n && arr[a] == gid) ? a : -1;
}

/* one sampled edge before relabelling */
typedef struct {
  int64_t src_gid;
  int32_t dst_local;
  int64_t eid;
} raw_edge;

/* ------------------------------------------------------------------ */
/* The mini-batch.                                                      */

/* Per edge type, an ascending list of edge IDs that no hop may sample (the
 * exclusion of an edge-seeded mini-batch); n == 0 excludes nothing. */
typedef struct {
  int64_t *eids;
  int64_t n;
} excl_list;

/* The hops of one mini-batch from a first frontier fr[t][0..fn[t]) that this
 * function takes over (and frees); fills b's blocks and input frontier. */
static int run_hops(const oracle_ntype *ntypes, int32_t n_ntypes,
                    const oracle_etype *etypes, int32_t n_etypes,
                    int64_t **fr, int64_t *fn, int32_t n_hops,
                    const int32_t *fanouts, uint64_t sigma, int32_t key_bits,
                    const excl_list *excl, oracle_blocks *b) {
  int status = ORACLE_OK;
  for (int32_t h = 0; h < n_hops && status == ORACLE_OK; ++h) {
    /* ---- Step 1: sample the neighbours of every (destination, etype)
     * pair of this hop's frontier, each pair independently. */
    raw_edge **sampled =
        (raw_edge **)calloc((size_t)n_etypes + 1, sizeof(raw_edge *));
    int64_t *n_sampled = (int64_t *)calloc((size_t)n_etypes + 1, sizeof(int64_t));
    if (!sampled || !n_sampled) {
      free(sampled);
      free(n_sampled);
      status = ORACLE_ENOMEM;
      break;
    }
    for (int32_t e = 0; e < n_etypes && status == ORACLE_OK; ++e) {
      const oracle_etype *et = &etypes[e];
      int32_t t = et->dst_type;
      int32_t k = fanouts[(int64_t)h * n_etypes + e];
      oedges *blk = &b->edges[(int64_t)h * n_etypes + e];
      blk->indptr = (int64_t *)malloc(sizeof(int64_t) * (size_t)(fn[t] + 1));
      if (!blk->indptr) {
        status = ORACLE_ENOMEM;
        break;
      }
      /* the block's CSC: destination i keeps min(avail, k) edges (every one
       * when k == -1), avail = its in-edges that are not excluded */
      blk->indptr[0] = 0;
      for (int64_t i = 0; i < fn[t]; ++i) {
        int64_t v = fr[t][i];
        int64_t avail = et->indptr[v + 1] - et->indptr[v];
        if (excl[e].n > 0)
          for (int64_t j = et->indptr[v]; j < et->indptr[v + 1]; ++j)
            if (find_sorted(excl[e].eids, excl[e].n, j) >= 0) --avail;
        int64_t kept = (k < 0 || avail <= k) ? avail : k;
        blk->indptr[i + 1] = blk->indptr[i] + kept;
      }
      int64_t cnt = blk->indptr[fn[t]];
      sampled[e] = (raw_edge *)malloc(sizeof(raw_edge) * (size_t)(cnt + 1));
      if (!sampled[e]) {
        status = ORACLE_ENOMEM;
        break;
      }
      /* every destination on its own; they share nothing, so an OpenMP build
       * runs them in parallel (the paper bundles this step with OpenMP, Sec.
       * 4.2.2), each writing its own slots of the block */
      int pair_status = ORACLE_OK;
#pragma omp parallel for schedule(dynamic, 8)
      for (int64_t i = 0; i < fn[t]; ++i) {
        int64_t v = fr[t][i];
        int64_t lo = et->indptr[v], hi = et->indptr[v + 1];
        int64_t *chosen = (int64_t *)malloc(sizeof(int64_t) * (size_t)(hi - lo + 1));
        int64_t nc = 0;
        int st = chosen ? select_pair(sigma, h, e, lo, hi, k, key_bits, excl[e].eids,
                                      excl[e].n, chosen, &nc)
                        : ORACLE_ENOMEM;
        if (st == ORACLE_OK && nc != blk->indptr[i + 1] - blk->indptr[i]) st = ORACLE_EINVAL;
        if (st == ORACLE_OK) {
          for (int64_t c = 0; c < nc; ++c) {
            raw_edge *r = &sampled[e][blk->indptr[i] + c];
            r->src_gid = et->indices[chosen[c]];
            r->dst_local = (int32_t)i;
            r->eid = chosen[c];
          }
        } else {
#pragma omp atomic write
          pair_status = st;
        }
        free(chosen);
      }
      if (pair_status != ORACLE_OK) {
        status = pair_status;
        break;
      }
      n_sampled[e] = cnt;
    }

    /* ---- Step 2: the frontier of the next hop, per node type: the unique
     * set of this hop's vertices -- the current frontier (kept in its order)
     * followed by the newly reached sources in ascending ID. */
    int64_t **nf = (int64_t **)calloc((size_t)n_ntypes, sizeof(int64_t *));
    int64_t *nfn = (int64_t *)calloc((size_t)n_ntypes, sizeof(int64_t));
    gid_pos **ftab = (gid_pos **)calloc((size_t)n_ntypes, sizeof(gid_pos *));
    int64_t *n_new = (int64_t *)calloc((size_t)n_ntypes, sizeof(int64_t));
    if (!nf || !nfn || !ftab || !n_new) status = ORACLE_ENOMEM;
    for (int32_t t = 0; t < n_ntypes && status == ORACLE_OK; ++t) {
      /* the current frontier as a (gid, position) lookup table */
      ftab[t] = (gid_pos *)malloc(sizeof(gid_pos) * (size_t)(fn[t] + 1));
      if (!ftab[t]) {
        status = ORACLE_ENOMEM;
        break;
      }
      for (int64_t i = 0; i < fn[t]; ++i) {
        ftab[t][i].gid = fr[t][i];
        ftab[t][i].pos = i;
      }
      qsort(ftab[t], (size_t)fn[t], sizeof(gid_pos), cmp_gid_pos);
      /* every sampled source of type t */
      int64_t total = 0;
      for (int32_t e = 0; e < n_etypes; ++e)
        if (etypes[e].src_type == t) total += n_sampled[e];
      int64_t *srcs = (int64_t *)malloc(sizeof(int64_t) * (size_t)(total + 1));
      if (!srcs) {
        status = ORACLE_ENOMEM;
        break;
      }
      int64_t m = 0;
      for (int32_t e = 0; e < n_etypes; ++e)
        if (etypes[e].src_type == t)
          for (int64_t j = 0; j < n_sampled[e]; ++j)
            srcs[m++] = sampled[e][j].src_gid;
      qsort(srcs, (size_t)m, sizeof(int64_t), cmp_i64);
      /* unique, and not already in the frontier */
      int64_t u = 0;
      for (int64_t j = 0; j < m; ++j) {
        if (j > 0 && srcs[j] == srcs[j - 1]) continue;
        if (find_gid_pos(ftab[t], fn[t], srcs[j]) >= 0) continue;
        srcs[u++] = srcs[j];
      }
      n_new[t] = u;
      nfn[t] = fn[t] + u;
      if (nfn[t] > INT32_MAX) {
        free(srcs);
        status = ORACLE_EUNSUPPORTED;
        break;
      }
      nf[t] = (int64_t *)malloc(sizeof(int64_t) * (size_t)(nfn[t] + 1));
      if (!nf[t]) {
        free(srcs);
        status = ORACLE_ENOMEM;
        break;
      }
      if (fn[t] > 0) memcpy(nf[t], fr[t], sizeof(int64_t) * (size_t)fn[t]);
      if (u > 0) memcpy(nf[t] + fn[t], srcs, sizeof(int64_t) * (size_t)u);
      free(srcs);
    }

    /* ---- Step 3: compaction -- relabel every sampled edge's source with
     * its position in the source list of its type; the destination already
     * carries its frontier position. */
    for (int32_t e = 0; e < n_etypes && status == ORACLE_OK; ++e) {
      int32_t s = etypes[e].src_type;
      oedges *blk = &b->edges[(int64_t)h * n_etypes + e];
      int64_t n = n_sampled[e];
      blk->n_edges = n;
      blk->src_local = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n + 1));
      blk->dst_local = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n + 1));
      blk->eid = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n + 1));
      if (!blk->src_local || !blk->dst_local || !blk->eid) {
        status = ORACLE_ENOMEM;
        break;
      }
#pragma omp parallel for schedule(static)
      for (int64_t j = 0; j < n; ++j) {
        int64_t g = sampled[e][j].src_gid;
        int64_t pos = find_gid_pos(ftab[s], fn[s], g);
        if (pos < 0) pos = fn[s] + find_sorted(nf[s] + fn[s], n_new[s], g);
        blk->src_local[j] = (int32_t)pos;
        blk->dst_local[j] = sampled[e][j].dst_local;
        blk->eid[j] = sampled[e][j].eid;
      }
    }

    /* record the hop's vertex lists; the next hop starts from them */
    for (int32_t t = 0; t < n_ntypes && status == ORACLE_OK; ++t) {
      onodes *nd = &b->nodes[(int64_t)h * n_ntypes + t];
      nd->n_dst = fn[t];
      nd->n_src = nfn[t];
      nd->src_gid = nf[t];
      nf[t] = NULL;
      free(fr[t]);
      fr[t] = (int64_t *)malloc(sizeof(int64_t) * (size_t)(nfn[t] + 1));
      if (!fr[t]) {
        status = ORACLE_ENOMEM;
        break;
      }
      if (nfn[t] > 0)
        memcpy(fr[t], nd->src_gid, sizeof(int64_t) * (size_t)nfn[t]);
      fn[t] = nfn[t];
    }

    for (int32_t e = 0; e < n_etypes; ++e) free(sampled[e]);
    free(sampled);
    free(n_sampled);
    if (nf)
      for (int32_t t = 0; t < n_ntypes; ++t) free(nf[t]);
    if (ftab)
      for (int32_t t = 0; t < n_ntypes; ++t) free(ftab[t]);
    free(nf);
    free(nfn);
    free(ftab);
    free(n_new);
  }

  /* the input frontier: what the feature gather reads */
  for (int32_t t = 0; t < n_ntypes && status == ORACLE_OK; ++t) {
    b->in_n[t] = fn[t];
    b->in_gid[t] = fr[t];
    fr[t] = NULL;
  }
  for (int32_t t = 0; t < n_ntypes; ++t) free(fr[t]);
  (void)ntypes;
  return status;
}

/* A blocks container for n_hops hops (everything zeroed). */
static oracle_blocks *new_blocks(int32_t n_hops, int32_t n_ntypes, int32_t n_etypes) {
  oracle_blocks *b = (oracle_blocks *)calloc(1, sizeof(oracle_blocks));
  if (!b) return NULL;
  b->n_hops = n_hops;
  b->n_ntypes = n_ntypes;
  b->n_etypes = n_etypes;
  b->nodes = (onodes *)calloc((size_t)n_hops * n_ntypes + 1, sizeof(onodes));
  b->edges = (oedges *)calloc((size_t)n_hops * n_etypes + 1, sizeof(oedges));
  b->in_n = (int64_t *)calloc((size_t)n_ntypes, sizeof(int64_t));
  b->in_gid = (int64_t **)calloc((size_t)n_ntypes, sizeof(int64_t *));
  if (!b->nodes || !b->edges || !b->in_n || !b->in_gid) {
    oracle_blocks_free(b);
    return NULL;
  }
  return b;
}

/* Shared argument checks of both kinds of mini-batch. */
static int check_common(const oracle_ntype *ntypes, int32_t n_ntypes,
                        const oracle_etype *etypes, int32_t n_etypes, int32_t n_hops,
                        const int32_t *fanouts, int32_t key_bits) {
  if (n_ntypes < 1 || n_etypes < 0 || !ntypes || (n_etypes > 0 && !etypes))
    return ORACLE_EINVAL;
  if (n_hops < 0 || key_bits < 1 || key_bits > 32) return ORACLE_EINVAL;
  if (n_hops > 0 && n_etypes > 0 && !fanouts) return ORACLE_EINVAL;
  for (int64_t i = 0; i < (int64_t)n_hops * n_etypes; ++i)
    if (fanouts[i] < -1) return ORACLE_EINVAL;
  for (int32_t e = 0; e < n_etypes; ++e)
    if (etypes[e].src_type < 0 || etypes[e].src_type >= n_ntypes ||
        etypes[e].dst_type < 0 || etypes[e].dst_type >= n_ntypes)
      return ORACLE_EINVAL;
  return ORACLE_OK;
}

/* Seeds: present, in range and unique within their type (the targets of a
 * mini-batch are a set of vertices, Sec. 3.2). */
static int check_seeds(const oracle_ntype *ntypes, int32_t n_ntypes,
                       const int64_t *const *seeds, const int64_t *n_seeds) {
  for (int32_t t = 0; t < n_ntypes; ++t) {
    if (n_seeds[t] < 0) return ORACLE_EINVAL;
    if (n_seeds[t] == 0) continue;
    if (!seeds || !seeds[t]) return ORACLE_EINVAL;
    int64_t *tmp = (int64_t *)malloc(sizeof(int64_t) * (size_t)n_seeds[t]);
    if (!tmp) return ORACLE_ENOMEM;
    memcpy(tmp, seeds[t], sizeof(int64_t) * (size_t)n_seeds[t]);
    qsort(tmp, (size_t)n_seeds[t], sizeof(int64_t), cmp_i64);
    int bad = 0;
    for (int64_t i = 0; i < n_seeds[t]; ++i) {
      if (tmp[i] < 0 || tmp[i] >= ntypes[t].num_nodes) bad = 1;
      if (i > 0 && tmp[i] == tmp[i - 1]) bad = 1;
    }
    free(tmp);
    if (bad) return ORACLE_EINVAL;
  }
  return ORACLE_OK;
}

int oracle_sample_blocks(const oracle_ntype *ntypes, int32_t n_ntypes,
                         const oracle_etype *etypes, int32_t n_etypes,
                         const int64_t *const *seeds, const int64_t *n_seeds,
                         int32_t n_hops, const int32_t *fanouts, uint64_t sigma,
                         int32_t key_bits, oracle_blocks **out) {
  if (!out) return ORACLE_EINVAL;
  *out = NULL;
  int status = check_common(ntypes, n_ntypes, etypes, n_etypes, n_hops, fanouts, key_bits);
  if (status != ORACLE_OK) return status;
  if (!n_seeds) return ORACLE_EINVAL;

  status = check_seeds(ntypes, n_ntypes, seeds, n_seeds);
  if (status != ORACLE_OK) return status;

  oracle_blocks *b = new_blocks(n_hops, n_ntypes, n_etypes);
  if (!b) return ORACLE_ENOMEM;
  /* frontier of the current hop, per node type: F[0][t] = seeds of t */
  int64_t *fn = (int64_t *)calloc((size_t)n_ntypes, sizeof(int64_t));
  int64_t **fr = (int64_t **)calloc((size_t)n_ntypes, sizeof(int64_t *));
  excl_list *none = (excl_list *)calloc((size_t)n_etypes + 1, sizeof(excl_list));
  if (!fn || !fr || !none) status = ORACLE_ENOMEM;
  for (int32_t t = 0; t < n_ntypes && status == ORACLE_OK; ++t) {
    fn[t] = n_seeds[t];
    fr[t] = (int64_t *)malloc(sizeof(int64_t) * (size_t)(fn[t] + 1));
    if (!fr[t]) {
      status = ORACLE_ENOMEM;
      break;
    }
    if (fn[t] > 0) memcpy(fr[t], seeds[t], sizeof(int64_t) * (size_t)fn[t]);
  }
  if (status == ORACLE_OK)
    status = run_hops(ntypes, n_ntypes, etypes, n_etypes, fr, fn, n_hops, fanouts, sigma,
                      key_bits, none, b);
  else if (fr)
    for (int32_t t = 0; t < n_ntypes; ++t) free(fr[t]);
  free(fr);
  free(fn);
  free(none);
  if (status != ORACLE_OK) {
    oracle_blocks_free(b);
    return status;
  }
  *out = b;
  return ORACLE_OK;
}

int oracle_blocks_nodes(const oracle_blocks *b, int32_t hop, int32_t ntype,
                        int64_t *n_dst, int64_t *n_src,
                        const int64_t **src_gid) {
  if (!b || hop < 0 || hop >= b->n_hops || ntype < 0 || ntype >= b->n_ntypes)
    return ORACLE_EINVAL;
  const onodes *nd = &b->nodes[(int64_t)hop * b->n_ntypes + ntype];
  if (n_dst) *n_dst = nd->n_dst;
  if (n_src) *n_src = nd->n_src;
  if (src_gid) *src_gid = nd->src_gid;
  return ORACLE_OK;
}

int oracle_blocks_edges(const oracle_blocks *b, int32_t hop, int32_t etype,
                        int64_t *n_edges, const int64_t **indptr,
                        const int32_t **src_local, const int32_t **dst_local,
                        const int64_t **eid) {
  if (!b || hop < 0 || hop >= b->n_hops || etype < 0 || etype >= b->n_etypes)
    return ORACLE_EINVAL;
  const oedges *ed = &b->edges[(int64_t)hop * b->n_etypes + etype];
  if (n_edges) *n_edges = ed->n_edges;
  if (indptr) *indptr = ed->indptr;
  if (src_local) *src_local = ed->src_local;
  if (dst_local) *dst_local = ed->dst_local;
  if (eid) *eid = ed->eid;
  return ORACLE_OK;
}

int oracle_blocks_input_nodes(const oracle_blocks *b, int32_t ntype,
                              int64_t *n, const int64_t **gid) {
  if (!b || ntype < 0 || ntype >= b->n_ntypes) return ORACLE_EINVAL;
  if (n) *n = b->in_n[ntype];
  if (gid) *gid = b->in_gid[ntype];
  return ORACLE_OK;
}

int oracle_gather_rows(const void *feat, int64_t n_rows, int64_t row_bytes,
                       const int64_t *ids, int64_t n, void *out) {
  if (n < 0 || row_bytes <= 0 || (n > 0 && (!feat || !ids || !out)))
    return ORACLE_EINVAL;
  for (int64_t i = 0; i < n; ++i)
    if (ids[i] < 0 || ids[i] >= n_rows) return ORACLE_EINVAL;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i)
    memcpy((char *)out + i * row_bytes,
           (const char *)feat + ids[i] * row_bytes, (size_t)row_bytes);
  return ORACLE_OK;
}

int oracle_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* ------------------------------------------------------------------ */
/* Edge-seeded mini-batches (link prediction).  The scheduler of Sec. 4.2.1
 * picks target edges instead of target vertices; the same neighbour
 * sampling, compaction and feature gather then run from the targets'
 * endpoints (Sec. 4.2.2 notes that the decomposition carries over to link
 * prediction).  Readings where the paper is silent:
 *  - a target is an edge ID (CSC slot) of an edge type; targets may repeat;
 *  - its endpoints are indices[eid] (source) and the destination whose
 *    in-edge slots hold eid;
 *  - optional negatives: n_neg per target, same source, destination drawn
 *    uniformly from the destination type by Philox4x32-10 (see
 *    oracle_negative_dst);
 *  - seeds of a node type: every endpoint and negative destination of that
 *    type, each once, in ascending ID;
 *  - exclusion 1 takes the target edges out of every hop's sampling;
 *    exclusion 2 also takes out each target's reverse edge, named by a
 *    caller-given map into a reverse edge type.                         */

int oracle_edge_dst(const int64_t *indptr, int64_t n_dst, int64_t eid, int64_t *dst) {
  if (!indptr || !dst || n_dst < 1 || eid < 0 || eid >= indptr[n_dst]) return ORACLE_EINVAL;
  /* the destination v with indptr[v] <= eid < indptr[v+1]: the largest v
   * whose first slot is not above eid */
  int64_t a = 0, b = n_dst - 1;
  while (a < b) {
    int64_t m = a + (b - a + 1) / 2;
    if (indptr[m] <= eid)
      a = m;
    else
      b = m - 1;
  }
  *dst = a;
  return ORACLE_OK;
}

int oracle_negative_dst(uint64_t sigma, int32_t etype, int64_t eid, int32_t k,
                        int64_t n_dst, int64_t *v) {
  if (!v || k < 0 || n_dst < 1) return ORACLE_EINVAL;
  /* counter (eid lo32, eid hi32, 2^31 | k, etype): the third word never has
   * its top bit set for a sampling key (a hop number), so the two streams
   * never share a counter */
  uint32_t ctr[4] = {(uint32_t)eid, (uint32_t)((uint64_t)eid >> 32), 0x80000000u | (uint32_t)k,
                     (uint32_t)etype};
  uint32_t seed_words[2] = {(uint32_t)sigma, (uint32_t)(sigma >> 32)};
  uint32_t out[4];
  oracle_philox4x32_10(ctr, seed_words, out);
  /* u uniform on [0, 2^64); v = floor(u * n / 2^64) is uniform on [0, n)
   * up to n / 2^64 */
  uint64_t u = (uint64_t)out[0] | ((uint64_t)out[1] << 32);
  *v = (int64_t)(((unsigned __int128)u * (unsigned __int128)(uint64_t)n_dst) >> 64);
  return ORACLE_OK;
}

/* ascending, duplicates removed; returns the new length */
static int64_t sort_unique(int64_t *a, int64_t n) {
  if (n == 0) return 0;
  qsort(a, (size_t)n, sizeof(int64_t), cmp_i64);
  int64_t u = 1;
  for (int64_t i = 1; i < n; ++i)
    if (a[i] != a[u - 1]) a[u++] = a[i];
  return u;
}

int oracle_sample_edge_blocks(const oracle_ntype *ntypes, int32_t n_ntypes,
                              const oracle_etype *etypes, int32_t n_etypes,
                              const oracle_edge_batch *batch, int32_t n_hops,
                              const int32_t *fanouts, uint64_t sigma, int32_t key_bits,
                              oracle_blocks **out) {
  if (!out) return ORACLE_EINVAL;
  *out = NULL;
  int status = check_common(ntypes, n_ntypes, etypes, n_etypes, n_hops, fanouts, key_bits);
  if (status != ORACLE_OK) return status;
  if (!batch || !batch->n_eids || batch->n_neg < 0 || batch->n_neg > ORACLE_MAX_NEG ||
      batch->exclude < 0 || batch->exclude > 2)
    return ORACLE_EINVAL;
  if (batch->exclude == 2 && (!batch->rev_etype || !batch->rev_eid)) return ORACLE_EINVAL;
  const int32_t R = n_etypes, T = n_ntypes, Q = batch->n_neg;

  /* every target: in range; with exclusion 2 its reverse must be an edge of
   * the reverse type that runs the other way */
  for (int32_t e = 0; e < R; ++e) {
    const int64_t n = batch->n_eids[e];
    if (n < 0 || (n > 0 && (!batch->eids || !batch->eids[e]))) return ORACLE_EINVAL;
    const oracle_etype *et = &etypes[e];
    const int64_t n_dst = ntypes[et->dst_type].num_nodes;
    for (int64_t i = 0; i < n; ++i) {
      const int64_t j = batch->eids[e][i];
      if (j < 0 || j >= et->nnz) return ORACLE_EINVAL;
    }
    if (batch->exclude != 2 || n == 0) continue;
    const int32_t r = batch->rev_etype[e];
    if (r < 0) continue;
    if (r >= R || etypes[r].src_type != et->dst_type || etypes[r].dst_type != et->src_type ||
        !batch->rev_eid[e])
      return ORACLE_EINVAL;
    const int64_t rn_dst = ntypes[etypes[r].dst_type].num_nodes;
    for (int64_t i = 0; i < n; ++i) {
      const int64_t j = batch->eids[e][i];
      const int64_t rj = batch->rev_eid[e][j];
      int64_t v, rv;
      if (rj < 0 || rj >= etypes[r].nnz) return ORACLE_EINVAL;
      if (oracle_edge_dst(et->indptr, n_dst, j, &v) != ORACLE_OK ||
          oracle_edge_dst(etypes[r].indptr, rn_dst, rj, &rv) != ORACLE_OK)
        return ORACLE_EINVAL;
      if (etypes[r].indices[rj] != v || rv != et->indices[j]) return ORACLE_EINVAL;
    }
  }

  oracle_blocks *b = new_blocks(n_hops, n_ntypes, n_etypes);
  if (!b) return ORACLE_ENOMEM;
  b->n_neg = Q;
  b->seed_n = (int64_t *)calloc((size_t)T, sizeof(int64_t));
  b->seed_gid = (int64_t **)calloc((size_t)T, sizeof(int64_t *));
  b->pair_n = (int64_t *)calloc((size_t)R + 1, sizeof(int64_t));
  b->pos_src = (int32_t **)calloc((size_t)R + 1, sizeof(int32_t *));
  b->pos_dst = (int32_t **)calloc((size_t)R + 1, sizeof(int32_t *));
  b->neg_dst = (int32_t **)calloc((size_t)R + 1, sizeof(int32_t *));
  /* per etype: endpoint IDs of every target, negative destinations */
  int64_t **src = (int64_t **)calloc((size_t)R + 1, sizeof(int64_t *));
  int64_t **dst = (int64_t **)calloc((size_t)R + 1, sizeof(int64_t *));
  int64_t **neg = (int64_t **)calloc((size_t)R + 1, sizeof(int64_t *));
  excl_list *excl = (excl_list *)calloc((size_t)R + 1, sizeof(excl_list));
  int64_t *fn = (int64_t *)calloc((size_t)T, sizeof(int64_t));
  int64_t **fr = (int64_t **)calloc((size_t)T, sizeof(int64_t *));
  if (!b->seed_n || !b->seed_gid || !b->pair_n || !b->pos_src || !b->pos_dst ||
      !b->neg_dst || !src || !dst || !neg || !excl || !fn || !fr)
    status = ORACLE_ENOMEM;

  /* 1. endpoints and negatives */
  for (int32_t e = 0; e < R && status == ORACLE_OK; ++e) {
    const oracle_etype *et = &etypes[e];
    const int64_t n = batch->n_eids[e];
    const int64_t n_dst = ntypes[et->dst_type].num_nodes;
    src[e] = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n + 1));
    dst[e] = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n + 1));
    neg[e] = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n * Q + 1));
    if (!src[e] || !dst[e] || !neg[e]) {
      status = ORACLE_ENOMEM;
      break;
    }
    for (int64_t i = 0; i < n && status == ORACLE_OK; ++i) {
      const int64_t j = batch->eids[e][i];
      src[e][i] = et->indices[j];
      status = oracle_edge_dst(et->indptr, n_dst, j, &dst[e][i]);
      for (int32_t k = 0; k < Q && status == ORACLE_OK; ++k)
        status = oracle_negative_dst(sigma, e, j, k, n_dst, &neg[e][i * Q + k]);
    }
  }

  /* 2. seeds per node type: the endpoints of that type, once each, ascending */
  for (int32_t t = 0; t < T && status == ORACLE_OK; ++t) {
    int64_t cap = 0;
    for (int32_t e = 0; e < R; ++e) {
      if (etypes[e].src_type == t) cap += batch->n_eids[e];
      if (etypes[e].dst_type == t) cap += batch->n_eids[e] * (1 + Q);
    }
    int64_t *all = (int64_t *)malloc(sizeof(int64_t) * (size_t)(cap + 1));
    if (!all) {
      status = ORACLE_ENOMEM;
      break;
    }
    int64_t m = 0;
    for (int32_t e = 0; e < R; ++e) {
      const int64_t n = batch->n_eids[e];
      if (etypes[e].src_type == t)
        for (int64_t i = 0; i < n; ++i) all[m++] = src[e][i];
      if (etypes[e].dst_type == t) {
        for (int64_t i = 0; i < n; ++i) all[m++] = dst[e][i];
        for (int64_t i = 0; i < n * Q; ++i) all[m++] = neg[e][i];
      }
    }
    b->seed_n[t] = sort_unique(all, m);
    b->seed_gid[t] = all;
  }

  /* 3. the pair graphs: local IDs (positions among the seeds) */
  for (int32_t e = 0; e < R && status == ORACLE_OK; ++e) {
    const int32_t s = etypes[e].src_type, d = etypes[e].dst_type;
    const int64_t n = batch->n_eids[e];
    b->pair_n[e] = n;
    b->pos_src[e] = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n + 1));
    b->pos_dst[e] = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n + 1));
    b->neg_dst[e] = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n * Q + 1));
    if (!b->pos_src[e] || !b->pos_dst[e] || !b->neg_dst[e]) {
      status = ORACLE_ENOMEM;
      break;
    }
    for (int64_t i = 0; i < n; ++i) {
      b->pos_src[e][i] = (int32_t)find_sorted(b->seed_gid[s], b->seed_n[s], src[e][i]);
      b->pos_dst[e][i] = (int32_t)find_sorted(b->seed_gid[d], b->seed_n[d], dst[e][i]);
    }
    for (int64_t i = 0; i < n * Q; ++i)
      b->neg_dst[e][i] = (int32_t)find_sorted(b->seed_gid[d], b->seed_n[d], neg[e][i]);
  }

  /* 4. the excluded edges, per edge type, ascending and unique */
  if (batch->exclude >= 1 && status == ORACLE_OK) {
    for (int32_t e = 0; e < R && status == ORACLE_OK; ++e) {
      int64_t cap = batch->n_eids[e];
      if (batch->exclude == 2)
        for (int32_t f = 0; f < R; ++f)
          if (batch->rev_etype[f] == e) cap += batch->n_eids[f];
      excl[e].eids = (int64_t *)malloc(sizeof(int64_t) * (size_t)(cap + 1));
      if (!excl[e].eids) {
        status = ORACLE_ENOMEM;
        break;
      }
      int64_t m = 0;
      for (int64_t i = 0; i < batch->n_eids[e]; ++i) excl[e].eids[m++] = batch->eids[e][i];
      if (batch->exclude == 2)
        for (int32_t f = 0; f < R; ++f)
          if (batch->rev_etype[f] == e)
            for (int64_t i = 0; i < batch->n_eids[f]; ++i)
              excl[e].eids[m++] = batch->rev_eid[f][batch->eids[f][i]];
      excl[e].n = sort_unique(excl[e].eids, m);
    }
  }

  /* 5. the hops, from the seeds */
  for (int32_t t = 0; t < T && status == ORACLE_OK; ++t) {
    fn[t] = b->seed_n[t];
    fr[t] = (int64_t *)malloc(sizeof(int64_t) * (size_t)(fn[t] + 1));
    if (!fr[t]) {
      status = ORACLE_ENOMEM;
      break;
    }
    if (fn[t] > 0) memcpy(fr[t], b->seed_gid[t], sizeof(int64_t) * (size_t)fn[t]);
  }
  if (status == ORACLE_OK)
    status = run_hops(ntypes, n_ntypes, etypes, n_etypes, fr, fn, n_hops, fanouts, sigma,
                      key_bits, excl, b);
  else if (fr)
    for (int32_t t = 0; t < T; ++t) free(fr[t]);

  for (int32_t e = 0; e < R; ++e) {
    if (src) free(src[e]);
    if (dst) free(dst[e]);
    if (neg) free(neg[e]);
    if (excl) free(excl[e].eids);
  }
  free(src);
  free(dst);
  free(neg);
  free(excl);
  free(fr);
  free(fn);
  if (status != ORACLE_OK) {
    oracle_blocks_free(b);
    return status;
  }
  *out = b;
  return ORACLE_OK;
}

int oracle_blocks_seeds(const oracle_blocks *b, int32_t ntype, int64_t *n,
                        const int64_t **gid) {
  if (!b || !b->seed_n || ntype < 0 || ntype >= b->n_ntypes) return ORACLE_EINVAL;
  if (n) *n = b->seed_n[ntype];
  if (gid) *gid = b->seed_gid[ntype];
  return ORACLE_OK;
}

int oracle_blocks_pairs(const oracle_blocks *b, int32_t etype, int64_t *n_pos,
                        const int32_t **pos_src, const int32_t **pos_dst,
                        int64_t *n_negs, const int32_t **neg_dst) {
  if (!b || !b->pair_n || etype < 0 || etype >= b->n_etypes) return ORACLE_EINVAL;
  if (n_pos) *n_pos = b->pair_n[etype];
  if (pos_src) *pos_src = b->pos_src[etype];
  if (pos_dst) *pos_dst = b->pos_dst[etype];
  if (n_negs) *n_negs = b->pair_n[etype] * b->n_neg;
  if (neg_dst) *neg_dst = b->neg_dst[etype];
  return ORACLE_OK;
}

/* ------------------------------------------------------------------ */
/* Layer-wise sampling (LADIES; Sec. 4.2.2 names it as fitting the same
 * decomposition; the algorithm is Zou et al., NeurIPS 2019, Algorithm 1).
 * Instead of K neighbours per vertex, each hop draws a fixed number of
 * vertices per node type for the whole layer, with probability proportional
 * to their layer-dependent importance, and keeps every edge from the drawn
 * vertices (and the frontier) into the frontier.  Readings where the papers
 * leave room (listed in the design notes):
 *  - candidates of type t: the in-neighbours of the frontier over every edge
 *    type whose source type is t, minus the frontier itself;
 *  - importance: LADIES' column norm of the row-normalised adjacency,
 *    sum over the candidate's edges u -> v into the frontier of 1 / deg_e(v)^2,
 *    kept in fixed point as floor(2^32 / deg_e(v)^2) so that sums are exact;
 *  - n[h][t] i.i.d. draws with replacement (LADIES Algorithm 1): draw k takes
 *    r = floor(x * total / 2^64), x = word0 | word1 << 32 of Philox4x32-10 at
 *    counter (k lo32, k hi32, 2^30 | h, t) under key sigma, and picks the
 *    candidate whose interval [prefix, prefix + weight) holds r, candidates in
 *    ascending ID; n = -1 takes every candidate, 0 none;
 *  - the next frontier is the frontier followed by the distinct drawn
 *    vertices in ascending ID; the block of the hop keeps every in-edge of a
 *    frontier vertex whose source is in the next frontier.               */

uint64_t oracle_layer_weight(int64_t deg) {
  if (deg <= 0) return 0;
  const unsigned __int128 d2 = (unsigned __int128)(uint64_t)deg * (uint64_t)deg;
  return (uint64_t)(((unsigned __int128)1 << 32) / d2);
}

uint64_t oracle_layer_draw(uint64_t sigma, int32_t hop, int32_t ntype, int64_t k,
                           uint64_t total) {
  uint32_t ctr[4] = {(uint32_t)k, (uint32_t)((uint64_t)k >> 32), 0x40000000u | (uint32_t)hop,
                     (uint32_t)ntype};
  uint32_t seed_words[2] = {(uint32_t)sigma, (uint32_t)(sigma >> 32)};
  uint32_t out[4];
  oracle_philox4x32_10(ctr, seed_words, out);
  uint64_t x = (uint64_t)out[0] | ((uint64_t)out[1] << 32);
  return (uint64_t)(((unsigned __int128)x * total) >> 64);
}

int oracle_sample_layers(const oracle_ntype *ntypes, int32_t n_ntypes,
                         const oracle_etype *etypes, int32_t n_etypes,
                         const int64_t *const *seeds, const int64_t *n_seeds, int32_t n_hops,
                         const int32_t *layer_sizes, uint64_t sigma, oracle_blocks **out) {
  if (!out) return ORACLE_EINVAL;
  *out = NULL;
  if (n_ntypes < 1 || n_etypes < 0 || !ntypes || (n_etypes > 0 && !etypes) || n_hops < 0 ||
      !n_seeds || (n_hops > 0 && !layer_sizes))
    return ORACLE_EINVAL;
  for (int64_t i = 0; i < (int64_t)n_hops * n_ntypes; ++i)
    if (layer_sizes[i] < -1) return ORACLE_EINVAL;
  for (int32_t e = 0; e < n_etypes; ++e)
    if (etypes[e].src_type < 0 || etypes[e].src_type >= n_ntypes || etypes[e].dst_type < 0 ||
        etypes[e].dst_type >= n_ntypes)
      return ORACLE_EINVAL;
  int status = check_seeds(ntypes, n_ntypes, seeds, n_seeds);
  if (status != ORACLE_OK) return status;
  const int32_t T = n_ntypes, R = n_etypes;
  oracle_blocks *b = new_blocks(n_hops, T, R);
  if (!b) return ORACLE_ENOMEM;
  int64_t *fn = (int64_t *)calloc((size_t)T, sizeof(int64_t));
  int64_t **fr = (int64_t **)calloc((size_t)T, sizeof(int64_t *));
  /* per type: importance of every vertex, and membership of the frontier and
   * of the candidate set (dense arrays over the type's vertices) */
  uint64_t **wt = (uint64_t **)calloc((size_t)T, sizeof(uint64_t *));
  char **in_f = (char **)calloc((size_t)T, sizeof(char *));
  char **is_c = (char **)calloc((size_t)T, sizeof(char *));
  if (!fn || !fr || !wt || !in_f || !is_c) status = ORACLE_ENOMEM;
  for (int32_t t = 0; t < T && status == ORACLE_OK; ++t) {
    const int64_t n = ntypes[t].num_nodes;
    fn[t] = n_seeds[t];
    fr[t] = (int64_t *)malloc(sizeof(int64_t) * (size_t)(fn[t] + 1));
    wt[t] = (uint64_t *)calloc((size_t)n + 1, sizeof(uint64_t));
    in_f[t] = (char *)calloc((size_t)n + 1, 1);
    is_c[t] = (char *)calloc((size_t)n + 1, 1);
    if (!fr[t] || !wt[t] || !in_f[t] || !is_c[t]) {
      status = ORACLE_ENOMEM;
      break;
    }
    if (fn[t] > 0) memcpy(fr[t], seeds[t], sizeof(int64_t) * (size_t)fn[t]);
  }

  for (int32_t h = 0; h < n_hops && status == ORACLE_OK; ++h) {
    /* ---- the frontier, as a membership array */
    for (int32_t t = 0; t < T; ++t)
      for (int64_t i = 0; i < fn[t]; ++i) in_f[t][fr[t][i]] = 1;
    /* ---- importance of every candidate: its edges into the frontier */
    for (int32_t e = 0; e < R; ++e) {
      const oracle_etype *et = &etypes[e];
      const int32_t s = et->src_type, d = et->dst_type;
      for (int64_t i = 0; i < fn[d]; ++i) {
        const int64_t v = fr[d][i];
        const int64_t lo = et->indptr[v], hi = et->indptr[v + 1];
        const uint64_t w = oracle_layer_weight(hi - lo);
        for (int64_t j = lo; j < hi; ++j) {
          const int64_t u = et->indices[j];
          if (in_f[s][u]) continue;
          is_c[s][u] = 1;
          wt[s][u] += w;
        }
      }
    }
    /* ---- draws per node type; the next frontier */
    int64_t **nf = (int64_t **)calloc((size_t)T, sizeof(int64_t *));
    int64_t *nfn = (int64_t *)calloc((size_t)T, sizeof(int64_t));
    if (!nf || !nfn) status = ORACLE_ENOMEM;
    for (int32_t t = 0; t < T && status == ORACLE_OK; ++t) {
      const int64_t n = ntypes[t].num_nodes;
      const int32_t k = layer_sizes[(int64_t)h * T + t];
      /* candidates in ascending ID, their weight prefix */
      int64_t nc = 0;
      for (int64_t u = 0; u < n; ++u) nc += is_c[t][u];
      int64_t *cand = (int64_t *)malloc(sizeof(int64_t) * (size_t)(nc + 1));
      uint64_t *pre = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)(nc + 1));
      char *drawn = (char *)calloc((size_t)nc + 1, 1);
      if (!cand || !pre || !drawn) {
        free(cand);
        free(pre);
        free(drawn);
        status = ORACLE_ENOMEM;
        break;
      }
      int64_t m = 0;
      uint64_t total = 0;
      for (int64_t u = 0; u < n; ++u)
        if (is_c[t][u]) {
          cand[m] = u;
          pre[m] = total;
          total += wt[t][u];
          ++m;
        }
      if (k < 0) {
        for (int64_t i = 0; i < nc; ++i) drawn[i] = 1;
      } else if (total > 0) {
        for (int64_t q = 0; q < k; ++q) {
          const uint64_t r = oracle_layer_draw(sigma, h, t, q, total);
          /* the candidate whose interval holds r: the last one whose prefix
           * is not above r (zero-weight candidates have empty intervals) */
          int64_t a = 0, z = nc - 1;
          while (a < z) {
            int64_t mid = a + (z - a + 1) / 2;
            if (pre[mid] <= r)
              a = mid;
            else
              z = mid - 1;
          }
          drawn[a] = 1;
        }
      }
      int64_t nd = 0;
      for (int64_t i = 0; i < nc; ++i) nd += drawn[i];
      nfn[t] = fn[t] + nd;
      if (nfn[t] > INT32_MAX) status = ORACLE_EUNSUPPORTED;
      nf[t] = (int64_t *)malloc(sizeof(int64_t) * (size_t)(nfn[t] + 1));
      if (!nf[t] && status == ORACLE_OK) status = ORACLE_ENOMEM;
      if (status == ORACLE_OK) {
        if (fn[t] > 0) memcpy(nf[t], fr[t], sizeof(int64_t) * (size_t)fn[t]);
        int64_t p = fn[t];
        for (int64_t i = 0; i < nc; ++i)
          if (drawn[i]) nf[t][p++] = cand[i];
      }
      /* clean the dense arrays for the next hop */
      for (int64_t i = 0; i < nc; ++i) {
        is_c[t][cand[i]] = 0;
        wt[t][cand[i]] = 0;
      }
      free(cand);
      free(pre);
      free(drawn);
    }
    for (int32_t t = 0; t < T; ++t)
      for (int64_t i = 0; i < fn[t]; ++i) in_f[t][fr[t][i]] = 0;

    /* ---- the block: every in-edge of the frontier from the next frontier;
     * local IDs by lookup in the next frontier */
    gid_pos **ntab = (gid_pos **)calloc((size_t)T, sizeof(gid_pos *));
    if (!ntab && status == ORACLE_OK) status = ORACLE_ENOMEM;
    for (int32_t t = 0; t < T && status == ORACLE_OK; ++t) {
      ntab[t] = (gid_pos *)malloc(sizeof(gid_pos) * (size_t)(nfn[t] + 1));
      if (!ntab[t]) {
        status = ORACLE_ENOMEM;
        break;
      }
      for (int64_t i = 0; i < nfn[t]; ++i) {
        ntab[t][i].gid = nf[t][i];
        ntab[t][i].pos = i;
      }
      qsort(ntab[t], (size_t)nfn[t], sizeof(gid_pos), cmp_gid_pos);
    }
    for (int32_t e = 0; e < R && status == ORACLE_OK; ++e) {
      const oracle_etype *et = &etypes[e];
      const int32_t s = et->src_type, d = et->dst_type;
      oedges *blk = &b->edges[(int64_t)h * R + e];
      int64_t cap = 0;
      for (int64_t i = 0; i < fn[d]; ++i) cap += et->indptr[fr[d][i] + 1] - et->indptr[fr[d][i]];
      blk->indptr = (int64_t *)malloc(sizeof(int64_t) * (size_t)(fn[d] + 1));
      blk->src_local = (int32_t *)malloc(sizeof(int32_t) * (size_t)(cap + 1));
      blk->dst_local = (int32_t *)malloc(sizeof(int32_t) * (size_t)(cap + 1));
      blk->eid = (int64_t *)malloc(sizeof(int64_t) * (size_t)(cap + 1));
      if (!blk->indptr || !blk->src_local || !blk->dst_local || !blk->eid) {
        status = ORACLE_ENOMEM;
        break;
      }
      int64_t cnt = 0;
      blk->indptr[0] = 0;
      for (int64_t i = 0; i < fn[d]; ++i) {
        const int64_t v = fr[d][i];
        for (int64_t j = et->indptr[v]; j < et->indptr[v + 1]; ++j) {
          const int64_t pos = find_gid_pos(ntab[s], nfn[s], et->indices[j]);
          if (pos < 0) continue;
          blk->src_local[cnt] = (int32_t)pos;
          blk->dst_local[cnt] = (int32_t)i;
          blk->eid[cnt] = j;
          ++cnt;
        }
        blk->indptr[i + 1] = cnt;
      }
      blk->n_edges = cnt;
    }
    /* record the hop's vertex lists; the next hop starts from them */
    for (int32_t t = 0; t < T && status == ORACLE_OK; ++t) {
      onodes *nd = &b->nodes[(int64_t)h * T + t];
      nd->n_dst = fn[t];
      nd->n_src = nfn[t];
      nd->src_gid = nf[t];
      nf[t] = NULL;
      free(fr[t]);
      fr[t] = (int64_t *)malloc(sizeof(int64_t) * (size_t)(nfn[t] + 1));
      if (!fr[t]) {
        status = ORACLE_ENOMEM;
        break;
      }
      if (nfn[t] > 0) memcpy(fr[t], nd->src_gid, sizeof(int64_t) * (size_t)nfn[t]);
      fn[t] = nfn[t];
    }
    if (ntab)
      for (int32_t t = 0; t < T; ++t) free(ntab[t]);
    free(ntab);
    if (nf)
      for (int32_t t = 0; t < T; ++t) free(nf[t]);
    free(nf);
    free(nfn);
  }
  for (int32_t t = 0; t < T && status == ORACLE_OK; ++t) {
    b->in_n[t] = fn[t];
    b->in_gid[t] = fr[t];
    fr[t] = NULL;
  }
  for (int32_t t = 0; t < T; ++t) {
    if (fr) free(fr[t]);
    if (wt) free(wt[t]);
    if (in_f) free(in_f[t]);
    if (is_c) free(is_c[t]);
  }
  free(fr);
  free(fn);
  free(wt);
  free(in_f);
  free(is_c);
  if (status != ORACLE_OK) {
    oracle_blocks_free(b);
    return status;
  }
  *out = b;
  return ORACLE_OK;
}
