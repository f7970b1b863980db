/*
 * Test driver for the oracle under the host sanitizers (AddressSanitizer and
 * UndefinedBehaviorSanitizer): runs every entry point of oracle.h on seeded
 * random heterographs -- vertex-seeded, edge-seeded (no exclusion and
 * exclusion of the targets, 0-2 negatives) and layer-wise mini-batches, the
 * gather, and the argument errors -- and reads back every output array.  Built by
 * tests/test_oracle_sanitize.py with gcc; a sanitizer report or a wrong status
 * fails the run.  Exit status 0 means every call behaved.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "oracle.h"

static uint64_t rng_state = 0x243F6A8885A308D3ull;
static uint64_t next_u64(void) { /* splitmix64 */
  uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
static int64_t below(int64_t n) { return n > 0 ? (int64_t)(next_u64() % (uint64_t)n) : 0; }

static int failures = 0;
#define EXPECT(cond, ...)                  \
  do {                                     \
    if (!(cond)) {                         \
      fprintf(stderr, __VA_ARGS__);        \
      fprintf(stderr, "\n");               \
      ++failures;                          \
    }                                      \
  } while (0)

typedef struct {
  int32_t T, R;
  int64_t nn[4];
  oracle_ntype nt[4];
  oracle_etype et[6];
  int64_t *indptr[6], *indices[6];
  float *feat[4];
} graph;

/* distinct sources per destination, ascending; degree 0..max_deg, one hub
 * of degree up to a few thousand on some edge types */
static void make_graph(graph *g) {
  g->T = 1 + (int32_t)below(4);
  g->R = 1 + (int32_t)below(6);
  for (int32_t t = 0; t < g->T; ++t) {
    g->nn[t] = below(3000);
    g->feat[t] = NULL;
    if (below(5) > 0 && g->nn[t] > 0) {
      g->feat[t] = (float *)malloc(sizeof(float) * 3 * (size_t)g->nn[t]);
      for (int64_t i = 0; i < 3 * g->nn[t]; ++i) g->feat[t][i] = (float)below(1000);
    }
    g->nt[t].num_nodes = g->nn[t];
    g->nt[t].feat = g->feat[t];
    g->nt[t].row_bytes = g->feat[t] ? 12 : 0;
  }
  for (int32_t e = 0; e < g->R; ++e) {
    int32_t s = (int32_t)below(g->T), d = (int32_t)below(g->T);
    int64_t ns = g->nn[s], nd = g->nn[d];
    g->indptr[e] = (int64_t *)malloc(sizeof(int64_t) * (size_t)(nd + 1));
    int64_t cap = 1024;
    g->indices[e] = (int64_t *)malloc(sizeof(int64_t) * (size_t)cap);
    unsigned char *mark = (unsigned char *)calloc((size_t)ns + 1, 1);
    int64_t nnz = 0;
    g->indptr[e][0] = 0;
    for (int64_t v = 0; v < nd; ++v) {
      int64_t deg = below(12);
      if (below(500) == 0) deg = below(4000);
      if (deg > ns) deg = ns;
      /* the chosen sources, in ascending ID */
      int64_t got = 0;
      while (got < deg) {
        int64_t u = below(ns);
        if (!mark[u]) mark[u] = 1, ++got;
      }
      for (int64_t u = 0; u < ns && deg > 0; ++u)
        if (mark[u]) {
          if (nnz == cap) {
            cap *= 2;
            g->indices[e] = (int64_t *)realloc(g->indices[e], sizeof(int64_t) * (size_t)cap);
          }
          g->indices[e][nnz++] = u;
          mark[u] = 0;
        }
      g->indptr[e][v + 1] = nnz;
    }
    free(mark);
    g->et[e].src_type = s;
    g->et[e].dst_type = d;
    g->et[e].nnz = nnz;
    g->et[e].indptr = g->indptr[e];
    g->et[e].indices = g->indices[e];
  }
}

static void free_graph(graph *g) {
  for (int32_t t = 0; t < g->T; ++t) free(g->feat[t]);
  for (int32_t e = 0; e < g->R; ++e) {
    free(g->indptr[e]);
    free(g->indices[e]);
  }
}

/* reads every array of a result and checks the simple invariants */
static void read_back(const graph *g, const oracle_blocks *b, int32_t H) {
  for (int32_t h = 0; h < H; ++h) {
    for (int32_t t = 0; t < g->T; ++t) {
      int64_t nd = -1, ns = -1;
      const int64_t *sg = NULL;
      EXPECT(oracle_blocks_nodes(b, h, t, &nd, &ns, &sg) == ORACLE_OK, "nodes");
      EXPECT(nd >= 0 && ns >= nd, "hop %d type %d: %lld dst, %lld src", h, t, (long long)nd,
             (long long)ns);
      for (int64_t i = 0; i < ns; ++i)
        EXPECT(sg[i] >= 0 && sg[i] < g->nn[t], "source out of range");
    }
    for (int32_t e = 0; e < g->R; ++e) {
      int64_t ne = -1, nd = 0, ns = 0;
      const int64_t *ip = NULL, *eid = NULL, *sg = NULL;
      const int32_t *sl = NULL, *dl = NULL;
      EXPECT(oracle_blocks_edges(b, h, e, &ne, &ip, &sl, &dl, &eid) == ORACLE_OK, "edges");
      EXPECT(oracle_blocks_nodes(b, h, g->et[e].dst_type, &nd, &ns, &sg) == ORACLE_OK, "n");
      EXPECT(ip[0] == 0 && ip[nd] == ne, "block CSC ends");
      for (int64_t j = 0; j < ne; ++j) {
        EXPECT(eid[j] >= 0 && eid[j] < g->et[e].nnz, "edge ID out of range");
        EXPECT(dl[j] >= 0 && dl[j] < nd, "destination local ID out of range");
        EXPECT(sl[j] >= 0, "source local ID negative");
      }
    }
  }
  for (int32_t t = 0; t < g->T; ++t) {
    int64_t n = -1;
    const int64_t *gid = NULL;
    EXPECT(oracle_blocks_input_nodes(b, t, &n, &gid) == ORACLE_OK, "input");
    if (g->feat[t] && n > 0) {
      char *out = (char *)malloc((size_t)n * 12);
      EXPECT(oracle_gather_rows(g->feat[t], g->nn[t], 12, gid, n, out) == ORACLE_OK, "gather");
      for (int64_t i = 0; i < n; ++i)
        EXPECT(memcmp(out + 12 * i, (const char *)g->feat[t] + 12 * gid[i], 12) == 0,
               "gathered row");
      free(out);
    }
  }
}

/* distinct seeds of one type */
static int64_t *pick_seeds(int64_t n_nodes, int64_t want, int64_t *n) {
  if (want > n_nodes) want = n_nodes;
  int64_t *s = (int64_t *)malloc(sizeof(int64_t) * (size_t)(want + 1));
  unsigned char *mark = (unsigned char *)calloc((size_t)n_nodes + 1, 1);
  int64_t k = 0;
  while (k < want) {
    int64_t v = below(n_nodes);
    if (!mark[v]) mark[v] = 1, s[k++] = v;
  }
  free(mark);
  *n = k;
  return s;
}

static void vertex_batches(const graph *g) {
  int64_t *seeds[4] = {0}, ns[4] = {0};
  for (int32_t t = 0; t < g->T; ++t)
    if (below(2) == 0) seeds[t] = pick_seeds(g->nn[t], below(60), &ns[t]);
  int32_t H = (int32_t)below(4);
  int32_t fan[3 * 6];
  for (int32_t i = 0; i < H * g->R; ++i) fan[i] = (int32_t)below(8) - 1;
  int32_t kb = below(3) == 0 ? 1 + (int32_t)below(8) : 32;
  oracle_blocks *b = NULL;
  int st = oracle_sample_blocks(g->nt, g->T, g->et, g->R, (const int64_t *const *)seeds, ns, H,
                                fan, next_u64(), kb, &b);
  EXPECT(st == ORACLE_OK, "sample_blocks status %d", st);
  if (st == ORACLE_OK) {
    read_back(g, b, H);
    oracle_blocks_free(b);
  }
  /* a repeated seed is refused */
  for (int32_t t = 0; t < g->T; ++t)
    if (ns[t] > 0) {
      int64_t *dup = (int64_t *)malloc(sizeof(int64_t) * (size_t)(ns[t] + 1));
      memcpy(dup, seeds[t], sizeof(int64_t) * (size_t)ns[t]);
      dup[ns[t]] = seeds[t][0];
      int64_t *s2[4];
      int64_t n2[4];
      memcpy(s2, seeds, sizeof(s2));
      memcpy(n2, ns, sizeof(n2));
      s2[t] = dup;
      n2[t] = ns[t] + 1;
      b = NULL;
      EXPECT(oracle_sample_blocks(g->nt, g->T, g->et, g->R, (const int64_t *const *)s2, n2, H,
                                  fan, 1, 32, &b) == ORACLE_EINVAL,
             "repeated seed accepted");
      free(dup);
      break;
    }
  /* layer-wise from the same seeds */
  int32_t sizes[3 * 4];
  for (int32_t i = 0; i < H * g->T; ++i) sizes[i] = (int32_t)below(40) - 1;
  b = NULL;
  st = oracle_sample_layers(g->nt, g->T, g->et, g->R, (const int64_t *const *)seeds, ns, H,
                            sizes, next_u64(), &b);
  EXPECT(st == ORACLE_OK, "sample_layers status %d", st);
  if (st == ORACLE_OK) {
    read_back(g, b, H);
    oracle_blocks_free(b);
  }
  for (int32_t t = 0; t < g->T; ++t) free(seeds[t]);
}

static void edge_batches(const graph *g) {
  int64_t *eids[6] = {0}, n_eids[6] = {0};
  int32_t rev_etype[6];
  int64_t *rev_eid[6] = {0};
  for (int32_t e = 0; e < g->R; ++e) {
    rev_etype[e] = -1;
    if (g->et[e].nnz > 0 && below(2) == 0) {
      n_eids[e] = 1 + below(20);
      eids[e] = (int64_t *)malloc(sizeof(int64_t) * (size_t)n_eids[e]);
      for (int64_t i = 0; i < n_eids[e]; ++i) eids[e][i] = below(g->et[e].nnz);
    }
  }
  oracle_edge_batch eb;
  eb.eids = (const int64_t *const *)eids;
  eb.n_eids = n_eids;
  eb.n_neg = (int32_t)below(3);
  eb.exclude = (int32_t)below(2); /* 0 or 1: mode 2 needs reverse types */
  eb.rev_etype = rev_etype;
  eb.rev_eid = (const int64_t *const *)rev_eid;
  int32_t H = (int32_t)below(3);
  int32_t fan[2 * 6];
  for (int32_t i = 0; i < H * g->R; ++i) fan[i] = (int32_t)below(6) - 1;
  oracle_blocks *b = NULL;
  int st = oracle_sample_edge_blocks(g->nt, g->T, g->et, g->R, &eb, H, fan, next_u64(), 32, &b);
  EXPECT(st == ORACLE_OK, "sample_edge_blocks status %d", st);
  if (st == ORACLE_OK) {
    read_back(g, b, H);
    for (int32_t t = 0; t < g->T; ++t) {
      int64_t n = 0;
      const int64_t *gid = NULL;
      EXPECT(oracle_blocks_seeds(b, t, &n, &gid) == ORACLE_OK, "seeds");
      for (int64_t i = 1; i < n; ++i) EXPECT(gid[i - 1] < gid[i], "seeds not ascending");
    }
    for (int32_t e = 0; e < g->R; ++e) {
      int64_t np = 0, nn = 0;
      const int32_t *ps = NULL, *pd = NULL, *nd = NULL;
      EXPECT(oracle_blocks_pairs(b, e, &np, &ps, &pd, &nn, &nd) == ORACLE_OK, "pairs");
      EXPECT(np == n_eids[e] && nn == np * eb.n_neg, "pair counts");
      for (int64_t i = 0; i < np; ++i) EXPECT(ps[i] >= 0 && pd[i] >= 0, "pair IDs");
    }
    oracle_blocks_free(b);
  }
  /* a target out of range is refused */
  for (int32_t e = 0; e < g->R; ++e)
    if (n_eids[e] > 0) {
      const int64_t keep = eids[e][0];
      eids[e][0] = g->et[e].nnz;
      b = NULL;
      EXPECT(oracle_sample_edge_blocks(g->nt, g->T, g->et, g->R, &eb, H, fan, 3, 32, &b) ==
                 ORACLE_EINVAL,
             "target out of range accepted");
      eids[e][0] = keep;
      break;
    }
  for (int32_t e = 0; e < g->R; ++e) free(eids[e]);
}

int main(int argc, char **argv) {
  int rounds = argc > 1 ? atoi(argv[1]) : 60;
  for (int r = 0; r < rounds; ++r) {
    graph g;
    memset(&g, 0, sizeof(g));
    make_graph(&g);
    EXPECT(oracle_check_graph(g.nt, g.T, g.et, g.R) == ORACLE_OK, "graph check");
    vertex_batches(&g);
    edge_batches(&g);
    free_graph(&g);
  }
  /* single-pair selection and the generator on edge cases */
  int64_t out[64], n = 0;
  EXPECT(oracle_select(1, 0, 0, 10, 10, 3, 32, out, &n) == ORACLE_OK && n == 0, "empty pair");
  EXPECT(oracle_select(1, 0, 0, 0, 40, 5, 32, out, &n) == ORACLE_OK && n == 5, "select 5");
  EXPECT(oracle_select(1, 0, 0, 0, 40, -2, 32, out, &n) == ORACLE_EINVAL, "fanout -2");
  EXPECT(oracle_select(1, 0, 0, 0, 40, 5, 0, out, &n) == ORACLE_EINVAL, "key bits 0");
  uint32_t ctr[4] = {0, 0, 0, 0}, key[2] = {0, 0}, o[4];
  oracle_philox4x32_10(ctr, key, o);
  int64_t v = -1;
  const int64_t ip[4] = {0, 2, 2, 5};
  EXPECT(oracle_edge_dst(ip, 3, 4, &v) == ORACLE_OK && v == 2, "edge dst");
  EXPECT(oracle_edge_dst(ip, 3, 5, &v) == ORACLE_EINVAL, "edge dst out of range");
  EXPECT(oracle_negative_dst(7, 0, 3, 1, 100, &v) == ORACLE_OK && v >= 0 && v < 100, "negative");
  EXPECT(oracle_layer_weight(1) == (uint64_t)1 << 32, "weight of degree 1");
  EXPECT(oracle_layer_draw(5, 0, 0, 0, 0) == 0, "draw with total 0");
  if (failures) {
    fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  printf("oracle sanitizer run: %d graphs, every call as expected\n", rounds);
  return 0;
}
