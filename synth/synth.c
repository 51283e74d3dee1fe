/*
 * synth.c - seeded synthetic inputs shared by the oracle and the HIP path.
 *
 * This file holds none of the method's arithmetic: it only produces inputs.
 *   - Chung-Lu power-law graphs (each unordered pair {u,v} is an independent
 *     Bernoulli edge with p = min(1, w_u w_v / S)), generated in O(n + m)
 *     with the geometric-skip method of Miller & Hagberg, "Efficient
 *     generation of networks with given expected degrees" (WAW 2011).
 *     Only the edges inside one partition's node set V_p = local + halo are
 *     materialised, so a 111M-node graph never has to be held whole.
 *   - A random-range partitioner: node ids go through a seeded permutation
 *     and partition p owns the ids whose permuted position falls in the p-th
 *     of P contiguous ranges.
 *   - The partition view G_p: the subgraph induced on V_p, as a symmetric
 *     CSR with int64 row offsets and int32 partition-local column ids
 *     (local nodes [0,L) then halo nodes [L,L+H), each sorted by global id).
 *   - N(0,1) feature rows (Box-Muller on a counter-based hash of
 *     (seed, global id, column)), as fp32 or bf16 (round to nearest even).
 *   - Seed schedules: a seeded permutation of local ids picks the train set,
 *     each epoch reshuffles it, batches are consecutive chunks.
 *
 * Randomness is splitmix64 (Steele, Lea & Flood, OOPSLA 2014) used as a
 * counter-based generator, so results do not depend on the thread count.
 */
#define _GNU_SOURCE
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <stdio.h>

static int verbose(void) { const char* e = getenv("SYNTH_VERBOSE"); return e && *e == '1'; }
#define PHASE(name) do { if (verbose()) fprintf(stderr, "synth: %-24s %8.2fs\n", name, omp_get_wtime() - t_start); } while (0)

/* ------------------------------------------------------------------ RNG */
static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}
typedef struct { uint64_t s; } rng_t;
static inline rng_t rng_make(uint64_t seed, uint64_t stream, uint64_t phase) {
  rng_t r;
  r.s = mix64(seed * 0x9e3779b97f4a7c15ULL ^ mix64(stream + 0x632be59bd9b4e019ULL) ^
              (phase + 1) * 0xd1b54a32d192ed03ULL);
  return r;
}
static inline uint64_t rng_next(rng_t* r) {
  r->s += 0x9e3779b97f4a7c15ULL;
  return mix64(r->s);
}
/* uniform in (0, 1] */
static inline double rng_unif(rng_t* r) { return ((double)((rng_next(r) >> 11) + 1)) * 0x1.0p-53; }

/* ------------------------------------------------ seeded permutation of [0,n) */
typedef struct {
  uint32_t half;
  uint64_t mask, n, keys[4];
} feistel_t;

static feistel_t feistel_make(uint64_t n, uint64_t seed, uint64_t which) {
  feistel_t f;
  uint32_t bits = 2;
  while ((1ULL << bits) < n) bits += 2;
  f.half = bits / 2;
  f.mask = (1ULL << f.half) - 1;
  f.n = n;
  for (int r = 0; r < 4; r++) f.keys[r] = mix64(seed ^ mix64(which * 4 + r + 0x5851f42d4c957f2dULL));
  return f;
}
/* Four-round balanced Feistel network on 2*half bits, restricted to [0,n)
 * by cycle walking: a bijection of [0,n). */
static inline uint64_t feistel_perm(const feistel_t* f, uint64_t x) {
  do {
    uint64_t l = x >> f->half, r = x & f->mask;
    for (int k = 0; k < 4; k++) {
      uint64_t nl = r;
      r = l ^ (mix64(r ^ f->keys[k]) & f->mask);
      l = nl;
    }
    x = (l << f->half) | r;
  } while (x >= f->n);
  return x;
}

/* --------------------------------------------------------- Chung-Lu weights */
/* w_i = w_max * ((i + i0) / i0)^(-g), g = 1/(beta-1), i = 0..n-1, with
 * w_max = sqrt(n * mean) (so that w_u w_v / S <= 1) and i0 chosen so that
 * the mean weight equals `mean`. */
static double weight_sum_ratio(uint64_t n, double g, double i0) {
  uint64_t m = n < (1ULL << 16) ? n : (1ULL << 16);
  double s = 0.0;
  for (uint64_t i = 0; i < m; i++) s += pow(((double)i + i0) / i0, -g);
  if (m < n) {
    double a = ((double)m - 0.5 + i0) / i0, b = ((double)n - 0.5 + i0) / i0;
    if (fabs(g - 1.0) < 1e-12)
      s += i0 * log(b / a);
    else
      s += i0 / (1.0 - g) * (pow(b, 1.0 - g) - pow(a, 1.0 - g));
  }
  return s;
}

int synth_weights(uint64_t n, double beta, double mean, double* w_out, double* i0_out) {
  if (n < 2 || beta <= 1.0 || mean <= 0.0) return -1;
  double g = 1.0 / (beta - 1.0), wmax = sqrt((double)n * mean);
  double lo = log(1e-9), hi = log(1e15);
  for (int it = 0; it < 80; it++) {
    double mid = 0.5 * (lo + hi), i0 = exp(mid);
    double m = wmax * weight_sum_ratio(n, g, i0) / (double)n;
    if (m < mean) lo = mid; else hi = mid;
  }
  double i0 = exp(0.5 * (lo + hi));
  if (i0_out) *i0_out = i0;
  if (w_out) {
#pragma omp parallel for schedule(static)
    for (uint64_t i = 0; i < n; i++) w_out[i] = wmax * pow(((double)i + i0) / i0, -g);
  }
  return 0;
}

/* ------------------------------------------------------------- edge chunks */
typedef struct {
  uint32_t* uv; /* pairs (u, v), weight-index space */
  uint64_t len, cap;
} chunk_t;

static inline int chunk_push(chunk_t* c, uint32_t u, uint32_t v) {
  if (c->len == c->cap) {
    uint64_t nc = c->cap ? c->cap * 2 : 1024;
    uint32_t* p = (uint32_t*)realloc(c->uv, nc * 2 * sizeof(uint32_t));
    if (!p) return -1;
    c->uv = p;
    c->cap = nc;
  }
  c->uv[2 * c->len] = u;
  c->uv[2 * c->len + 1] = v;
  c->len++;
  return 0;
}

static inline double edge_prob(double wu, double wv, double S, int sym) {
  double p = wu * wv / S;
  if (p > 1.0) p = 1.0;
  /* "directed then symmetrized": the undirected pair exists if either
   * independent directed draw succeeds. */
  if (sym) p = 1.0 - (1.0 - p) * (1.0 - p);
  return p;
}

/* Geometric-skip walk of pairs (u, seq[pos]) for pos in [pos0, len), with
 * seq ascending in weight index (so weights non-increasing). seq == NULL
 * means the identity sequence. */
static int walk_pairs(uint32_t u, const uint32_t* seq, uint64_t pos0, uint64_t len, const double* w,
                      double S, int sym, rng_t* r, chunk_t* out) {
  uint64_t pos = pos0;
  if (pos >= len) return 0;
  double wu = w[u];
  double p = edge_prob(wu, w[seq ? seq[pos] : pos], S, sym);
  while (pos < len && p > 0.0) {
    if (p < 1.0) {
      double skip = floor(log(rng_unif(r)) / log1p(-p));
      if (skip >= (double)(len - pos)) break;
      pos += (uint64_t)skip;
    }
    uint32_t v = seq ? seq[pos] : (uint32_t)pos;
    double q = edge_prob(wu, w[v], S, sym);
    if (rng_unif(r) <= q / p)
      if (chunk_push(out, u, v)) return -1;
    p = q;
    pos++;
  }
  return 0;
}

/* ----------------------------------------------------- partition view G_p */
typedef struct {
  int64_t L, H, nnz;
  int64_t* indptr;     /* [L+H+1] */
  int32_t* indices;    /* [nnz]   partition-local ids, ascending per row */
  int32_t* local_gid;  /* [L] */
  int32_t* halo_gid;   /* [H] */
  int64_t* halo_degree;/* [H] row length in G_p */
  int64_t edges_a, edges_b; /* undirected edges: with a local end / halo-halo */
  double i0;
} synth_graph;

static int cmp_u64(const void* a, const void* b) {
  uint64_t x = *(const uint64_t*)a, y = *(const uint64_t*)b;
  return x < y ? -1 : x > y;
}
static int cmp_i32(const void* a, const void* b) {
  int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
  return x < y ? -1 : x > y;
}

void synth_graph_free(synth_graph* g) {
  if (!g) return;
  free(g->indptr);
  free(g->indices);
  free(g->local_gid);
  free(g->halo_gid);
  free(g->halo_degree);
  free(g);
}

/* Build G_p for partition `part` of P. n nodes, Chung-Lu exponent beta,
 * mean degree `mean`; sym != 0 draws directed edges and symmetrises. */
synth_graph* synth_partition_graph(uint64_t n, double beta, double mean, int sym, int P, int part,
                                   uint64_t seed, int threads) {
  if (n < 2 || n >= (1ULL << 31) || P < 1 || part < 0 || part >= P) return NULL;
  if (threads > 0) omp_set_num_threads(threads);
  double t_start = omp_get_wtime();
  synth_graph* G = (synth_graph*)calloc(1, sizeof(synth_graph));
  double* w = (double*)malloc(n * sizeof(double));
  uint8_t* cls = (uint8_t*)calloc(n, 1); /* 1 local, 2 halo */
  if (!G || !w || !cls) goto fail;
  /* For the directed-then-symmetrised case the per-direction weights have
   * mean `mean` (mean out-degree). */
  if (synth_weights(n, beta, mean, w, &G->i0)) goto fail;
  double S = 0.0;
  for (uint64_t i = 0; i < n; i++) S += w[i];

  /* weight index i -> global id gid(i) -> partition of gid */
  feistel_t fid = feistel_make(n, seed, 1), fpart = feistel_make(n, seed, 2);
  uint64_t lo = (uint64_t)part * n / (uint64_t)P, hi = (uint64_t)(part + 1) * n / (uint64_t)P;
  uint32_t* gid = (uint32_t*)malloc(n * sizeof(uint32_t));
  if (!gid) goto fail;
#pragma omp parallel for schedule(static)
  for (uint64_t i = 0; i < n; i++) {
    uint64_t g = feistel_perm(&fid, i);
    gid[i] = (uint32_t)g;
    uint64_t pp = feistel_perm(&fpart, g);
    cls[i] = (pp >= lo && pp < hi) ? 1 : 0;
  }
  PHASE("weights+ids");
  uint64_t nloc = 0;
  for (uint64_t i = 0; i < n; i++) nloc += cls[i] == 1;
  uint32_t* locseq = (uint32_t*)malloc((nloc ? nloc : 1) * sizeof(uint32_t));
  if (!locseq) { free(gid); goto fail; }
  {
    uint64_t k = 0;
    for (uint64_t i = 0; i < n; i++)
      if (cls[i] == 1) locseq[k++] = (uint32_t)i;
  }

  const uint64_t CH = 1 << 10;
  uint64_t nch = (n + CH - 1) / CH;
  chunk_t* chA = (chunk_t*)calloc(nch, sizeof(chunk_t));
  int err = 0;
  /* Phase A: every pair with at least one local end. A local u walks all
   * v > u; a non-local u walks only the local v > u. */
#pragma omp parallel for schedule(dynamic, 1)
  for (uint64_t c = 0; c < nch; c++) {
    uint64_t u0 = c * CH, u1 = u0 + CH < n ? u0 + CH : n;
    /* first local position > u0 */
    uint64_t a = 0, b = nloc;
    while (a < b) { uint64_t m = (a + b) / 2; if (locseq[m] <= u0) a = m + 1; else b = m; }
    uint64_t lp = a;
    for (uint64_t u = u0; u < u1; u++) {
      while (lp < nloc && locseq[lp] <= u) lp++;
      rng_t r = rng_make(seed, u, 1);
      int e;
      if (cls[u] == 1)
        e = walk_pairs((uint32_t)u, NULL, u + 1, n, w, S, sym, &r, &chA[c]);
      else
        e = walk_pairs((uint32_t)u, locseq, lp, nloc, w, S, sym, &r, &chA[c]);
      if (e) err = 1;
    }
  }
  PHASE("phase A");
  if (err) { free(gid); free(locseq); goto fail_ch; }
  /* halo = non-local ends of phase-A edges */
  uint64_t ea = 0;
  for (uint64_t c = 0; c < nch; c++) {
    ea += chA[c].len;
    for (uint64_t e = 0; e < chA[c].len; e++) {
      uint32_t u = chA[c].uv[2 * e], v = chA[c].uv[2 * e + 1];
      if (cls[u] != 1) cls[u] = 2;
      if (cls[v] != 1) cls[v] = 2;
    }
  }
  uint64_t nhalo = 0;
  for (uint64_t i = 0; i < n; i++) nhalo += cls[i] == 2;
  uint32_t* haloseq = (uint32_t*)malloc((nhalo ? nhalo : 1) * sizeof(uint32_t));
  {
    uint64_t k = 0;
    for (uint64_t i = 0; i < n; i++)
      if (cls[i] == 2) haloseq[k++] = (uint32_t)i;
  }
  /* Phase B: halo-halo pairs, each halo u walks the halo v > u. */
  uint64_t nchb = (nhalo + CH - 1) / CH;
  chunk_t* chB = (chunk_t*)calloc(nchb ? nchb : 1, sizeof(chunk_t));
#pragma omp parallel for schedule(dynamic, 1)
  for (uint64_t c = 0; c < nchb; c++) {
    uint64_t p0 = c * CH, p1 = p0 + CH < nhalo ? p0 + CH : nhalo;
    for (uint64_t p = p0; p < p1; p++) {
      uint32_t u = haloseq[p];
      rng_t r = rng_make(seed, u, 2);
      if (walk_pairs(u, haloseq, p + 1, nhalo, w, S, sym, &r, &chB[c])) err = 1;
    }
  }
  PHASE("phase B");
  uint64_t eb = 0;
  for (uint64_t c = 0; c < nchb; c++) eb += chB[c].len;

  /* partition-local ids: local sorted by gid, then halo sorted by gid */
  int32_t* pl = (int32_t*)malloc(n * sizeof(int32_t));
  uint64_t* key = (uint64_t*)malloc((nloc > nhalo ? nloc : nhalo) * sizeof(uint64_t) + 8);
  G->L = (int64_t)nloc;
  G->H = (int64_t)nhalo;
  G->local_gid = (int32_t*)malloc((nloc ? nloc : 1) * sizeof(int32_t));
  G->halo_gid = (int32_t*)malloc((nhalo ? nhalo : 1) * sizeof(int32_t));
  if (err || !pl || !key || !G->local_gid || !G->halo_gid) {
    free(pl); free(key); free(gid); free(locseq); free(haloseq);
    for (uint64_t c = 0; c < nchb; c++) free(chB[c].uv);
    free(chB);
    goto fail_ch;
  }
#pragma omp parallel for schedule(static)
  for (uint64_t i = 0; i < n; i++) pl[i] = -1;
  for (uint64_t k = 0; k < nloc; k++) key[k] = ((uint64_t)gid[locseq[k]] << 32) | locseq[k];
  qsort(key, nloc, sizeof(uint64_t), cmp_u64);
  for (uint64_t k = 0; k < nloc; k++) {
    pl[key[k] & 0xffffffffULL] = (int32_t)k;
    G->local_gid[k] = (int32_t)(key[k] >> 32);
  }
  for (uint64_t k = 0; k < nhalo; k++) key[k] = ((uint64_t)gid[haloseq[k]] << 32) | haloseq[k];
  qsort(key, nhalo, sizeof(uint64_t), cmp_u64);
  for (uint64_t k = 0; k < nhalo; k++) {
    pl[key[k] & 0xffffffffULL] = (int32_t)(nloc + k);
    G->halo_gid[k] = (int32_t)(key[k] >> 32);
  }
  free(key);
  free(gid);
  free(locseq);
  free(haloseq);

  PHASE("local ids");
  /* symmetric CSR over L+H rows, without atomics: every thread counts and
   * fills the same round-robin set of chunks, with its own cursors. */
  int64_t R = G->L + G->H;
  int nt = omp_get_max_threads();
  G->indptr = (int64_t*)calloc((size_t)R + 1, sizeof(int64_t));
  int64_t* cur = (int64_t*)calloc((size_t)nt * (size_t)R, sizeof(int64_t));
  if (!G->indptr || !cur) { free(cur); free(pl); goto fail_all; }
  for (int pass = 0; pass < 2; pass++) {
    chunk_t* ch = pass ? chB : chA;
    uint64_t nc = pass ? nchb : nch;
#pragma omp parallel num_threads(nt)
    {
      int64_t* mine = cur + (size_t)omp_get_thread_num() * (size_t)R;
#pragma omp for schedule(static, 1)
      for (uint64_t c = 0; c < nc; c++)
        for (uint64_t e = 0; e < ch[c].len; e++) {
          mine[pl[ch[c].uv[2 * e]]]++;
          mine[pl[ch[c].uv[2 * e + 1]]]++;
        }
    }
  }
  /* row offsets, then per-thread start cursors inside each row */
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < R; i++) {
    int64_t s = 0;
    for (int t = 0; t < nt; t++) s += cur[(size_t)t * R + i];
    G->indptr[i + 1] = s;
  }
  for (int64_t i = 0; i < R; i++) G->indptr[i + 1] += G->indptr[i];
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < R; i++) {
    int64_t o = G->indptr[i];
    for (int t = 0; t < nt; t++) {
      int64_t c = cur[(size_t)t * R + i];
      cur[(size_t)t * R + i] = o;
      o += c;
    }
  }
  G->nnz = G->indptr[R];
  G->indices = (int32_t*)malloc((size_t)(G->nnz ? G->nnz : 1) * sizeof(int32_t));
  if (!G->indices) { free(cur); free(pl); goto fail_all; }
  for (int pass = 0; pass < 2; pass++) {
    chunk_t* ch = pass ? chB : chA;
    uint64_t nc = pass ? nchb : nch;
#pragma omp parallel num_threads(nt)
    {
      int64_t* mine = cur + (size_t)omp_get_thread_num() * (size_t)R;
#pragma omp for schedule(static, 1)
      for (uint64_t c = 0; c < nc; c++) {
        for (uint64_t e = 0; e < ch[c].len; e++) {
          int32_t a = pl[ch[c].uv[2 * e]], b = pl[ch[c].uv[2 * e + 1]];
          G->indices[mine[a]++] = b;
          G->indices[mine[b]++] = a;
        }
        free(ch[c].uv);
        ch[c].uv = NULL;
      }
    }
  }
  PHASE("csr fill");
  free(cur);
  free(pl);
  free(chA);
  free(chB);
#pragma omp parallel for schedule(dynamic, 4096)
  for (int64_t i = 0; i < R; i++)
    qsort(G->indices + G->indptr[i], (size_t)(G->indptr[i + 1] - G->indptr[i]), sizeof(int32_t), cmp_i32);
  PHASE("row sort");
  G->halo_degree = (int64_t*)malloc((size_t)(G->H ? G->H : 1) * sizeof(int64_t));
  for (int64_t h = 0; h < G->H; h++) G->halo_degree[h] = G->indptr[G->L + h + 1] - G->indptr[G->L + h];
  G->edges_a = (int64_t)ea;
  G->edges_b = (int64_t)eb;
  free(w);
  free(cls);
  return G;

fail_all:
  for (uint64_t c = 0; c < nchb; c++) free(chB[c].uv);
  free(chB);
  chB = NULL;
fail_ch:
  for (uint64_t c = 0; c < nch; c++) free(chA[c].uv);
  free(chA);
fail:
  free(w);
  free(cls);
  synth_graph_free(G);
  return NULL;
}

/* ------------------------------------------------------------- features */
static inline uint16_t f32_to_bf16_rne(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

/* out[r*d + c] = N(0,1) value of (seed, gid[r], c); dtype 0 fp32, 1 bf16 */
void synth_features(const int32_t* gid, int64_t rows, int32_t d, int32_t dtype, uint64_t seed,
                    void* out, int threads) {
  if (threads > 0) omp_set_num_threads(threads);
#pragma omp parallel for schedule(static, 1024)
  for (int64_t r = 0; r < rows; r++) {
    uint64_t g = (uint64_t)(uint32_t)gid[r];
    for (int32_t c = 0; c < d; c += 2) {
      uint64_t h1 = mix64(seed ^ mix64((g << 20) ^ (uint64_t)c ^ 0x1234567ULL));
      uint64_t h2 = mix64(h1 ^ 0xa0761d6478bd642fULL);
      double u1 = ((double)((h1 >> 11) + 1)) * 0x1.0p-53, u2 = ((double)(h2 >> 11)) * 0x1.0p-53;
      double rad = sqrt(-2.0 * log(u1));
      float z0 = (float)(rad * cos(6.283185307179586 * u2));
      float z1 = (float)(rad * sin(6.283185307179586 * u2));
      if (dtype == 0) {
        float* o = (float*)out + (size_t)r * d;
        o[c] = z0;
        if (c + 1 < d) o[c + 1] = z1;
      } else {
        uint16_t* o = (uint16_t*)out + (size_t)r * d;
        o[c] = f32_to_bf16_rne(z0);
        if (c + 1 < d) o[c + 1] = f32_to_bf16_rne(z1);
      }
    }
  }
}

/* ----------------------------------------------------------- seed schedule */
static void shuffle_i32(int32_t* a, int64_t n, rng_t* r) {
  for (int64_t i = n - 1; i > 0; i--) {
    int64_t j = (int64_t)(rng_next(r) % (uint64_t)(i + 1));
    int32_t t = a[i]; a[i] = a[j]; a[j] = t;
  }
}

/* Train set: the first ceil(pct*L/100) entries of a seeded permutation of
 * [0,L). Returns its size; fills `out` (capacity L) with the train set
 * shuffled for `epoch`. */
int64_t synth_epoch_order(int64_t L, int32_t pct, uint64_t seed, int64_t epoch, int32_t* out) {
  if (L <= 0 || pct <= 0 || pct > 100) return -1;
  int64_t T = ((int64_t)pct * L + 99) / 100;
  for (int64_t i = 0; i < L; i++) out[i] = (int32_t)i;
  rng_t r = rng_make(seed, 0x7472616eULL, 3);
  shuffle_i32(out, L, &r);
  rng_t re = rng_make(seed, (uint64_t)epoch, 4);
  shuffle_i32(out, T, &re);
  return T;
}
