/*
 * oracle.c - plain, slow, single-threaded CPU oracle of MassiveGNN's
 * per-minibatch path for one partition (arXiv 2410.22697).
 *
 * TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the bench's
 * CPU-baseline leg may load this library; the product path never does.
 * It shares no code, header, table or helper with the HIP library.
 *
 * What it computes, in the paper's order (Algorithm 2, PREFETCH_WITH_EVICTION,
 * and EVICT_AND_REPLACE; scoring rules of Section IV-B; Eq. 1):
 *   initialize_prefetcher (Algorithm 1): BUF = the f share of the halo with
 *     the largest degrees,
 *     S_E = 1 on BUF, S_A = -1 on BUF and 0 on the other halo nodes,
 *     alpha = gamma^Delta.
 *   NeighborSampler: uniform fanout sampling without replacement, hop by hop
 *     (Section V: a fixed-size uniform set of neighbours per node; the
 *     recursion over layers of Section I). The uniform choice is made
 *     deterministic with counter-based Philox4x32-10 keys (Salmon, Moraes,
 *     Dror & Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3", SC'11).
 *   V^{l|s}, V^{h|s}, Hits, Misses: set intersections with V^l, V^h, BUF.
 *   S_E decay on buffered nodes not sampled this step.
 *   Local copy, buffer copy, miss fetch (the remote store).
 *   S_A += 1 on every miss.
 *   Every Delta steps: evict buffered nodes with S_E < alpha, replace them
 *   by the unbuffered halo nodes with the highest S_A, swap the scores.
 *
 * Readings taken where the paper is silent or ambiguous (each also listed in
 * the design notes):
 *   - The sampler walks G_p, the subgraph induced on local + halo nodes.
 *   - Fanouts are hop-first; every hop samples for the whole frontier and the
 *     new nodes are appended, so frontier k is a prefix of frontier k+1.
 *   - Philox key of CSR position j of node v at step t, hop k (1-based):
 *     word (j mod 4) of Philox4x32-10(counter = (j/4, v, t, k),
 *     key = (seed_lo, seed_hi)). A row with d <= fanout keeps every position;
 *     otherwise the fanout positions with the smallest (key, j) are kept.
 *     Emitted in ascending j. New frontier nodes in ascending id.
 *   - t is a global step counter across epochs; a round runs after step t
 *     iff t > 0 and t mod Delta == 0.
 *   - alpha = a_Delta with a_0 = 1.0f, a_{i+1} = fl32(a_i * gamma); strict <.
 *   - Decay runs every step (rounds included) before the round; S_A += 1 on
 *     misses every step (rounds included) before the round.
 *   - Candidates: halo nodes with S_A >= 0, ordered by (S_A desc, rank asc);
 *     rank orders halo nodes by (degree desc, global id asc).
 *   - k' = min(|E|, |C|); if fewer candidates than evictions, the k' slots
 *     with the smallest (S_E, rank) are evicted.
 *   - E (ascending slot) is paired with R in candidate order.
 *   - Swap: evicted node's S_A := its last S_E; slot's new S_E := the
 *     replacement's last S_A; replacement's S_A := -1.
 *   - cap = floor(H * pct / 100). All scores fp32.
 */
#define _POSIX_C_SOURCE 199309L
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <time.h>

enum {
  OR_OK = 0,
  OR_EINVAL = -1,
  OR_ENOMEM = -3,
  OR_ESTATE = -5,
};

/* ------------------------------------------------------------ Philox4x32-10 */
/* SC'11, Section 4: each round multiplies counter words 0 and 2 by the
 * constants M0, M1 (full 64-bit products), then permutes and mixes with the
 * round key; the key is bumped by the Weyl constants W0, W1 between rounds. */
void oracle_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
  uint32_t x0 = ctr_in[0], x1 = ctr_in[1], x2 = ctr_in[2], x3 = ctr_in[3];
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int round = 0; round < 10; round++) {
    if (round > 0) {
      k0 += W0;
      k1 += W1;
    }
    uint64_t p0 = (uint64_t)M0 * x0;
    uint64_t p1 = (uint64_t)M1 * x2;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t y0 = hi1 ^ x1 ^ k0;
    uint32_t y1 = lo1;
    uint32_t y2 = hi0 ^ x3 ^ k1;
    uint32_t y3 = lo0;
    x0 = y0; x1 = y1; x2 = y2; x3 = y3;
  }
  out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* ------------------------------------------------------------------ state */
typedef struct {
  int32_t L, H;
  const int64_t* indptr;     /* [L+H+1] G_p */
  const int32_t* indices;    /* [nnz] */
  const int32_t* halo_gid;   /* [H] */
  const int64_t* halo_degree;/* [H] */
  const void* local_feat;    /* [L * row_bytes] */
  const void* halo_store;    /* [H * row_bytes] remote store */
  int64_t row_bytes;
  int32_t K;
  int32_t fanout[8];
  int32_t buffer_pct;
  float gamma;
  int32_t delta;
  uint64_t seed;
} oracle_args;

typedef struct {
  oracle_args a;
  /* prefetcher state (Table I) */
  int64_t cap;
  int32_t* rank;      /* [H] rank of halo node h */
  int32_t* slot_id;   /* [cap] BUF: halo node held by slot s */
  int32_t* slot_of;   /* [H] slot of h, -1 if h not in BUF */
  float* S_E;         /* [cap] */
  float* S_A;         /* [H] */
  uint8_t* buf;       /* [cap * row_bytes] buffered feature rows */
  float alpha;
  int64_t t;          /* steps sampled so far */
  int pending_round;  /* the last sampled step still owes its evict call */
  /* outputs of the last step */
  int32_t* F;         /* frontier, [n_K] */
  int64_t nF_cap;
  int64_t n[9], e[8];
  int32_t* blk_indptr[8];
  int32_t* blk_indices[8];
  uint8_t* mask;      /* 0 local, 1 hit, 2 miss */
  uint8_t* feat;      /* [n_K * row_bytes] */
  int64_t hits, misses, local;
  /* scratch */
  int32_t* pos;       /* [L+H] position in F or -1 */
  /* time per phase, seconds (sample, dedup, classify, score, gather, evict) */
  double tphase[6];
} oracle_ctx;

static double now_s(void) {
  struct timespec ts;
  clock_gettime(CLOCK_MONOTONIC, &ts);
  return (double)ts.tv_sec + 1e-9 * (double)ts.tv_nsec;
}

static const oracle_ctx* g_rank_ctx; /* qsort comparators need the context */

/* rank order: degree desc, global id asc */
static int cmp_rank(const void* pa, const void* pb) {
  int32_t x = *(const int32_t*)pa, y = *(const int32_t*)pb;
  int64_t dx = g_rank_ctx->a.halo_degree[x], dy = g_rank_ctx->a.halo_degree[y];
  if (dx != dy) return dx > dy ? -1 : 1;
  int32_t gx = g_rank_ctx->a.halo_gid[x], gy = g_rank_ctx->a.halo_gid[y];
  return gx < gy ? -1 : gx > gy;
}

void oracle_destroy(oracle_ctx* c) {
  if (!c) return;
  free(c->rank); free(c->slot_id); free(c->slot_of); free(c->S_E); free(c->S_A); free(c->buf);
  free(c->F); free(c->mask); free(c->feat); free(c->pos);
  for (int k = 0; k < 8; k++) { free(c->blk_indptr[k]); free(c->blk_indices[k]); }
  free(c);
}

/* INITIALIZE_PREFETCHER (Algorithm 1). */
int oracle_init(const oracle_args* a, oracle_ctx** out) {
  *out = NULL;
  if (!a || a->L < 0 || a->H < 0 || (int64_t)a->L + a->H <= 0 || a->K < 1 || a->K > 8 ||
      a->row_bytes <= 0 || a->buffer_pct < 0 || a->buffer_pct > 100 || a->delta < 1 ||
      !(a->gamma > 0.0f && a->gamma <= 1.0f) || !a->indptr || !a->indices)
    return OR_EINVAL;
  for (int k = 0; k < a->K; k++)
    if (a->fanout[k] < 1) return OR_EINVAL;
  oracle_ctx* c = (oracle_ctx*)calloc(1, sizeof(oracle_ctx));
  if (!c) return OR_ENOMEM;
  c->a = *a;
  int64_t H = a->H, R = (int64_t)a->L + a->H;
  c->cap = H * a->buffer_pct / 100;
  c->rank = (int32_t*)malloc(sizeof(int32_t) * (size_t)(H ? H : 1));
  c->slot_id = (int32_t*)malloc(sizeof(int32_t) * (size_t)(c->cap ? c->cap : 1));
  c->slot_of = (int32_t*)malloc(sizeof(int32_t) * (size_t)(H ? H : 1));
  c->S_E = (float*)malloc(sizeof(float) * (size_t)(c->cap ? c->cap : 1));
  c->S_A = (float*)malloc(sizeof(float) * (size_t)(H ? H : 1));
  c->buf = (uint8_t*)malloc((size_t)(c->cap ? c->cap : 1) * (size_t)a->row_bytes);
  c->pos = (int32_t*)malloc(sizeof(int32_t) * (size_t)R);
  if (!c->rank || !c->slot_id || !c->slot_of || !c->S_E || !c->S_A || !c->buf || !c->pos) {
    oracle_destroy(c);
    return OR_ENOMEM;
  }
  for (int64_t v = 0; v < R; v++) c->pos[v] = -1;
  /* Algorithm 1 fills the buffer with the highest-degree share f of the halo:
   * order the halo by degree (ties by global id) */
  int32_t* order = (int32_t*)malloc(sizeof(int32_t) * (size_t)(H ? H : 1));
  if (!order) { oracle_destroy(c); return OR_ENOMEM; }
  for (int64_t h = 0; h < H; h++) order[h] = (int32_t)h;
  g_rank_ctx = c;
  qsort(order, (size_t)H, sizeof(int32_t), cmp_rank);
  for (int64_t r = 0; r < H; r++) c->rank[order[r]] = (int32_t)r;
  for (int64_t h = 0; h < H; h++) {
    c->slot_of[h] = -1;
    c->S_A[h] = 0.0f;                       /* Algorithm 1: unbuffered halo nodes start at 0 */
  }
  for (int64_t s = 0; s < c->cap; s++) {
    int32_t h = order[s];
    c->slot_id[s] = h;
    c->slot_of[h] = (int32_t)s;
    c->S_E[s] = 1.0f;                       /* Algorithm 1: buffered nodes start at 1 */
    c->S_A[h] = -1.0f;                      /* ... and carry -1 as their S_A */
    memcpy(c->buf + (size_t)s * a->row_bytes,
           (const uint8_t*)a->halo_store + (size_t)h * a->row_bytes, (size_t)a->row_bytes);
  }
  free(order);
  /* Eq. 1 with S_E at its initial value 1: alpha = gamma^Delta, as Delta
   * successive fp32 multiplies. */
  float al = 1.0f;
  for (int32_t i = 0; i < a->delta; i++) al = al * a->gamma;
  c->alpha = al;
  c->t = 0;
  *out = c;
  return OR_OK;
}

static int grow_i32(int32_t** p, int64_t* capn, int64_t need) {
  if (need <= *capn) return 0;
  int64_t nc = need > 2 * *capn ? need : 2 * *capn;
  int32_t* q = (int32_t*)realloc(*p, sizeof(int32_t) * (size_t)nc);
  if (!q) return -1;
  *p = q;
  *capn = nc;
  return 0;
}

static int cmp_u64(const void* pa, const void* pb) {
  uint64_t x = *(const uint64_t*)pa, y = *(const uint64_t*)pb;
  return x < y ? -1 : x > y;
}
static int cmp_i32(const void* pa, const void* pb) {
  int32_t x = *(const int32_t*)pa, y = *(const int32_t*)pb;
  return x < y ? -1 : x > y;
}

/* Uniform fanout choice for one row: fills sel[0..m) with the chosen CSR
 * positions (ascending) and returns m = min(d, fo). */
static int64_t choose_positions(const oracle_ctx* c, int32_t v, int64_t d, int32_t fo, int32_t k,
                                int64_t* sel, uint64_t* keybuf) {
  if (d <= fo) {
    for (int64_t j = 0; j < d; j++) sel[j] = j;
    return d;
  }
  uint32_t key[2] = {(uint32_t)c->a.seed, (uint32_t)(c->a.seed >> 32)};
  uint32_t words[4];
  for (int64_t j = 0; j < d; j++) {
    if (j % 4 == 0) {
      uint32_t ctr[4] = {(uint32_t)(j / 4), (uint32_t)v, (uint32_t)c->t, (uint32_t)k};
      oracle_philox4x32_10(ctr, key, words);
    }
    /* (key, position) packed so that the sort orders by key then by j */
    keybuf[j] = ((uint64_t)words[j % 4] << 32) | (uint64_t)j;
  }
  qsort(keybuf, (size_t)d, sizeof(uint64_t), cmp_u64);
  for (int32_t i = 0; i < fo; i++) sel[i] = (int64_t)(keybuf[i] & 0xffffffffu);
  /* emit in ascending position */
  for (int32_t i = 1; i < fo; i++) {
    int64_t x = sel[i];
    int32_t p = i;
    while (p > 0 && sel[p - 1] > x) { sel[p] = sel[p - 1]; p--; }
    sel[p] = x;
  }
  return fo;
}

/* PREFETCH_WITH_EVICTION for the batch `seeds` at step t (Algorithm 2),
 * except the eviction round, which oracle_evict_step runs afterwards. */
int oracle_sample(oracle_ctx* c, const int32_t* seeds, int32_t n0) {
  if (c->pending_round) return OR_ESTATE;
  if (n0 < 0 || (n0 > 0 && !seeds)) return OR_EINVAL;
  const int32_t L = c->a.L;
  for (int32_t i = 0; i < n0; i++)
    if (seeds[i] < 0 || seeds[i] >= L) return OR_EINVAL;   /* seeds are local nodes */
  double t0 = now_s();

  /* frontier F_0 = seeds */
  if (grow_i32(&c->F, &c->nF_cap, n0 > 0 ? n0 : 1)) return OR_ENOMEM;
  int64_t nF = 0;
  for (int32_t i = 0; i < n0; i++) {
    if (c->pos[seeds[i]] >= 0) {                             /* duplicate seed */
      for (int64_t q = 0; q < nF; q++) c->pos[c->F[q]] = -1;
      return OR_EINVAL;
    }
    c->pos[seeds[i]] = (int32_t)nF;
    c->F[nF++] = seeds[i];
  }
  c->n[0] = nF;

  int64_t maxdeg = 0;
  double t_sample = 0.0, t_dedup = 0.0;
  int rc = OR_OK;
  int64_t* sel = NULL;
  uint64_t* keybuf = NULL;
  int32_t* raw = NULL;
  int32_t* uniq = NULL;
  int64_t sel_cap = 0;

  for (int32_t k = 1; k <= c->a.K; k++) {
    double ta = now_s();
    const int32_t fo = c->a.fanout[k - 1];
    const int64_t nprev = nF;
    /* NeighborSampler, hop k, for every node of F_{k-1} */
    int64_t E = 0;
    for (int64_t i = 0; i < nprev; i++) {
      int64_t d = c->a.indptr[c->F[i] + 1] - c->a.indptr[c->F[i]];
      E += d < fo ? d : fo;
      if (d > maxdeg) maxdeg = d;
    }
    if (maxdeg + 1 > sel_cap) {
      sel_cap = maxdeg + 1;
      free(sel); free(keybuf);
      sel = (int64_t*)malloc(sizeof(int64_t) * (size_t)sel_cap);
      keybuf = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)sel_cap);
      if (!sel || !keybuf) { rc = OR_ENOMEM; goto done; }
    }
    free(c->blk_indptr[k - 1]);
    free(c->blk_indices[k - 1]);
    c->blk_indptr[k - 1] = (int32_t*)malloc(sizeof(int32_t) * (size_t)(nprev + 1));
    c->blk_indices[k - 1] = (int32_t*)malloc(sizeof(int32_t) * (size_t)(E ? E : 1));
    free(raw);
    raw = (int32_t*)malloc(sizeof(int32_t) * (size_t)(E ? E : 1));
    if (!c->blk_indptr[k - 1] || !c->blk_indices[k - 1] || !raw) { rc = OR_ENOMEM; goto done; }
    int32_t* bptr = c->blk_indptr[k - 1];
    int64_t o = 0;
    for (int64_t i = 0; i < nprev; i++) {
      int32_t v = c->F[i];
      int64_t start = c->a.indptr[v], d = c->a.indptr[v + 1] - start;
      bptr[i] = (int32_t)o;
      int64_t m = choose_positions(c, v, d, fo, k, sel, keybuf);
      for (int64_t q = 0; q < m; q++) raw[o++] = c->a.indices[start + sel[q]];
    }
    bptr[nprev] = (int32_t)o;
    c->e[k - 1] = E;
    double tb = now_s();
    t_sample += tb - ta;

    /* dedup: new = ascending unique {u sampled : u not in F}; F <- F ++ new */
    free(uniq);
    uniq = (int32_t*)malloc(sizeof(int32_t) * (size_t)(E ? E : 1));
    if (!uniq) { rc = OR_ENOMEM; goto done; }
    memcpy(uniq, raw, sizeof(int32_t) * (size_t)E);
    qsort(uniq, (size_t)E, sizeof(int32_t), cmp_i32);
    if (grow_i32(&c->F, &c->nF_cap, nF + E + 1)) { rc = OR_ENOMEM; goto done; }
    for (int64_t q = 0; q < E; q++) {
      int32_t u = uniq[q];
      if (q > 0 && uniq[q - 1] == u) continue;
      if (c->pos[u] >= 0) continue;
      c->pos[u] = (int32_t)nF;
      c->F[nF++] = u;
    }
    c->n[k] = nF;
    /* relabel every sampled neighbour to its position in F */
    for (int64_t q = 0; q < E; q++) c->blk_indices[k - 1][q] = c->pos[raw[q]];
    t_dedup += now_s() - tb;
  }
  {
    double tc = now_s();
    const int64_t nK = nF;
    free(c->mask);
    free(c->feat);
    c->mask = (uint8_t*)malloc((size_t)(nK ? nK : 1));
    c->feat = (uint8_t*)malloc((size_t)(nK ? nK : 1) * (size_t)c->a.row_bytes);
    if (!c->mask || !c->feat) { rc = OR_ENOMEM; goto done; }
    /* V^{l|s}, V^{h|s}; Hits = V^{h|s} in BUF; Misses = V^{h|s} not in BUF */
    c->hits = c->misses = c->local = 0;
    for (int64_t i = 0; i < nK; i++) {
      int32_t v = c->F[i];
      if (v < L) { c->mask[i] = 0; c->local++; }
      else if (c->slot_of[v - L] >= 0) { c->mask[i] = 1; c->hits++; }
      else { c->mask[i] = 2; c->misses++; }
    }
    double td = now_s();
    /* Algorithm 2 decay: a buffered node that this step did not sample has
     * its S_E multiplied by gamma */
    for (int64_t s = 0; s < c->cap; s++) {
      int32_t h = c->slot_id[s];
      int sampled = c->pos[L + h] >= 0;
      if (!sampled) c->S_E[s] = c->S_E[s] * c->a.gamma;
    }
    /* Algorithm 2 scoring: each missed halo node gains one in S_A */
    for (int64_t i = 0; i < nK; i++)
      if (c->mask[i] == 2) {
        int32_t h = c->F[i] - L;
        c->S_A[h] = c->S_A[h] + 1.0f;
      }
    double te = now_s();
    /* B^l <- local features; B^h <- BUF[Hits]; B^h <- fetched Misses */
    const int64_t b = c->a.row_bytes;
    for (int64_t i = 0; i < nK; i++) {
      int32_t v = c->F[i];
      const uint8_t* src;
      if (c->mask[i] == 0) src = (const uint8_t*)c->a.local_feat + (size_t)v * b;
      else if (c->mask[i] == 1) src = c->buf + (size_t)c->slot_of[v - L] * b;
      else src = (const uint8_t*)c->a.halo_store + (size_t)(v - L) * b;
      memcpy(c->feat + (size_t)i * b, src, (size_t)b);
    }
    double tf = now_s();
    c->tphase[0] += t_sample;
    c->tphase[1] += t_dedup;
    c->tphase[2] += td - tc;
    c->tphase[3] += te - td;
    c->tphase[4] += tf - te;
    (void)t0;
  }
done:
  for (int64_t q = 0; q < nF; q++) c->pos[c->F[q]] = -1;
  free(sel); free(keybuf); free(raw); free(uniq);
  if (rc == OR_OK) {
    c->t += 1;
    c->pending_round = 1;
  }
  return rc;
}

/* candidate order: S_A desc, rank asc */
static const oracle_ctx* g_cand_ctx;
static int cmp_cand(const void* pa, const void* pb) {
  int32_t x = *(const int32_t*)pa, y = *(const int32_t*)pb;
  float sx = g_cand_ctx->S_A[x], sy = g_cand_ctx->S_A[y];
  if (sx != sy) return sx > sy ? -1 : 1;
  int32_t rx = g_cand_ctx->rank[x], ry = g_cand_ctx->rank[y];
  return rx < ry ? -1 : rx > ry;
}
/* eviction order when candidates run short: S_E asc, rank asc */
static int cmp_evict(const void* pa, const void* pb) {
  int32_t x = *(const int32_t*)pa, y = *(const int32_t*)pb;
  float ex = g_cand_ctx->S_E[x], ey = g_cand_ctx->S_E[y];
  if (ex != ey) return ex < ey ? -1 : 1;
  int32_t rx = g_cand_ctx->rank[g_cand_ctx->slot_id[x]], ry = g_cand_ctx->rank[g_cand_ctx->slot_id[y]];
  return rx < ry ? -1 : rx > ry;
}

/* The round for the step just sampled: runs iff that step t satisfies
 * t > 0 and t mod Delta == 0 (EVICT_AND_REPLACE + the buffer update of
 * Algorithm 2). Writes k' and, when the arrays are given, the evicted halo
 * nodes, the slots they held and their replacements. */
int oracle_evict_step(oracle_ctx* c, int32_t* evicted, int32_t* slots, int32_t* replaced, int64_t* k_out) {
  if (!c->pending_round) return OR_ESTATE;
  c->pending_round = 0;
  *k_out = 0;
  int64_t t = c->t - 1;
  if (!(t > 0 && t % c->a.delta == 0)) return OR_OK;
  double t0 = now_s();
  const int64_t H = c->a.H, cap = c->cap, b = c->a.row_bytes;
  /* V^{h|e}: slots with S_E < alpha, ascending */
  int32_t* E = (int32_t*)malloc(sizeof(int32_t) * (size_t)(cap ? cap : 1));
  int32_t* C = (int32_t*)malloc(sizeof(int32_t) * (size_t)(H ? H : 1));
  if (!E || !C) { free(E); free(C); return OR_ENOMEM; }
  int64_t nE = 0, nC = 0;
  for (int64_t s = 0; s < cap; s++)
    if (c->S_E[s] < c->alpha) E[nE++] = (int32_t)s;
  /* candidates m = max(S_A), repeatedly: the unbuffered halo nodes sorted */
  for (int64_t h = 0; h < H; h++)
    if (c->S_A[h] >= 0.0f) C[nC++] = (int32_t)h;
  g_cand_ctx = c;
  qsort(C, (size_t)nC, sizeof(int32_t), cmp_cand);
  int64_t kk = nE < nC ? nE : nC;
  if (kk < nE) {
    qsort(E, (size_t)nE, sizeof(int32_t), cmp_evict);
    qsort(E, (size_t)kk, sizeof(int32_t), cmp_i32);
  }
  /* swap scores and buffer entries, reading every old value first */
  float* oldSE = (float*)malloc(sizeof(float) * (size_t)(kk ? kk : 1));
  float* oldSA = (float*)malloc(sizeof(float) * (size_t)(kk ? kk : 1));
  if (!oldSE || !oldSA) { free(E); free(C); free(oldSE); free(oldSA); return OR_ENOMEM; }
  for (int64_t i = 0; i < kk; i++) {
    oldSE[i] = c->S_E[E[i]];
    oldSA[i] = c->S_A[C[i]];
  }
  for (int64_t i = 0; i < kk; i++) {
    int32_t s = E[i], e = c->slot_id[s], r = C[i];
    if (evicted) evicted[i] = e;
    if (slots) slots[i] = s;
    if (replaced) replaced[i] = r;
    c->S_A[e] = oldSE[i];            /* evicted node: S_A := last S_E */
    c->S_E[s] = oldSA[i];            /* replacement: S_E := last S_A */
    c->S_A[r] = -1.0f;               /* replacement is now buffered */
    c->slot_of[e] = -1;
    c->slot_id[s] = r;
    c->slot_of[r] = s;
    memcpy(c->buf + (size_t)s * b, (const uint8_t*)c->a.halo_store + (size_t)r * b, (size_t)b);
  }
  *k_out = kk;
  free(E); free(C); free(oldSE); free(oldSA);
  c->tphase[5] += now_s() - t0;
  return OR_OK;
}

/* The sampler's choice for one row, outside any context: the neighbour ids
 * chosen for node v at step t, hop k (1-based), written to out (room for
 * min(d, fanout)). Returns how many. Used to check single rows of large
 * runs. */
int64_t oracle_sample_row(const int64_t* indptr, const int32_t* indices, int32_t v, int64_t t, int32_t k,
                          int32_t fanout, uint64_t seed, int32_t* out) {
  oracle_ctx c;
  memset(&c, 0, sizeof c);
  c.a.seed = seed;
  c.t = t;
  int64_t start = indptr[v], d = indptr[v + 1] - start;
  int64_t* sel = (int64_t*)malloc(sizeof(int64_t) * (size_t)(d + 1));
  uint64_t* keybuf = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)(d + 1));
  if (!sel || !keybuf) { free(sel); free(keybuf); return -1; }
  int64_t m = choose_positions(&c, v, d, fanout, k, sel, keybuf);
  for (int64_t q = 0; q < m; q++) out[q] = indices[start + sel[q]];
  free(sel);
  free(keybuf);
  return m;
}

/* ---------------------------------------------------------------- access */
int64_t oracle_cap(const oracle_ctx* c) { return c->cap; }
float oracle_alpha(const oracle_ctx* c) { return c->alpha; }
int64_t oracle_t(const oracle_ctx* c) { return c->t; }
void oracle_sizes(const oracle_ctx* c, int64_t* n, int64_t* e, int64_t* counts) {
  for (int k = 0; k <= c->a.K; k++) n[k] = c->n[k];
  for (int k = 0; k < c->a.K; k++) e[k] = c->e[k];
  counts[0] = c->local; counts[1] = c->hits; counts[2] = c->misses;
}
const int32_t* oracle_nodes(const oracle_ctx* c) { return c->F; }
const int32_t* oracle_block_indptr(const oracle_ctx* c, int k) { return c->blk_indptr[k]; }
const int32_t* oracle_block_indices(const oracle_ctx* c, int k) { return c->blk_indices[k]; }
const uint8_t* oracle_mask(const oracle_ctx* c) { return c->mask; }
const uint8_t* oracle_feat(const oracle_ctx* c) { return c->feat; }
const int32_t* oracle_rank(const oracle_ctx* c) { return c->rank; }
void oracle_get_state(const oracle_ctx* c, int32_t* slot_id, float* S_E, float* S_A) {
  if (slot_id) memcpy(slot_id, c->slot_id, sizeof(int32_t) * (size_t)c->cap);
  if (S_E) memcpy(S_E, c->S_E, sizeof(float) * (size_t)c->cap);
  if (S_A) memcpy(S_A, c->S_A, sizeof(float) * (size_t)c->a.H);
}
const uint8_t* oracle_buffer_rows(const oracle_ctx* c) { return c->buf; }
void oracle_phase_times(const oracle_ctx* c, double* out6) { memcpy(out6, c->tphase, sizeof(c->tphase)); }
