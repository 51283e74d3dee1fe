// sample_kernels.hpp - fanout sampling, frontier dedup and relabel (one hop
// of the NeighborSampler of Algorithm 2, DGL block convention).
#pragma once

#include "common.hpp"

namespace ms {

constexpr int kScanNT = 1024;       // threads per scan block
constexpr int kScanItems = 4;       // items per thread
constexpr int kScanTile = kScanNT * kScanItems;

__device__ __forceinline__ int64_t size_of(const int64_t* p, int64_t c) { return p ? *p : c; }

// Sum of partials[0..b) computed by the whole block (b is at most a few
// thousand): the exclusive prefix of block b without a separate scan kernel.
template <int NT>
__device__ __forceinline__ int32_t preceding_sum(const int32_t* __restrict__ partials, int64_t b, int32_t* lds) {
  int32_t s = 0;
  for (int64_t i = threadIdx.x; i < b; i += NT) s += partials[i];
  return block_sum<NT>(s, lds);
}

// Single-pass scan by decoupled look-back: tile b publishes its aggregate,
// then its inclusive prefix once the tiles before it are known. flags[b] =
// tag << 32 | value, tag = 2 * epoch (aggregate) or 2 * epoch + 1 (inclusive
// prefix); the epoch differs for every launch, so flags are never cleared.
// Tiles are blocks in blockIdx order. Each XCD dispatches its blocks in
// order, so the lowest unfinished tile is always resident and every wait
// ends. The wait is bounded all the same: past the limit the step is flagged
// (status bit 8) and the tile goes on with the values it has.
constexpr int kLookbackSpins = 1 << 20;

__device__ __forceinline__ uint32_t lookback_exclusive(uint64_t* flags, int64_t b, uint32_t agg, uint32_t epoch,
                                                       int32_t* status, uint32_t* excl_lds) {
  const uint32_t t_agg = 2u * epoch, t_inc = 2u * epoch + 1u;
  if (wave_id() == 0) {
    const int lane = lane_id();
    if (lane == 0)
      __hip_atomic_store(&flags[b], ((uint64_t)(b == 0 ? t_inc : t_agg) << 32) | agg, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    uint32_t excl = 0;
    int64_t p = b - 1;  // the window is tiles p - 63 .. p, lane l on tile p - l
    int spins = 0;
    while (p >= 0) {
      const int64_t i = p - lane;
      // before tile 0: an inclusive prefix of zero
      const uint64_t f = i >= 0 ? __hip_atomic_load(&flags[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                                : ((uint64_t)t_inc << 32);
      const uint32_t tag = (uint32_t)(f >> 32);
      const uint64_t ready = ballot(tag == t_agg || tag == t_inc);
      const uint64_t inc = ballot(tag == t_inc);
      // lanes 0..k must be ready, k = the nearest inclusive prefix (or the window)
      const int k = inc ? __ffsll((unsigned long long)inc) - 1 : MS_WAVE - 1;
      const uint64_t need = k == MS_WAVE - 1 ? ~0ull : ((2ull << k) - 1);
      if ((ready & need) == need) {
        excl += wave_sum(lane <= k ? (uint32_t)f : 0u);
        if (inc) break;
        p -= MS_WAVE;
        continue;
      }
      if (++spins > kLookbackSpins) {
        if (lane == 0) atomicOr(status, 8);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    if (lane == 0) {
      if (b > 0)
        __hip_atomic_store(&flags[b], ((uint64_t)t_inc << 32) | (excl + agg), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      *excl_lds = excl;
    }
  }
  __syncthreads();
  return *excl_lds;
}

// ------------------------------------------------------ per-row counts + scan
// Block b < nbk: the rows of tile b get min(deg(F[i]), fo) positions; the
// tile's exclusive prefix comes from the single-pass scan, and bptr[0..n]
// gets the offsets. Rows longer than big_min go to the front of big_rows (one
// global atomic per block). With small_end > 0 the other rows go to its back,
// the r-th listed one at big_rows[small_end - 1 - r]: with n <= small_end
// rows the two parts never meet, and the one-wave-per-row sampler then finds
// a row for each of its first n waves. Every load of a thread is issued
// before the first is used.
// Blocks b >= nbk relabel the previous hop's sampled ids (rel_ids, if given):
// that work depends on the same kernels and shares the launch.
// For hop 1 (seeds given) the rows are the seed batch: the launch also checks
// each seed (a local id, not repeated: the first to mark pos_of keeps it) and
// places it, F_0 = seeds, pos_of[seed] = its position, n_0 = n0; a bad seed
// sets the step's status, which every later kernel checks first.
__device__ __forceinline__ void relabel_tiles(int32_t* __restrict__ ids, int64_t e, const int32_t* __restrict__ pos_of,
                                              int64_t b, int64_t nblocks) {
  for (int64_t b0 = b * kScanTile; b0 < e; b0 += nblocks * kScanTile) {
    int32_t u[kScanItems], p[kScanItems];
    // lanes past the end read the last id (or its new value, also a valid
    // index) and store nothing
#pragma unroll
    for (int it = 0; it < kScanItems; ++it) {
      const int64_t i = b0 + (int64_t)it * kScanNT + threadIdx.x;
      u[it] = ids[i < e ? i : e - 1];
    }
#pragma unroll
    for (int it = 0; it < kScanItems; ++it) pin(u[it]);
#pragma unroll
    for (int it = 0; it < kScanItems; ++it) p[it] = pos_of[u[it]];
#pragma unroll
    for (int it = 0; it < kScanItems; ++it) pin(p[it]);
#pragma unroll
    for (int it = 0; it < kScanItems; ++it) {
      const int64_t i = b0 + (int64_t)it * kScanNT + threadIdx.x;
      if (i < e) ids[i] = p[it];
    }
  }
}

__global__ __launch_bounds__(kScanNT) void k_row_scan(const int64_t* __restrict__ csr_indptr,
                                                      int32_t* __restrict__ nodes, StepSizes* sz, int hop,
                                                      int32_t fo, int32_t* __restrict__ bptr, uint64_t* flags,
                                                      uint32_t epoch, int32_t* __restrict__ big_rows,
                                                      int64_t big_min, int64_t nbk, int32_t* __restrict__ rel_ids,
                                                      int32_t* __restrict__ pos_of, int64_t small_end,
                                                      const int32_t* __restrict__ seeds, int32_t n0, int32_t L) {
  __shared__ int32_t lds[kScanNT / MS_WAVE + 1];
  __shared__ int32_t big_lds[kScanTile];  // long rows from the front, the others from the back
  __shared__ int32_t big_n, small_n;
  __shared__ unsigned long long big_base, small_base;
  __shared__ uint32_t excl_lds;
  if (sz->status) return;
  if ((int64_t)blockIdx.x >= nbk) {
    if (rel_ids) relabel_tiles(rel_ids, sz->e[hop - 2], pos_of, blockIdx.x - nbk, gridDim.x - nbk);
    return;
  }
  // hop 1 with seeds: the rows are the seeds, which this launch checks and
  // places (F_0 = seeds, pos_of[seed] = its position; an out-of-range or
  // repeated seed flags the step, which every later kernel then abandons)
  const int64_t n = seeds ? (int64_t)n0 : sz->n[hop - 1];
  if (seeds && blockIdx.x == 0 && threadIdx.x == 0) sz->n[0] = n0;
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  if (threadIdx.x == 0) big_n = small_n = 0;
  __syncthreads();
  int32_t c[kScanItems] = {};
  int32_t s = 0;
  if ((int64_t)blockIdx.x * kScanTile < n) {
    int32_t v[kScanItems];
    int64_t lo[kScanItems], hi[kScanItems];
#pragma unroll
    for (int it = 0; it < kScanItems; ++it) v[it] = (seeds ? seeds : nodes)[base + it < n ? base + it : n - 1];
#pragma unroll
    for (int it = 0; it < kScanItems; ++it) pin(v[it]);
    if (seeds) {
#pragma unroll
      for (int it = 0; it < kScanItems; ++it) {
        const int64_t i = base + it;
        const int32_t x = v[it];
        const bool ok = x >= 0 && x < L;
        if (i < n) {
          if (!ok) {
            atomicOr(&sz->status, 1);
          } else {
            if (atomicCAS(&pos_of[x], -1, (int32_t)i) != -1) atomicOr(&sz->status, 2);
            nodes[i] = x;
          }
        }
        v[it] = ok ? x : 0;  // an in-range row for the loads below (the step is abandoned anyway)
      }
    }
#pragma unroll
    for (int it = 0; it < kScanItems; ++it) {
      lo[it] = csr_indptr[v[it]];
      hi[it] = csr_indptr[v[it] + 1];
    }
#pragma unroll
    for (int it = 0; it < kScanItems; ++it) {
      pin(lo[it]);
      pin(hi[it]);
    }
#pragma unroll
    for (int it = 0; it < kScanItems; ++it) {
      const int64_t i = base + it;
      if (i < n) {
        const int64_t d = hi[it] - lo[it];
        c[it] = d < fo ? (int32_t)d : fo;
        s += c[it];
        if (d > big_min)
          big_lds[atomicAdd(&big_n, 1)] = (int32_t)i;
        else if (small_end)
          big_lds[kScanTile - 1 - atomicAdd(&small_n, 1)] = (int32_t)i;
      }
    }
  }
  int32_t tot;
  const int32_t ex = block_exclusive_scan<kScanNT>(s, lds, &tot);  // (its barriers complete the big_lds appends)
  const uint32_t before = lookback_exclusive(flags, blockIdx.x, (uint32_t)tot, epoch, &sz->status, &excl_lds);
  int64_t run = (int64_t)before + ex;
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t i = base + it;
    if (i < n) {
      run += c[it];
      bptr[i + 1] = (int32_t)run;
    }
  }
  if (threadIdx.x == 0) {
    if (blockIdx.x == 0) {
      bptr[0] = 0;
      sz->n[hop] = n;  // new nodes are added by k_bits_scan
    }
    if ((int64_t)blockIdx.x == nbk - 1) sz->e[hop - 1] = (int64_t)before + tot;
    big_base = big_n ? atomicAdd((unsigned long long*)&sz->n_big[hop - 1], (unsigned long long)big_n) : 0ull;
    small_base = small_n ? atomicAdd((unsigned long long*)&sz->n_small[hop - 1], (unsigned long long)small_n) : 0ull;
  }
  __syncthreads();
  for (int j = threadIdx.x; j < big_n; j += kScanNT) big_rows[big_base + j] = big_lds[j];
  for (int j = threadIdx.x; j < small_n; j += kScanNT)
    big_rows[small_end - 1 - (int64_t)(small_base + j)] = big_lds[kScanTile - 1 - j];
}

// Exclusive scan of partials[0..nb) in place (one block). Writes the total
// to *total_out (if given) as int64, plus `add`.
__global__ __launch_bounds__(kScanNT) void k_scan_partials(int32_t* __restrict__ partials, int64_t nb,
                                                           int64_t* total_out, const int64_t* add) {
  __shared__ int32_t lds[kScanNT / MS_WAVE + 1];
  int32_t carry = 0;
  for (int64_t b0 = 0; b0 < nb; b0 += (int64_t)kScanNT * kScanItems) {
    int32_t v[kScanItems];
    int32_t s = 0;
#pragma unroll
    for (int it = 0; it < kScanItems; ++it) {
      const int64_t i = b0 + (int64_t)threadIdx.x * kScanItems + it;
      v[it] = i < nb ? partials[i] : 0;
      s += v[it];
    }
    int32_t tot;
    int32_t ex = block_exclusive_scan<kScanNT>(s, lds, &tot) + carry;
#pragma unroll
    for (int it = 0; it < kScanItems; ++it) {
      const int64_t i = b0 + (int64_t)threadIdx.x * kScanItems + it;
      if (i < nb) partials[i] = ex;
      ex += v[it];
    }
    carry += tot;
  }
  if (threadIdx.x == 0 && total_out) *total_out = (int64_t)carry + (add ? *add : 0);
}

// --------------------------------------------------------------- sampler
// One wavefront per frontier node. Rows with d <= fanout are copied. For
// longer rows the choice is the fanout positions of smallest (key, j),
// found in two stages:
//   1. a threshold pass draws every key (lane q of an iteration draws one
//      Philox block = keys of positions 4q..4q+3) and keeps, in ascending j,
//      the (key, j) pairs with key < tau; tau is set so that about
//      fanout + 3*sqrt(fanout) + 3 keys survive, and is bisected if fewer than
//      fanout or more than the list capacity survive (rare);
//   2. a bitwise search over ballots finds the fanout-th smallest surviving
//      key T (it starts below tau's top bit), ties at T are taken in list
//      order (= ascending j), and the chosen positions are written in
//      ascending j.
// The chosen ids not yet in the frontier are marked in the new-node bitmap
// as they are written. Rows longer than big_min (listed by k_row_scan) are
// taken first. Where the frontier is small, so that its few longest rows bound
// the hop's time, each of them gets a whole block: its waves filter
// consecutive quarters of the row with the same tau, and the four candidate
// lists, concatenated in order, are the row's list in ascending j. Otherwise
// (many rows keep the chip busy) each gets one wave, ahead of the shorter
// rows. Other rows get one wave each.
constexpr int kSampleWaves = 4;  // k_sample_blocks: waves per block (a long row's quarters)
constexpr int kRowWaves = 2;     // k_sample_waves: waves per workgroup (one row each)
constexpr int kCandSlots = 5;                   // candidates per lane in the selection
constexpr int kCandCap = kCandSlots * MS_WAVE;  // candidates per wave (LDS): 320, so the
                                                // largest fanout (256) keeps 64 of slack for ties
constexpr int64_t kBigRow = 2048;
constexpr int64_t kBigBlocks = 2048;  // blocks that walk the big list (8 per CU)
constexpr int64_t kBlockRowsMax = 65536;  // frontiers up to this size sample long rows by blocks
constexpr int kTauIters = 64;         // threshold passes: x4 growth (<= 16) then bisection (<= 33)

struct SampleArgs {
  const int64_t* csr_indptr;
  const int32_t* csr_indices;
  const int32_t* nodes;
  StepSizes* sz;
  const int32_t* bptr;
  int32_t* out;
  int32_t hop;  // 1-based
  int32_t fo;
  uint32_t t;
  uint32_t key0, key1;
  double mu32;              // (fo + 3 sqrt(fo) + 3) * 2^32
  int64_t big_min;          // rows longer than this are listed in big_rows
  const int32_t* big_rows;  // appended by k_row_scan
  int64_t row_waves;        // k_sample_waves: small_end of k_row_scan (the other rows' list ends there)
  int64_t big_blocks;       // k_sample_blocks: blocks [0, big_blocks) walk the big list, one row per
                            // block; the rest take all other rows, one per wave
  const int32_t* pos_of;    // frontier position of an id, or -1
  uint32_t* bits;           // new-node bitmap
  int32_t* err;             // threshold search could not isolate a candidate set
  int32_t tau_iters;        // threshold passes allowed per row (kTauIters)
};

// Philox4x32-10 with counter (q, v, t, hop) for every q of one row. Words 1-3
// of the counter are the same across the row, so round 1's product of word 2
// (t) and round 2's product of word 0 (which round 1 builds from t, v and the
// key only) are computed once per row; the other rounds are the published
// block function unchanged (see philox4x32_10).
struct PhiloxRow {
  uint32_t x1, y1;      // words 0 and 1 after round 1
  uint32_t a2hi, a2lo;  // round 2's 64-bit product of word 0
  uint32_t hop, k0, k1;
  __device__ __forceinline__ PhiloxRow(uint32_t v, uint32_t t, uint32_t hop_, uint32_t key0, uint32_t key1)
      : hop(hop_), k0(key0), k1(key1) {
    const uint64_t b1 = (uint64_t)0xCD9E8D57u * t;
    x1 = (uint32_t)(b1 >> 32) ^ v ^ key0;
    y1 = (uint32_t)b1;
    const uint64_t a2 = (uint64_t)0xD2511F53u * x1;
    a2hi = (uint32_t)(a2 >> 32);
    a2lo = (uint32_t)a2;
  }
  // the block of counter q, given round 1's product of word 0, a1 = M0 * q
  // (a lane's consecutive iterations add M0 * 64 to it instead of
  // multiplying again)
  __device__ __forceinline__ uint4 from_a1(uint64_t a1) const {
    const uint32_t z1 = (uint32_t)(a1 >> 32) ^ hop ^ k1, w1 = (uint32_t)a1;
    uint32_t r0 = k0 + 0x9E3779B9u, r1 = k1 + 0xBB67AE85u;  // round 2's key
    const uint64_t b2 = (uint64_t)0xCD9E8D57u * z1;
    uint4 c = make_uint4((uint32_t)(b2 >> 32) ^ y1 ^ r0, (uint32_t)b2, a2hi ^ w1 ^ r1, a2lo);
#pragma unroll
    for (int r = 2; r < 10; ++r) {
      r0 += 0x9E3779B9u;
      r1 += 0xBB67AE85u;
      const uint64_t a = (uint64_t)0xD2511F53u * c.x;
      const uint64_t b = (uint64_t)0xCD9E8D57u * c.z;
      c = make_uint4(xor3_key((uint32_t)(b >> 32), c.y, r0), (uint32_t)b, xor3_key((uint32_t)(a >> 32), c.w, r1),
                     (uint32_t)a);
    }
    return c;
  }
};

__device__ __forceinline__ uint64_t first_tau(double mu32, int64_t d) {
  const double t = mu32 / (double)d + 1.0;
  return t >= 4294967296.0 ? (1ull << 32) : (uint64_t)t;
}

// Threshold bookkeeping: returns true when the count is acceptable, else
// moves tau (bisection once both sides are known).
struct TauSearch {
  uint64_t lo = 0, hi = (1ull << 32) + 1, tau;
  __device__ bool step(int cnt, int fo, int cap, bool* fail) {
    const uint64_t full = 1ull << 32;
    if (cnt >= fo && cnt <= cap) return true;
    if (cnt < fo) {
      lo = tau;
      tau = (hi > full) ? (tau * 4 > full ? full : tau * 4) : (lo + hi) / 2;
    } else {
      hi = tau;
      tau = (lo + hi) / 2;
    }
    if (hi <= full && hi - lo <= 1) *fail = true;
    return false;
  }
};

__device__ __forceinline__ void emit_id(int32_t* __restrict__ out, int p, int32_t u, const int32_t* __restrict__ pos_of,
                                        uint32_t* __restrict__ bits) {
  out[p] = u;
  // a no-return atomic OR, with no read of the word first: a read would put a
  // second dependent load on the row's last steps (hop 3: 181 against 184 us)
  if (pos_of[u] < 0) atomicOr(&bits[u >> 5], 1u << (u & 31));
}

// Selection among cnt <= kCandCap candidates held in LDS in ascending j
// (list[i] = key << 32 | j); writes the fo chosen neighbours to out in
// ascending j. One wavefront; element i sits in slot i / 64 of lane i % 64.
__device__ __forceinline__ void select_emit(const uint64_t* list, int cnt, int fo, uint64_t tau,
                                            const int32_t* __restrict__ nb, int32_t* __restrict__ out,
                                            const int32_t* __restrict__ pos_of, uint32_t* __restrict__ bits) {
  const int lane = lane_id();
  const int S = (cnt + MS_WAVE - 1) / MS_WAVE;  // 1..kCandSlots
  uint32_t key[kCandSlots], pos[kCandSlots];
  bool valid[kCandSlots];
#pragma unroll
  for (int s = 0; s < kCandSlots; ++s) {
    const int idx = s * MS_WAVE + lane;
    valid[s] = s < S && idx < cnt;
    const uint64_t e = valid[s] ? list[idx] : 0ull;
    key[s] = (uint32_t)(e >> 32);
    pos[s] = (uint32_t)e;
  }
  // T = largest x with count(key < x) < fo; every key is below tau
  uint32_t T = 0;
  const uint64_t tm1 = tau - 1;
  const int top = tm1 == 0 ? 0 : 63 - __clzll(tm1);
  for (int b = top; b >= 0; --b) {
    const uint32_t trial = T | (1u << b);
    int c = __popcll(ballot(valid[0] && key[0] < trial));
    // unrolled with static indices (a loop to S would index the arrays
    // dynamically); S is the same in every lane
#pragma unroll
    for (int s = 1; s < kCandSlots; ++s)
      if (s < S) c += __popcll(ballot(valid[s] && key[s] < trial));
    if (c < fo) T = trial;
  }
  int n_lt = 0;
  uint64_t lt[kCandSlots], eq[kCandSlots];
#pragma unroll
  for (int s = 0; s < kCandSlots; ++s) {
    lt[s] = ballot(valid[s] && key[s] < T);
    eq[s] = ballot(valid[s] && key[s] == T);
    n_lt += __popcll(lt[s]);
  }
  const int need = fo - n_lt;
  int eq_before = 0;  // ties in earlier slots (all lanes)
  int p_before = 0;   // selected in earlier slots
#pragma unroll
  for (int s = 0; s < kCandSlots; ++s) {
    const bool is_lt = (lt[s] >> lane) & 1ull, is_eq = (eq[s] >> lane) & 1ull;
    const bool sel = is_lt || (is_eq && eq_before + lanes_below(eq[s]) < need);
    const uint64_t sm = ballot(sel);
    if (sel) emit_id(out, p_before + lanes_below(sm), nb[pos[s]], pos_of, bits);
    p_before += __popcll(sm);
    eq_before += __popcll(eq[s]);
  }
}

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Appends to c (at cnt, in ascending j) the candidates (key << 32 | j) among
// the four keys of block q = q0 + lane whose key is <= tm1, stopping at
// kCandCap entries but counting them all. Every lane's four positions exist;
// mn is the smallest of the lane's four keys.
// A row's ~fanout + 3 sqrt(fanout) + 3 candidates are spread over its
// iterations, so an iteration with a candidate usually has one, or a few in
// different lanes: when no lane has two, a lane's candidate is its smallest
// key and its list index the running count plus the candidate lanes below it.
__device__ __forceinline__ void take_block(uint4 k4, uint32_t mn, uint32_t q, uint32_t tm1, uint64_t* c, int& cnt) {
  pin(k4.x);
  pin(k4.y);
  pin(k4.z);
  pin(k4.w);
  const uint64_t m0 = ballot(k4.x <= tm1), m1 = ballot(k4.y <= tm1), m2 = ballot(k4.z <= tm1),
                 m3 = ballot(k4.w <= tm1);
  const uint64_t any = m0 | m1 | m2 | m3;
  if (!any) return;
  const uint64_t bit = 1ull << lane_id();
  const int n_any = __popcll(any);
  if (__popcll(m0) + __popcll(m1) + __popcll(m2) + __popcll(m3) == n_any) {  // one per candidate lane
    if (any & bit) {
      const uint32_t s = (m0 & bit) ? 0u : (m1 & bit) ? 1u : (m2 & bit) ? 2u : 3u;
      const int p = cnt + lanes_below(any);
      if (p < kCandCap) c[p] = ((uint64_t)mn << 32) | (4 * q + s);
    }
    cnt += n_any;
    return;
  }
  // lower lanes first, then s within the lane
  int p = cnt + lanes_below(m0) + lanes_below(m1) + lanes_below(m2) + lanes_below(m3);
  const uint64_t m[4] = {m0, m1, m2, m3};
#pragma unroll
  for (int s = 0; s < 4; ++s)
    if (m[s] & bit) {
      if (p < kCandCap) c[p] = ((uint64_t)word_of(k4, s) << 32) | (4 * q + s);
      ++p;
    }
  cnt += __popcll(m0) + __popcll(m1) + __popcll(m2) + __popcll(m3);
}

__device__ __forceinline__ uint32_t min4(const uint4& w) { return min(min(w.x, w.y), min(w.z, w.w)); }

// Filters 4-position groups [g0, g1) of a row of d positions: appends to c, in
// ascending j, the candidates (key << 32 | j) whose key is <= tm1 (below tau),
// stopping at kCandCap entries but counting them all. One wavefront.
// The usual iteration of a long row has no key below tau, which one test on
// the smallest of each lane's four keys settles. (Two or four Philox blocks
// per lane in flight were measured slower: the loop is bound by VALU issue,
// not by the latency of its dependent multiplies.)
__device__ __forceinline__ int filter_groups(const PhiloxRow& ph, uint32_t g0, uint32_t g1, uint32_t d32,
                                             uint32_t tm1, uint64_t* c) {
  const int lane = lane_id();
  int cnt = 0;
  const uint32_t gf = min(g1, d32 / 4);  // groups below gf are whole
  uint64_t a1 = (uint64_t)0xD2511F53u * (g0 + lane);
  for (uint32_t q0 = g0; q0 < g1; q0 += MS_WAVE, a1 += (uint64_t)0xD2511F53u * MS_WAVE) {
    const uint32_t q = q0 + lane;
    const uint4 wv = ph.from_a1(a1);
    if (q0 + MS_WAVE <= gf) {  // every position of this iteration exists
      const uint32_t mn = min4(wv);
      if (!ballot(mn <= tm1)) continue;
      take_block(wv, mn, q, tm1, c, cnt);
      continue;
    }
    const bool in = q < g1;
    const uint64_t m0 = ballot(in && 4 * q < d32 && wv.x <= tm1);
    const uint64_t m1 = ballot(in && 4 * q + 1 < d32 && wv.y <= tm1);
    const uint64_t m2 = ballot(in && 4 * q + 2 < d32 && wv.z <= tm1);
    const uint64_t m3 = ballot(in && 4 * q + 3 < d32 && wv.w <= tm1);
    if (!(m0 | m1 | m2 | m3)) continue;
    int p = cnt + lanes_below(m0) + lanes_below(m1) + lanes_below(m2) + lanes_below(m3);
    const uint64_t bit = 1ull << lane;
    const uint64_t m[4] = {m0, m1, m2, m3};
#pragma unroll
    for (int s = 0; s < 4; ++s)
      if (m[s] & bit) {
        if (p < kCandCap) c[p] = ((uint64_t)word_of(wv, s) << 32) | (4 * q + s);
        ++p;
      }
    cnt += __popcll(m0) + __popcll(m1) + __popcll(m2) + __popcll(m3);
  }
  return cnt;
}

// Large frontiers (many rows keep the chip busy): every row one per wave, the
// long ones (waves [0, n_big), the front of the row list) dispatched first,
// then the others (waves [n_big, n), its back); waves from n on find no row.
// Workgroups of two waves: a workgroup holds its LDS until its last wave
// ends, and rows of a power-law frontier end at very different times, so
// smaller workgroups keep more waves resident (hop 3 on the papers-sized
// share: 212 us with four waves per workgroup, 199 us with two).
__global__ __launch_bounds__(kRowWaves* MS_WAVE) void k_sample_waves(SampleArgs a) {
  __shared__ uint64_t cand[kRowWaves][kCandCap];
  if (a.sz->status) return;
  const int lane = lane_id(), wave = wave_uniform(wave_id());
  const int64_t w = (int64_t)blockIdx.x * kRowWaves + wave;
  const int64_t nbig = a.sz->n_big[a.hop - 1];
  if (w >= a.sz->n[a.hop - 1]) return;
  const int64_t row = wave_uniform((int32_t)a.big_rows[w < nbig ? w : a.row_waves - 1 - (w - nbig)]);
  // the row, its node and its extent are the same in every lane
  const int32_t v = wave_uniform(a.nodes[row]);
  const int64_t start = wave_uniform(a.csr_indptr[v]);
  const int64_t d = wave_uniform(a.csr_indptr[v + 1]) - start;
  const int32_t fo = a.fo;
  int32_t* out = a.out + a.bptr[row];
  const int32_t* nb = a.csr_indices + start;
  if (d <= fo) {
    for (int64_t j = lane; j < d; j += MS_WAVE) emit_id(out, (int)j, nb[j], a.pos_of, a.bits);
    return;
  }
  uint64_t* c = cand[wave];
  TauSearch ts;
  ts.tau = first_tau(a.mu32, d);
  int cnt = 0;
  bool fail = false, ok = false;
  const uint32_t d32 = (uint32_t)d;  // a row is shorter than 2^31
  const PhiloxRow ph((uint32_t)v, a.t, (uint32_t)a.hop, a.key0, a.key1);
  for (int iter = 0; iter < a.tau_iters && !fail; ++iter) {
    cnt = filter_groups(ph, 0, (d32 + 3) / 4, d32, (uint32_t)(ts.tau - 1), c);
    if (ts.step(cnt, fo, kCandCap, &fail)) {
      ok = true;
      break;
    }
  }
  if (!ok) {
    if (lane == 0) atomicOr(a.err, 4);
    return;
  }
  wave_lds_sync();
  select_emit(c, cnt, fo, ts.tau, nb, out, a.pos_of, a.bits);
}

// One row by one wavefront (skipped if it is longer than skip_above).
__device__ __forceinline__ void sample_row_wave(const SampleArgs& a, int64_t row, uint64_t* c,
                                                int64_t skip_above = INT64_MAX) {
  const int lane = lane_id();
  const int32_t fo = a.fo;
  // the row, its node and its extent are the same in every lane
  const int32_t v = wave_uniform(a.nodes[row]);
  const int64_t start = wave_uniform(a.csr_indptr[v]);
  const int64_t d = wave_uniform(a.csr_indptr[v + 1]) - start;
  if (d > skip_above) return;
  int32_t* out = a.out + a.bptr[row];
  const int32_t* nb = a.csr_indices + start;
  if (d <= fo) {
    for (int64_t j = lane; j < d; j += MS_WAVE) emit_id(out, (int)j, nb[j], a.pos_of, a.bits);
    return;
  }
  TauSearch ts;
  ts.tau = first_tau(a.mu32, d);
  int cnt = 0;
  bool fail = false, ok = false;
  const uint32_t d32 = (uint32_t)d;  // a row is shorter than 2^31
  const PhiloxRow ph((uint32_t)v, a.t, (uint32_t)a.hop, a.key0, a.key1);
  for (int iter = 0; iter < a.tau_iters && !ok && !fail; ++iter) {
    cnt = filter_groups(ph, 0, (d32 + 3) / 4, d32, (uint32_t)(ts.tau - 1), c);
    ok = ts.step(cnt, fo, kCandCap, &fail);
  }
  if (!ok) {
    if (lane == 0) atomicOr(a.err, 4);
    return;
  }
  wave_lds_sync();
  select_emit(c, cnt, fo, ts.tau, nb, out, a.pos_of, a.bits);
  // (a wave samples one row: no fence at the end, which would hold the wave
  // until its stores and bitmap atomics have completed)
}

// Small frontiers: the long rows one per block, the blocks walking the big
// list; every other row one per wave.
__global__ __launch_bounds__(kSampleWaves* MS_WAVE) void k_sample_blocks(SampleArgs a) {
  __shared__ uint64_t cand[kSampleWaves][kCandCap];
  if (a.sz->status) return;
  const int lane = lane_id(), wave = wave_uniform(wave_id());
  const int32_t fo = a.fo;
  if ((int64_t)blockIdx.x < a.big_blocks) {
    __shared__ uint64_t merged[kCandCap];
    __shared__ int counts[kSampleWaves];
    // long rows, one per block at a time
    const int64_t n_big = a.sz->n_big[a.hop - 1];
    for (int64_t b = blockIdx.x; b < n_big; b += a.big_blocks) {
      const int64_t row = wave_uniform((int32_t)a.big_rows[b]);
      const int32_t v = wave_uniform(a.nodes[row]);
      const int64_t start = wave_uniform(a.csr_indptr[v]);
      const int64_t d = wave_uniform(a.csr_indptr[v + 1]) - start;  // > big_min >= fo
      int32_t* out = a.out + a.bptr[row];
      const int32_t* nb = a.csr_indices + start;
      const uint32_t d32 = (uint32_t)d;
      const PhiloxRow ph((uint32_t)v, a.t, (uint32_t)a.hop, a.key0, a.key1);
      // this wave's quarter of the row's groups, in whole wave iterations
      const uint32_t groups = (d32 + 3) / 4;
      const uint32_t per = (groups + kSampleWaves * MS_WAVE - 1) / (kSampleWaves * MS_WAVE) * MS_WAVE;
      const uint32_t g0 = min(groups, (uint32_t)wave * per), g1 = min(groups, g0 + per);
      TauSearch ts;
      ts.tau = first_tau(a.mu32, d);
      int total = 0;
      bool fail = false, ok = false;
      for (int iter = 0; iter < a.tau_iters; ++iter) {
        const int cnt = filter_groups(ph, g0, g1, d32, (uint32_t)(ts.tau - 1), cand[wave]);
        if (lane == 0) counts[wave] = cnt;
        __syncthreads();
        total = 0;
        for (int x = 0; x < kSampleWaves; ++x) total += counts[x];
        // every wave takes the same decision from the same total
        ok = ts.step(total, fo, kCandCap, &fail);
        if (ok || fail) break;
        __syncthreads();  // the next pass rewrites cand and counts
      }
      if (!ok) {
        if (threadIdx.x == 0) atomicOr(a.err, 4);
        return;  // every wave of the block leaves together
      }
      // the four lists, in order, are the row's candidates in ascending j
      int before = 0;
      for (int x = 0; x < wave; ++x) before += counts[x];
      for (int i = lane; i < counts[wave]; i += MS_WAVE) merged[before + i] = cand[wave][i];
      __syncthreads();
      if (wave == 0) select_emit(merged, total, fo, ts.tau, nb, out, a.pos_of, a.bits);
      if (b + a.big_blocks < n_big) __syncthreads();  // merged and counts are reused for the next row
    }
    return;
  }
  const int64_t row = (int64_t)(blockIdx.x - a.big_blocks) * kSampleWaves + wave;
  if (row >= a.sz->n[a.hop - 1]) return;
  // rows longer than big_min are taken by the big list
  sample_row_wave(a, row, cand[wave], a.big_min);
}

// ------------------------------------------------------------ dedup/relabel
// New nodes in ascending id: F[n_{k-1} + rank] = u, pos_of[u] = that
// position, with the rank from the single-pass scan of the bitmap's
// popcounts; the bitmap is cleared for the next hop. The last tile writes
// n_k. The new nodes below L (local ids) are the prefix at id L: the thread
// whose words hold id L writes that count (the last tile, if every id is
// below L). (bits holds W + 4 words, the last four always zero.)
__global__ __launch_bounds__(kScanNT) void k_bits_scan(uint32_t* __restrict__ bits, int64_t W, int32_t L,
                                                       StepSizes* sz, int hop, uint64_t* flags, uint32_t epoch,
                                                       int32_t* __restrict__ nodes, int32_t* __restrict__ pos_of) {
  __shared__ int32_t lds[kScanNT / MS_WAVE + 1];
  __shared__ uint32_t excl_lds;
  if (sz->status) return;
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  uint4 w4 = make_uint4(0u, 0u, 0u, 0u);
  if (base < W) w4 = *reinterpret_cast<const uint4*>(bits + base);
  const uint32_t w[kScanItems] = {w4.x, w4.y, w4.z, w4.w};
  const int32_t s = __popc(w[0]) + __popc(w[1]) + __popc(w[2]) + __popc(w[3]);
  int32_t tot;
  const int32_t ex = block_exclusive_scan<kScanNT>(s, lds, &tot);
  const uint32_t before = lookback_exclusive(flags, blockIdx.x, (uint32_t)tot, epoch, &sz->status, &excl_lds);
  const int64_t n_prev = sz->n[hop - 1];
  const int64_t wL = (int64_t)(L >> 5);
  if (wL < W && wL >= base && wL < base + kScanItems) {
    int32_t below = 0;
#pragma unroll
    for (int it = 0; it < kScanItems; ++it) {
      if (base + it < wL) below += __popc(w[it]);
      else if (base + it == wL) below += __popc(w[it] & ((1u << (L & 31)) - 1u));
    }
    sz->n_local_new[hop - 1] = (int64_t)before + ex + below;
  }
  int64_t off = n_prev + before + ex;
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    uint32_t x = w[it];
    if (!x) continue;
    const int32_t ubase = (int32_t)((base + it) << 5);
    while (x) {
      const int b = __ffs(x) - 1;
      x &= x - 1;
      const int32_t u = ubase + b;
      nodes[off] = u;
      pos_of[u] = (int32_t)off;
      ++off;
    }
    bits[base + it] = 0u;
  }
  if (threadIdx.x == 0 && blockIdx.x == gridDim.x - 1) {
    sz->n[hop] = n_prev + before + tot;
    if (wL >= W) sz->n_local_new[hop - 1] = (int64_t)before + tot;  // every id is below L
  }
}

// Relabel the last hop's sampled ids to their frontier positions (earlier
// hops are relabelled by the next hop's k_row_scan).
__global__ __launch_bounds__(kScanNT) void k_relabel(int32_t* __restrict__ ids, const StepSizes* sz, int hop,
                                                     const int32_t* __restrict__ pos_of) {
  if (sz->status) return;
  relabel_tiles(ids, sz->e[hop - 1], pos_of, blockIdx.x, gridDim.x);
}

}  // namespace ms
