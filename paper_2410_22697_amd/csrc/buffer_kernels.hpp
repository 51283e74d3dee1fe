// buffer_kernels.hpp - halo prefetch buffer: lookup, scoring, gather,
// eviction select, replacement select, swap (Algorithm 2 and Section IV-B).
#pragma once

#include "common.hpp"
#include "sample_kernels.hpp"

namespace ms {

constexpr uint64_t kEmpty = ~0ull;

// 16- and 8-byte vectors of the copy kernels and the table windows
typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef unsigned int v2u __attribute__((ext_vector_type(2)));

// MurmurHash3 fmix32 finaliser (public domain).
__device__ __forceinline__ uint32_t fmix32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x85ebca6bu;
  x ^= x >> 13;
  x *= 0xc2b2ae35u;
  x ^= x >> 16;
  return x;
}

// Open-addressing table (linear probing, load <= 1/2): entry = slot << 32 | h.
__device__ __forceinline__ int32_t hash_find(const uint64_t* __restrict__ tab, uint32_t mask, int32_t h) {
  uint32_t i = fmix32((uint32_t)h) & mask;
  while (true) {
    const uint64_t e = tab[i];
    if ((uint32_t)e == (uint32_t)h) return (int32_t)(e >> 32);
    if (e == kEmpty) return -1;
    i = (i + 1) & mask;
  }
}

// The same search continued from entry i (after a window of entries that
// held neither h nor an empty entry).
__device__ __forceinline__ int32_t hash_find_from(const uint64_t* __restrict__ tab, uint32_t mask, int32_t h,
                                                  uint32_t i) {
  while (true) {
    const uint64_t e = tab[i];
    if ((uint32_t)e == (uint32_t)h) return (int32_t)(e >> 32);
    if (e == kEmpty) return -1;
    i = (i + 1) & mask;
  }
}

__global__ void k_hash_insert(uint64_t* __restrict__ tab, uint32_t mask, const int32_t* __restrict__ slot_id,
                              int64_t cap, const int64_t* __restrict__ gate) {
  if (gate && *gate == 0) return;
  for (int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; s < cap;
       s += (int64_t)gridDim.x * blockDim.x) {
    const int32_t h = slot_id[s];
    const uint64_t entry = ((uint64_t)(uint32_t)s << 32) | (uint32_t)h;
    uint32_t i = fmix32((uint32_t)h) & mask;
    while (atomicCAS((unsigned long long*)&tab[i], (unsigned long long)kEmpty, (unsigned long long)entry) !=
           (unsigned long long)kEmpty)
      i = (i + 1) & mask;
  }
}

template <typename T>
__global__ void k_fill(T* __restrict__ p, int64_t n, T v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// ------------------------------------------------------------- classify
// For every frontier node: local / buffer hit / miss against the buffer as it
// stands at the start of the step. Hits count this step for the lazy S_E
// decay (hitcnt); misses take S_A += 1. Rows go to two gather lists, (row,
// HBM slab row) and (row, halo id), compacted with wave ballots and one
// atomic per wave. Also clears pos_of for the next step.
struct ClassifyArgs {
  const int32_t* nodes;
  StepSizes* sz;
  int32_t K;
  int32_t L;
  const uint64_t* tab;
  uint32_t tmask;
  int32_t* hitcnt;
  float* S_A;                 // by halo rank, or by global id
  const int32_t* sa_idx;      // halo id -> its S_A index (rank, or global id)
  int32_t* pos_of;
  uint8_t* mask;
  int2* hbm_list;
  int2* miss_list;
  int32_t* miss_slot;         // per miss-list entry: the slot of a pending hit, else -1
  const int32_t* slot_round;  // round that last refilled each slot
  const int32_t* landed;      // round whose refill row has landed in each slot
  int32_t pend_round;         // refill of this round may still be in flight (-1: none)
  const int32_t* seeds;       // the step's seeds (their frontier positions are taken back if invalid)
  int32_t n0;
};

constexpr int kClsNT = 256;
constexpr int kClsItems = 4;  // rows per thread: one block classifies 1024 rows per pass
constexpr int kClsBlocks = 512;  // grid bound: the blocks stride over the frontier the step found

// Block-level aggregation: each block counts its rows per list, takes one
// base per list with a single atomic, and places rows with wave ballots. The
// step's local, hit and miss counts need no atomics here: the local rows are
// the seeds plus the new nodes below L that the dedup scans counted, and the
// completion kernel derives hits and misses from the two list lengths (and
// the hits on slots still refilling, counted here only while a refill is in
// flight). Hits add one to their slot's count with a no-return atomic.
// The loads of a thread go out in rounds, each for all its rows: the
// frontier ids; a window of four table entries from each id's probe start
// (the 16-byte pairs holding entries p & ~1 .. (p & ~1) + 3, which settle
// almost every search; the rare rest probes on one by one); the misses'
// S_A indices (rank or global id) and, while a refill is in flight, the hit
// slots' refill stamps. Lanes past the end and local rows load dummy
// (in-range) addresses and change nothing.
__global__ __launch_bounds__(kClsNT) void k_classify(ClassifyArgs a) {
  constexpr int NW = kClsNT / MS_WAVE;
  __shared__ int32_t wc[NW][3];          // per-wave counts: hbm list, host list, pending hits
  __shared__ unsigned long long base[2];
  if (a.sz->status) {
    // invalid seeds: every kernel of the step has skipped, and the frontier
    // positions the seed check marked are taken back, so the step leaves no trace
    if (a.sz->status & 3)
      for (int64_t i = (int64_t)blockIdx.x * kClsNT + threadIdx.x; i < a.n0; i += (int64_t)gridDim.x * kClsNT) {
        const int32_t v = a.seeds[i];
        if (v >= 0 && v < a.L) a.pos_of[v] = -1;
      }
    return;
  }
  const int64_t n = a.sz->n[a.K];
  const int lane = lane_id(), wave = wave_id();
  const int64_t tile = (int64_t)kClsNT * kClsItems;
  const bool pending = a.pend_round >= 0;
  for (int64_t b0 = (int64_t)blockIdx.x * tile; b0 < n; b0 += (int64_t)gridDim.x * tile) {
    int32_t v[kClsItems], slot[kClsItems];
#pragma unroll
    for (int it = 0; it < kClsItems; ++it) {
      // wave w of item it covers rows b0 + it*256 + w*64 + lane
      const int64_t i = b0 + (int64_t)it * kClsNT + threadIdx.x;
      v[it] = a.nodes[i < n ? i : n - 1];
    }
#pragma unroll
    for (int it = 0; it < kClsItems; ++it) pin(v[it]);
    {
      v4u w0[kClsItems], w1[kClsItems];
#pragma unroll
      for (int it = 0; it < kClsItems; ++it) {
        const uint32_t q = (fmix32((uint32_t)(v[it] - a.L)) & a.tmask) & ~1u;
        w0[it] = *reinterpret_cast<const v4u*>(a.tab + q);
        w1[it] = *reinterpret_cast<const v4u*>(a.tab + ((q + 2) & a.tmask));
      }
#pragma unroll
      for (int it = 0; it < kClsItems; ++it) {
        pin(w0[it]);
        pin(w1[it]);
      }
#pragma unroll
      for (int it = 0; it < kClsItems; ++it) {
        const int32_t h = v[it] - a.L;
        const uint32_t p = fmix32((uint32_t)h) & a.tmask;
        const uint64_t e[4] = {((uint64_t)w0[it].y << 32) | w0[it].x, ((uint64_t)w0[it].w << 32) | w0[it].z,
                               ((uint64_t)w1[it].y << 32) | w1[it].x, ((uint64_t)w1[it].w << 32) | w1[it].z};
        int32_t r = -2;  // -2: not settled by the window
#pragma unroll
        for (int x = 0; x < 4; ++x)
          if (r == -2 && x >= (int)(p & 1u)) {
            if ((uint32_t)e[x] == (uint32_t)h) r = (int32_t)(e[x] >> 32);
            else if (e[x] == kEmpty) r = -1;
          }
        if (v[it] < a.L) r = -1;
        else if (r == -2) r = hash_find_from(a.tab, a.tmask, h, ((p & ~1u) + 4) & a.tmask);
        slot[it] = r;
      }
    }
    int32_t sr[kClsItems], ld[kClsItems], rk[kClsItems];
#pragma unroll
    for (int it = 0; it < kClsItems; ++it) {
      const int32_t sl = slot[it] >= 0 ? slot[it] : 0;
      rk[it] = a.sa_idx[v[it] >= a.L && slot[it] < 0 ? v[it] - a.L : 0];
      sr[it] = 0;
      ld[it] = 0;
      if (pending) {  // the same in every lane
        sr[it] = a.slot_round[sl];
        ld[it] = __hip_atomic_load(&a.landed[sl], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
#pragma unroll
    for (int it = 0; it < kClsItems; ++it) {
      pin(sr[it]);
      pin(ld[it]);
      pin(rk[it]);
    }
    int cls[kClsItems];
    int32_t src[kClsItems], wslot[kClsItems];
    int ch = 0, cm = 0, cp = 0;  // hbm list, host list, pending hits
#pragma unroll
    for (int it = 0; it < kClsItems; ++it) {
      const int64_t i = b0 + (int64_t)it * kClsNT + threadIdx.x;
      cls[it] = -1;
      src[it] = 0;
      wslot[it] = -1;
      if (i < n) {
        a.pos_of[v[it]] = -1;
        const int32_t h = v[it] - a.L;
        if (v[it] < a.L) {
          cls[it] = 0;
          src[it] = v[it];
        } else if (slot[it] >= 0) {
          cls[it] = 1;
          src[it] = a.L + slot[it];
          atomicAdd(&a.hitcnt[slot[it]], 1);  // each slot once per step: no contention
          // a hit on a slot whose refill may not have landed reads the same
          // row from the host store
          if (pending && sr[it] == a.pend_round && ld[it] != a.pend_round) {
            cls[it] = 3;
            src[it] = h;
            wslot[it] = slot[it];
          }
        } else {
          cls[it] = 2;
          src[it] = h;
          atomicAdd(&a.S_A[rk[it]], 1.0f);
        }
        a.mask[i] = (uint8_t)(cls[it] == 3 ? 1 : cls[it]);
      }
      ch += __popcll(ballot(cls[it] == 0 || cls[it] == 1));
      cm += __popcll(ballot(cls[it] >= 2));
      if (pending) cp += __popcll(ballot(cls[it] == 3));
    }
    if (lane == 0) {
      wc[wave][0] = ch;
      wc[wave][1] = cm;
      wc[wave][2] = cp;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int th = 0, tm = 0, tp = 0;
      for (int w = 0; w < NW; ++w) {
        th += wc[w][0];
        tm += wc[w][1];
        tp += wc[w][2];
      }
      base[0] = th ? atomicAdd((unsigned long long*)&a.sz->n_hbm, (unsigned long long)th) : 0ull;
      base[1] = tm ? atomicAdd((unsigned long long*)&a.sz->n_miss, (unsigned long long)tm) : 0ull;
      if (tp) atomicAdd((unsigned long long*)&a.sz->n_pending, (unsigned long long)tp);
    }
    __syncthreads();
    // this wave's offset inside the block's share of each list
    unsigned long long oh = base[0], om = base[1];
    for (int w = 0; w < wave; ++w) {
      oh += wc[w][0];
      om += wc[w][1];
    }
#pragma unroll
    for (int it = 0; it < kClsItems; ++it) {
      const int64_t i = b0 + (int64_t)it * kClsNT + threadIdx.x;
      const uint64_t mh = ballot(cls[it] == 0 || cls[it] == 1);
      const uint64_t mm = ballot(cls[it] >= 2);
      if (cls[it] == 0 || cls[it] == 1) a.hbm_list[oh + lanes_below(mh)] = make_int2((int32_t)i, src[it]);
      else if (cls[it] >= 2) {
        a.miss_list[om + lanes_below(mm)] = make_int2((int32_t)i, src[it]);
        a.miss_slot[om + lanes_below(mm)] = wslot[it];
      }
      oh += __popcll(mh);
      om += __popcll(mm);
    }
    __syncthreads();
  }
}

// The step's completion, done by the step's last kernel on the side stream:
// the slots written through are stamped landed for round `round_id` (none if
// round_id < 0), and one block derives the step's counts (local rows: the
// seeds plus the new nodes below L of each hop; hits: the HBM list's buffer
// rows plus the hits read over the host link; misses: the rest of the host
// list), then copies the step's sizes and the eviction-round consistency flag
// into the pinned host mailbox (device view), made visible to the host. Every
// value it copies is final once classify has run (the round it checks ran
// before classify), and the host reads the mailbox only after the kernel ends.
constexpr int kSizeWords = (int)(sizeof(StepSizes) / 4);
static_assert(sizeof(StepSizes) % 4 == 0 && kSizeWords < 256, "mailbox copy: one word per thread");
struct StepTail {
  StepSizes* sz;
  int32_t K;
  const int32_t* bad;
  StepSizes* h_sz;
  int32_t* h_bad;
  int32_t* landed;
  int64_t cap;
  int32_t round_id;
  int32_t clear;  // the miss gather's last block clears the sizes (block 0 has published them by then)
};

// one whole block of at least kSizeWords + 1 threads
__device__ __forceinline__ void publish_step(const StepTail& t) {
  const int i = threadIdx.x;
  StepSizes* sz = t.sz;
  if (i == 0 && !sz->status) {
    int64_t local = sz->n[0];
    for (int k = 0; k < t.K; ++k) local += sz->n_local_new[k];
    sz->local = local;
    sz->hits = sz->n_hbm - local + sz->n_pending;
    sz->misses = sz->n_miss - sz->n_pending;
  }
  __syncthreads();
  if (i < kSizeWords) reinterpret_cast<int32_t*>(t.h_sz)[i] = reinterpret_cast<const int32_t*>(sz)[i];
  if (i == kSizeWords) *t.h_bad = *t.bad;
  __threadfence_system();
}

// ---------------------------------------------------------------- gather
// dst row list[x].x <- src row list[x].y, as a bit copy of row_bytes. The
// (row, chunk) work is flattened so every lane moves one vector per chunk
// whatever the row size. Each lane takes U chunks per pass: first every list
// entry, then every row load, then the stores, so all U loads of a lane are in
// flight together. No load may sit behind a branch (the compiler would sink it
// into the predicated store and wait for it there): in the last pass a lane
// past the end re-reads its first chunk, or, where re-reading costs host-link
// bytes, a dummy device row; the loaded values are pinned with an empty asm
// before the predicated stores.

// chunk cc of the flattened space -> (list entry, byte offset in the row);
// ONE: one chunk per row (no division)
template <typename V, bool ONE>
__device__ __forceinline__ void chunk_of(uint64_t cc, uint32_t cpr, uint64_t magic, uint64_t& task,
                                         uint64_t& off) {
  task = ONE ? cc : __umul64hi(cc, magic);
  off = (cc - task * cpr) * sizeof(V);
}

template <typename V, bool ONE, int U>
__device__ __forceinline__ void gather_body(const int2* __restrict__ list, const int64_t* __restrict__ count,
                                            const uint8_t* __restrict__ src, uint8_t* __restrict__ dst, int64_t rb,
                                            uint32_t cpr, uint64_t magic) {
  const uint64_t n = (uint64_t)*count;
  const uint64_t total = n * cpr;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t c = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; c < total; c += U * stride) {
    uint64_t task[U], off[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint64_t cc = c + u * stride;
      chunk_of<V, ONE>(cc < total ? cc : c, cpr, magic, task[u], off[u]);
    }
    int2 e[U];
#pragma unroll
    for (int u = 0; u < U; ++u) e[u] = list[task[u]];
    V v[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      v[u] = *reinterpret_cast<const V*>(src + (uint64_t)(uint32_t)e[u].y * rb + off[u]);
#pragma unroll
    for (int u = 0; u < U; ++u) asm volatile("" : "+v"(v[u]));
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (c + u * stride < total)
        __builtin_nontemporal_store(v[u], reinterpret_cast<V*>(dst + (uint64_t)(uint32_t)e[u].x * rb + off[u]));
  }
}

// local rows and buffer hits: HBM slab -> output rows. The next step's
// sampling runs beside it; its waves take the highest issue priority, so that
// on a CU they share, the gather's loads and stores go out first (31.3-31.5 us
// per launch against 32.0 on the papers-sized share).
template <typename V, bool ONE>
__global__ __launch_bounds__(256) void k_gather_hbm(const int2* __restrict__ list, const int64_t* __restrict__ count,
                                                    const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                                                    int64_t rb, uint32_t cpr, uint64_t magic) {
  __builtin_amdgcn_s_setprio(3);
  gather_body<V, ONE, 4>(list, count, src, dst, rb, cpr, magic);
}
// misses: pinned host store (over the host link) -> output rows. The list
// also holds the hits on slots whose refill had not landed when the step was
// classified; such a row is written into its buffer slot too (wslot >= 0), so
// a replacement row crosses the link once, together with the misses (the
// merged fetch of Algorithm 2), and the lane that writes its first chunk
// stamps the slot landed. Every kernel that reads a buffer row because of
// that stamp (a later HBM gather) runs after this one in stream order; a
// refill chunk that sees it skips a row this kernel writes anyway (same
// bytes). Block 0 publishes the step (the completion above) once its share
// of the rows is done, so no kernel follows this one in the step (publishing
// first, beside the next step's sampling, measured ~2% slower before the
// first round; publishing from the last block to finish, ~1% slower in the
// link-bound steps). The last block to finish then clears the step's sizes,
// so the slot's next step needs no clearing of its own (tail.clear).
// dummy: a device row of row_bytes that lanes past the end move onto itself.
template <typename V, bool ONE>
__global__ __launch_bounds__(256) void k_gather_miss(const int2* __restrict__ list, const int32_t* __restrict__ wslot,
                                                     const int64_t* __restrict__ count, const uint8_t* __restrict__ src,
                                                     uint8_t* __restrict__ dst, uint8_t* __restrict__ buf,
                                                     uint8_t* __restrict__ dummy, int64_t rb, uint32_t cpr,
                                                     uint64_t magic, StepTail tail) {
  constexpr int U = 4;
  const uint64_t n = (uint64_t)*count;
  const uint64_t total = n * cpr;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t c = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; c < total; c += U * stride) {
    uint64_t task[U], off[U];
    bool in[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint64_t cc = c + u * stride;
      in[u] = cc < total;
      chunk_of<V, ONE>(in[u] ? cc : c, cpr, magic, task[u], off[u]);
    }
    int2 e[U];
    int32_t ws[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      e[u] = list[task[u]];
      ws[u] = wslot[task[u]];
    }
    V v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint8_t* p = in[u] ? src + (uint64_t)(uint32_t)e[u].y * rb + off[u] : dummy + off[u];
      v[u] = *reinterpret_cast<const V*>(p);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      uint8_t* q = in[u] ? dst + (uint64_t)(uint32_t)e[u].x * rb + off[u] : dummy + off[u];
      __builtin_nontemporal_store(v[u], reinterpret_cast<V*>(q));
      if (in[u] && ws[u] >= 0) {
        *reinterpret_cast<V*>(buf + (uint64_t)(uint32_t)ws[u] * rb + off[u]) = v[u];
        if (off[u] == 0 && tail.round_id >= 0 && ws[u] < tail.cap)
          __hip_atomic_store(&tail.landed[ws[u]], tail.round_id, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
  if (blockIdx.x == 0) publish_step(tail);
  // the last block to finish clears the sizes for the slot's next step (every
  // block has read its count, and block 0 has published them, by then)
  __shared__ int last;
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence();
    last = atomicAdd(&tail.sz->blocks_done, 1) == (int)gridDim.x - 1;
  }
  __syncthreads();
  if (last && tail.clear) {
    __threadfence();
    for (int i = threadIdx.x; i < kSizeWords; i += blockDim.x) reinterpret_cast<int32_t*>(tail.sz)[i] = 0;
  }
}

// The step's completion as a kernel of its own, where no miss gather ends
// the step (the staged host link, which scatters the host rows with other
// kernels; a context without halo nodes): after the kernels that wrote the
// step's rows (a kernel boundary), the written-through slots are stamped
// landed, and block 0 publishes the step.
__global__ __launch_bounds__(256) void k_step_done(const int32_t* __restrict__ wslot,
                                                   const int64_t* __restrict__ count, int32_t* __restrict__ landed,
                                                   int64_t cap, int32_t round_id, StepSizes* __restrict__ sz, int32_t K,
                                                   const int32_t* __restrict__ bad, StepSizes* h_sz, int32_t* h_bad) {
  if (round_id >= 0) {
    const int64_t n = *count;
    for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < n; x += (int64_t)gridDim.x * blockDim.x) {
      const int32_t ws = wslot[x];
      if (ws >= 0 && ws < cap) __hip_atomic_store(&landed[ws], round_id, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  if (blockIdx.x == 0) {
    const StepTail t{sz, K, bad, h_sz, h_bad, landed, cap, round_id, 0};
    publish_step(t);
  }
}

// Eviction refill: pinned host store -> buffer slots, row by row (G lanes
// per row), in list order (replacements of highest S_A first), kRefillRows
// rows in flight per lane group. A row is copied unless its slot has landed
// already (written through by a miss gather) or k_swap flagged the entry; a
// row that is not copied moves the dummy device row onto itself instead, so
// no load or store is behind a branch. Each batch of rows is then published:
// release fence, then landed[slot] = round, which classify reads to serve
// hits on those slots from HBM.
constexpr int kRefillRows = 16;

template <typename V>
__global__ __launch_bounds__(256) void k_refill(const int2* __restrict__ list, const int64_t* __restrict__ count,
                                                const uint8_t* __restrict__ src, uint8_t* __restrict__ dst,
                                                uint8_t* __restrict__ dummy, int64_t rb, uint32_t cpr, uint32_t G,
                                                int32_t L, int32_t* __restrict__ landed, int32_t round_id,
                                                int32_t chunk, int32_t nchunks, Counters* __restrict__ ctr) {
  // this launch refills fill-list rows [lo, hi): chunk `chunk` of `nchunks`
  const int64_t k = *count;
  const int64_t lo = k * chunk / nchunks, hi = k * (chunk + 1) / nchunks;
  const int64_t n = hi - lo;
  list += lo;
  const int lane = lane_id();
  const int rpw = MS_WAVE / (int)G;  // row slots per wave (G divides the wave)
  const int sub = lane / (int)G, cl = lane % (int)G;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / MS_WAVE;
  const int64_t nwaves = (int64_t)gridDim.x * blockDim.x / MS_WAVE;
  const int64_t per = (int64_t)kRefillRows * rpw;
  for (int64_t base = wave * per; base < n; base += nwaves * per) {
    int2 e[kRefillRows];
    bool ok[kRefillRows];
#pragma unroll
    for (int u = 0; u < kRefillRows; ++u) {
      const int64_t r = base + (int64_t)u * rpw + sub;
      ok[u] = r < n;
      e[u] = list[ok[u] ? r : base];
    }
    int32_t lv[kRefillRows];
#pragma unroll
    for (int u = 0; u < kRefillRows; ++u) {
      ok[u] = ok[u] && e[u].x >= L && e[u].y >= 0;  // entries flagged inconsistent by k_swap are skipped
      lv[u] = __hip_atomic_load(&landed[ok[u] ? e[u].x - L : 0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
#pragma unroll
    for (int u = 0; u < kRefillRows; ++u) ok[u] = ok[u] && lv[u] != round_id;
    for (uint32_t ch = cl; ch < cpr; ch += G) {
      const uint64_t off = (uint64_t)ch * sizeof(V);
      V v[kRefillRows];
#pragma unroll
      for (int u = 0; u < kRefillRows; ++u)
        v[u] = *reinterpret_cast<const V*>((ok[u] ? src + (uint64_t)(uint32_t)e[u].y * rb : dummy) + off);
#pragma unroll
      for (int u = 0; u < kRefillRows; ++u)
        *reinterpret_cast<V*>((ok[u] ? dst + (uint64_t)(uint32_t)e[u].x * rb : dummy) + off) = v[u];
    }
    __threadfence();
    if (cl == 0) {
      unsigned long long copied = 0;
#pragma unroll
      for (int u = 0; u < kRefillRows; ++u)
        if (ok[u]) {
          __hip_atomic_store(&landed[e[u].x - L], round_id, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          copied += 1;
        }
      if (copied) atomicAdd((unsigned long long*)&ctr->refilled, copied);
    }
  }
}

// ------------------------------------------------------------ staged host link
// In the staged link mode the rows that cross the host link are gathered by
// host threads into pinned staging memory and moved by the DMA engines, so
// no kernel reads the host store. These kernels hand the row ids to the host
// and scatter the staged rows on the device.

// The host rows (.y) of the first min(*count, cap) entries of an (x, y)
// list, and that count, written into pinned host memory through its device
// views; made visible to the host before the kernel ends.
__global__ __launch_bounds__(256) void k_rows_out(const int2* __restrict__ list, const int64_t* __restrict__ count,
                                                  int64_t cap, int32_t* h_rows, int64_t* h_count) {
  const int64_t n = min(max(*count, (int64_t)0), cap);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    h_rows[i] = list[i].y;
  if (blockIdx.x == 0 && threadIdx.x == 0) *h_count = n;
  __threadfence_system();
}

// Misses: staged row r (miss-list entry lo + r, r < n) goes to output row
// list[lo + r].x, and into buffer slot wslot[lo + r] as well when that is
// >= 0 (a hit on a slot whose refill has not landed).
template <typename V, bool ONE>
__global__ __launch_bounds__(256) void k_scatter_rows(const uint8_t* __restrict__ stage, const int2* __restrict__ list,
                                                      const int32_t* __restrict__ wslot, int64_t lo, int64_t n,
                                                      uint8_t* __restrict__ dst, uint8_t* __restrict__ buf, int64_t rb,
                                                      uint32_t cpr, uint64_t magic) {
  const uint64_t total = (uint64_t)n * cpr;
  for (uint64_t c = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; c < total;
       c += (uint64_t)gridDim.x * blockDim.x) {
    uint64_t r, off;
    chunk_of<V, ONE>(c, cpr, magic, r, off);
    const V v = *reinterpret_cast<const V*>(stage + r * rb + off);
    const int2 e = list[lo + r];
    const int32_t ws = wslot[lo + r];
    __builtin_nontemporal_store(v, reinterpret_cast<V*>(dst + (uint64_t)(uint32_t)e.x * rb + off));
    if (ws >= 0) *reinterpret_cast<V*>(buf + (uint64_t)(uint32_t)ws * rb + off) = v;
  }
}

// Refill: staged row r (fill-list entry lo + r, r < n) goes into the slab
// row fill[lo + r].x, G lanes per row, under the rules of k_refill: skipped
// for an entry that k_swap flagged or a slot that has landed already, and
// published after a release fence with landed[slot] = round_id.
template <typename V>
__global__ __launch_bounds__(256) void k_refill_scatter(const uint8_t* __restrict__ stage,
                                                        const int2* __restrict__ fill, int64_t lo, int64_t n,
                                                        uint8_t* __restrict__ dst, int64_t rb, uint32_t cpr,
                                                        uint32_t G, int32_t L, int32_t* __restrict__ landed,
                                                        int32_t round_id, Counters* __restrict__ ctr) {
  const int lane = lane_id();
  const int rpw = MS_WAVE / (int)G;
  const int sub = lane / (int)G, cl = lane % (int)G;
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / MS_WAVE;
  const int64_t nwaves = (int64_t)gridDim.x * blockDim.x / MS_WAVE;
  for (int64_t r = wave * rpw + sub; r - sub < n; r += nwaves * rpw) {
    bool ok = r < n;
    const int2 e = ok ? fill[lo + r] : make_int2(-1, -1);
    ok = ok && e.x >= L && e.y >= 0;
    if (ok) ok = __hip_atomic_load(&landed[e.x - L], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != round_id;
    if (ok)
      for (uint32_t ch = cl; ch < cpr; ch += G) {
        const uint64_t off = (uint64_t)ch * sizeof(V);
        *reinterpret_cast<V*>(dst + (uint64_t)(uint32_t)e.x * rb + off) =
            *reinterpret_cast<const V*>(stage + (uint64_t)r * rb + off);
      }
    __threadfence();
    const uint64_t copied = __ballot(ok && cl == 0);
    if (ok && cl == 0) __hip_atomic_store(&landed[e.x - L], round_id, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (lane == 0 && copied) atomicAdd((unsigned long long*)&ctr->refilled, (unsigned long long)__popcll(copied));
  }
}

// ------------------------------------------------------------ lazy decay
// S_E[s] is multiplied by gamma once for every step in which slot s was not
// hit since the last materialisation: `steps` steps elapsed, hitcnt[s] of
// them hits. Same fp32 product sequence as one multiply per step.
__global__ void k_materialize(float* __restrict__ S_E, int32_t* __restrict__ hitcnt, int64_t cap, int32_t steps,
                              float gamma) {
  for (int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; s < cap; s += (int64_t)gridDim.x * blockDim.x) {
    const int32_t u = steps - hitcnt[s];
    float x = S_E[s];
    for (int32_t j = 0; j < u; ++j) x = __fmul_rn(x, gamma);
    S_E[s] = x;
    hitcnt[s] = 0;
  }
}

// ------------------------------------------------- ordered flag compaction
// E = [s : S_E[s] < alpha] in ascending s, as count / scan / emit.
__global__ __launch_bounds__(kScanNT) void k_evict_count(const float* __restrict__ S_E, int64_t cap, float alpha,
                                                         int32_t* __restrict__ partials, int64_t* __restrict__ total) {
  __shared__ int32_t lds[kScanNT / MS_WAVE + 1];
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  int32_t s = 0;
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t i = base + (int64_t)it * kScanNT + threadIdx.x;
    s += (i < cap && S_E[i] < alpha) ? 1 : 0;
  }
  s = block_sum<kScanNT>(s, lds);
  if (threadIdx.x == 0) {
    partials[blockIdx.x] = s;
    if (s) atomicAdd((unsigned long long*)total, (unsigned long long)s);
  }
}

__global__ __launch_bounds__(kScanNT) void k_evict_emit(const float* __restrict__ S_E, int64_t cap, float alpha,
                                                        const int32_t* __restrict__ partials,
                                                        int32_t* __restrict__ E) {
  __shared__ int32_t lds[kScanNT / MS_WAVE + 1];
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  bool f[kScanItems];
  int32_t s = 0;
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t i = base + it;
    f[it] = i < cap && S_E[i] < alpha;
    s += f[it];
  }
  const int32_t before = preceding_sum<kScanNT>(partials, blockIdx.x, lds);
  int32_t tot;
  int32_t o = block_exclusive_scan<kScanNT>(s, lds, &tot) + before;
#pragma unroll
  for (int it = 0; it < kScanItems; ++it)
    if (f[it]) E[o++] = (int32_t)(base + it);
}

// |C| = number of unbuffered halo nodes (S_A >= 0).
// k' = min(|E|, |C|) on the device; sets the select and the E narrowing up.
// |C| = H - cap always: a halo node has S_A = -1 exactly while it is buffered
// (init, and the swap's S_A := -1 for a replacement) and S_A >= 0 otherwise
// (misses only add to it; an evicted node gets its last S_E >= 0).
__global__ void k_round_setup(RoundState* __restrict__ rs, Counters* __restrict__ ctr, int64_t nC) {
  rs->nC = nC;
  const int64_t k = rs->nE < nC ? rs->nE : nC;
  rs->k = k;
  rs->need = k;
  rs->prefix = 0;
  rs->pmask = 0;
  rs->prefix_lo = 0;
  rs->pmask_lo = 0;
  rs->nE_sel = k < rs->nE ? rs->nE : 0;
  rs->k_sel = k < rs->nE ? k : 0;
  if (k > 0) {
    ctr->rounds += 1;
    ctr->evicted += k;
  }
}

template <typename T>
__global__ void k_fill_gated(T* __restrict__ p, int64_t n, T v, const int64_t* __restrict__ gate) {
  if (*gate == 0) return;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// ------------------------------------------------------ replacement select
// Candidate key: bitwise NOT of the fp32 bits of S_A >= 0, so ascending key
// is descending S_A. Radix select, 8 bits per pass from the top, finds the
// key T of the k'-th candidate and how many candidates with key T to take.
__device__ __forceinline__ uint32_t cand_key(float a) { return ~__float_as_uint(a); }

// One radix-select pass over the candidate keys (S_A >= 0, by rank) that
// match the prefix so far. Each thread takes four consecutive scores per
// iteration (one 16-byte load); a wave adds the lanes whose digit equals its
// first active lane's with one LDS atomic (most candidates have S_A = 0, one
// digit), the others one by one.
__global__ __launch_bounds__(256) void k_select_hist(const float* __restrict__ S_A, int64_t H,
                                                     const RoundState* __restrict__ rs, int shift,
                                                     uint32_t* __restrict__ ghist) {
  __shared__ uint32_t hist[256];
  if (rs->k == 0) return;
  hist[threadIdx.x] = 0;
  __syncthreads();
  const uint32_t prefix = rs->prefix, pmask = rs->pmask;
  const int lane = lane_id();
  const int64_t H4 = H / 4;
  const float4* S4 = reinterpret_cast<const float4*>(S_A);
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < (H + 3) / 4;
       q += (int64_t)gridDim.x * blockDim.x) {
    float a[4] = {-1.0f, -1.0f, -1.0f, -1.0f};
    if (q < H4) {
      const float4 x = S4[q];
      a[0] = x.x;
      a[1] = x.y;
      a[2] = x.z;
      a[3] = x.w;
    } else {
      for (int j = 0; j < 4; ++j)
        if (4 * q + j < H) a[j] = S_A[4 * q + j];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t k = cand_key(a[j]);
      const bool in = a[j] >= 0.0f && (k & pmask) == prefix;
      const uint32_t d = (k >> shift) & 255u;
      const uint64_t m = ballot(in);
      if (!m) continue;
      const int first = __ffsll((unsigned long long)m) - 1;
      const uint32_t d0 = __shfl(d, first, MS_WAVE);
      const uint64_t same = ballot(in && d == d0);
      if (lane == first) atomicAdd(&hist[d0], (uint32_t)__popcll(same));
      else if (in && d != d0) atomicAdd(&hist[d], 1u);
    }
  }
  __syncthreads();
  if (hist[threadIdx.x]) atomicAdd(&ghist[threadIdx.x], hist[threadIdx.x]);
}

__global__ __launch_bounds__(256) void k_select_pick(RoundState* __restrict__ rs, uint32_t* __restrict__ ghist,
                                                     int shift, int32_t* __restrict__ bad, int lo_word = 0) {
  __shared__ int64_t lds[256 / MS_WAVE + 1];
  __shared__ int32_t pick;
  __shared__ int64_t before;
  if (rs->k == 0) return;
  if (threadIdx.x == 0) {
    pick = -1;
    before = 0;
  }
  __syncthreads();
  const int64_t need = rs->need;
  const int64_t c = ghist[threadIdx.x];
  int64_t tot;
  const int64_t ex = block_exclusive_scan<256>(c, lds, &tot);
  if (ex < need && ex + c >= need) {
    pick = threadIdx.x;
    before = ex;
  }
  __syncthreads();
  ghist[threadIdx.x] = 0;
  if (threadIdx.x == 0) {
    if (pick < 0) {  // fewer candidates than asked for: never expected
      atomicOr(bad, 2);
      rs->need = 0;
    } else {
      rs->need = need - before;
      if (lo_word) {
        rs->prefix_lo |= (uint32_t)pick << shift;
        rs->pmask_lo |= 255u << shift;
      } else {
        rs->prefix |= (uint32_t)pick << shift;
        rs->pmask |= 255u << shift;
      }
    }
  }
}

// In rank order r: candidates with key < T go to (keys, vals) for sorting,
// the first `need` with key == T go straight to R[n_lt + ...]. S_A is kept by
// rank, so both passes read it (and h_of_rank) in order.
__global__ __launch_bounds__(kScanNT) void k_rank_count(const float* __restrict__ S_A, int64_t H,
                                                        RoundState* __restrict__ rs,
                                                        int32_t* __restrict__ p_lt, int32_t* __restrict__ p_eq) {
  __shared__ int32_t lds[kScanNT / MS_WAVE + 1];
  const uint32_t T = rs->prefix;
  const bool on = rs->k > 0;
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  float a[kScanItems];
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t r = base + (int64_t)it * kScanNT + threadIdx.x;
    a[it] = on && r < H ? S_A[r] : -1.0f;
  }
  int32_t clt = 0, ceq = 0;
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    if (a[it] >= 0.0f) {
      const uint32_t k = cand_key(a[it]);
      clt += k < T;
      ceq += k == T;
    }
  }
  clt = block_sum<kScanNT>(clt, lds);
  ceq = block_sum<kScanNT>(ceq, lds);
  if (threadIdx.x == 0) {
    p_lt[blockIdx.x] = clt;
    p_eq[blockIdx.x] = ceq;
    if (clt) atomicAdd((unsigned long long*)&rs->n_lt, (unsigned long long)clt);
    if (ceq) atomicAdd((unsigned long long*)&rs->n_eq, (unsigned long long)ceq);
  }
}

__global__ __launch_bounds__(kScanNT) void k_rank_emit(const float* __restrict__ S_A,
                                                       const int32_t* __restrict__ h_of_rank, int64_t H,
                                                       const RoundState* __restrict__ rs,
                                                       const int32_t* __restrict__ p_lt,
                                                       const int32_t* __restrict__ p_eq,
                                                       uint32_t* __restrict__ keys, int32_t* __restrict__ vals,
                                                       int32_t* __restrict__ R) {
  __shared__ int32_t lds[kScanNT / MS_WAVE + 1];
  if (rs->k == 0) return;
  const uint32_t T = rs->prefix;
  const int64_t need = rs->need, n_lt = rs->k - rs->need;
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  uint32_t k[kScanItems];
  float a[kScanItems];
  int32_t h[kScanItems];
  bool lt[kScanItems], eq[kScanItems];
  int32_t clt = 0, ceq = 0;
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t r = base + it;
    a[it] = r < H ? S_A[r] : -1.0f;
    h[it] = r < H ? h_of_rank[r] : -1;
  }
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    k[it] = cand_key(a[it]);
    lt[it] = a[it] >= 0.0f && k[it] < T;
    eq[it] = a[it] >= 0.0f && k[it] == T;
    clt += lt[it];
    ceq += eq[it];
  }
  const int32_t blt = preceding_sum<kScanNT>(p_lt, blockIdx.x, lds);
  const int32_t beq = preceding_sum<kScanNT>(p_eq, blockIdx.x, lds);
  int32_t tlt, teq;
  int64_t olt = (int64_t)block_exclusive_scan<kScanNT>(clt, lds, &tlt) + blt;
  int64_t oeq = (int64_t)block_exclusive_scan<kScanNT>(ceq, lds, &teq) + beq;
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    if (lt[it]) {
      keys[olt] = k[it];
      vals[olt] = h[it];
      ++olt;
    } else if (eq[it]) {
      if (oeq < need) R[n_lt + oeq] = h[it];
      ++oeq;
    }
  }
}

// S_A by halo id (for export), from either layout.
__global__ void k_scores_by_id(const float* __restrict__ S_A, const int32_t* __restrict__ sa_idx, int64_t H,
                               float* __restrict__ out) {
  for (int64_t h = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; h < H; h += (int64_t)gridDim.x * blockDim.x)
    out[h] = S_A[sa_idx[h]];
}

// ---------------------------------------- replacement select, S_A by global id
// With S_A over every global id g (non-halo ids hold -1 and are never
// candidates), the scan runs in id order, not rank order, so the rank is part
// of the key: candidate g has the 64-bit key (cand_key(S_A[g]), rank_g[g]),
// unique per candidate. An exact radix select over it, 8 bits per pass from
// the top (four passes on the score word, then four on the rank word), finds
// the k'-th smallest key T; the replacements are exactly the keys <= T, which
// are emitted and sorted by (score, rank). Each thread takes four
// consecutive entries per iteration; a wave adds the lanes whose digit equals
// its first active lane's with one LDS atomic.
__global__ __launch_bounds__(256) void k_gselect_hist(const float* __restrict__ S, const int32_t* __restrict__ rank_g,
                                                      int64_t n, const RoundState* __restrict__ rs, int lo_word,
                                                      int shift, uint32_t* __restrict__ ghist) {
  __shared__ uint32_t hist[256];
  if (rs->k == 0) return;
  hist[threadIdx.x] = 0;
  __syncthreads();
  const uint32_t ph = rs->prefix, mh = rs->pmask, pl = rs->prefix_lo, ml = rs->pmask_lo;
  const int lane = lane_id();
  const int64_t n4 = n / 4;
  const float4* S4 = reinterpret_cast<const float4*>(S);
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < (n + 3) / 4;
       q += (int64_t)gridDim.x * blockDim.x) {
    float a[4] = {-1.0f, -1.0f, -1.0f, -1.0f};
    if (q < n4) {
      const float4 x = S4[q];
      a[0] = x.x;
      a[1] = x.y;
      a[2] = x.z;
      a[3] = x.w;
    } else {
      for (int j = 0; j < 4; ++j)
        if (4 * q + j < n) a[j] = S[4 * q + j];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t k = cand_key(a[j]);
      bool in = a[j] >= 0.0f && (k & mh) == ph;
      uint32_t r = 0;
      if (lo_word && in) r = (uint32_t)rank_g[4 * q + j];
      in = in && (!lo_word || (r & ml) == pl);
      const uint32_t d = ((lo_word ? r : k) >> shift) & 255u;
      const uint64_t m = ballot(in);
      if (!m) continue;
      const int first = __ffsll((unsigned long long)m) - 1;
      const uint32_t d0 = __shfl(d, first, MS_WAVE);
      const uint64_t same = ballot(in && d == d0);
      if (lane == first) atomicAdd(&hist[d0], (uint32_t)__popcll(same));
      else if (in && d != d0) atomicAdd(&hist[d], 1u);
    }
  }
  __syncthreads();
  if (hist[threadIdx.x]) atomicAdd(&ghist[threadIdx.x], hist[threadIdx.x]);
}

__device__ __forceinline__ bool gsel_in(float a, uint32_t r, uint32_t th, uint32_t tl) {
  if (!(a >= 0.0f)) return false;
  const uint32_t k = cand_key(a);
  return k < th || (k == th && r <= tl);
}

// Per tile of kScanTile ids: how many replacements (keys <= T) it holds.
__global__ __launch_bounds__(kScanNT) void k_gsel_count(const float* __restrict__ S, const int32_t* __restrict__ rank_g,
                                                        int64_t n, const RoundState* __restrict__ rs,
                                                        int32_t* __restrict__ partials) {
  __shared__ int32_t lds[kScanNT / MS_WAVE + 1];
  const bool on = rs->k > 0;
  const uint32_t th = rs->prefix, tl = rs->prefix_lo;
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  int32_t c = 0;
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t g = base + (int64_t)it * kScanNT + threadIdx.x;
    if (on && g < n) {
      const float a = S[g];
      if (a >= 0.0f) c += gsel_in(a, (uint32_t)rank_g[g], th, tl);
    }
  }
  c = block_sum<kScanNT>(c, lds);
  if (threadIdx.x == 0) partials[blockIdx.x] = c;
}

// Emits the replacements in id order as (rank, halo id) pairs at the tile's
// prefix (partials scanned by k_scan_partials).
__global__ __launch_bounds__(kScanNT) void k_gsel_emit(const float* __restrict__ S, const int32_t* __restrict__ rank_g,
                                                       const int32_t* __restrict__ h_of_rank, int64_t n,
                                                       const RoundState* __restrict__ rs,
                                                       const int32_t* __restrict__ partials, uint32_t* __restrict__ keys,
                                                       int32_t* __restrict__ vals) {
  __shared__ int32_t lds[kScanNT / MS_WAVE + 1];
  if (rs->k == 0) return;
  const uint32_t th = rs->prefix, tl = rs->prefix_lo;
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  bool f[kScanItems];
  int32_t r[kScanItems];
  int32_t c = 0;
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t g = base + it;
    const float a = g < n ? S[g] : -1.0f;
    r[it] = a >= 0.0f ? rank_g[g] : 0;
    f[it] = gsel_in(a, (uint32_t)r[it], th, tl);
    c += f[it];
  }
  int32_t tot;
  int64_t o = (int64_t)block_exclusive_scan<kScanNT>(c, lds, &tot) + partials[blockIdx.x];
#pragma unroll
  for (int it = 0; it < kScanItems; ++it)
    if (f[it]) {
      keys[o] = (uint32_t)r[it];
      vals[o] = h_of_rank[r[it]];
      ++o;
    }
}

// After the sort by rank: each pair's key becomes its candidate key (the
// score word), for the stable sort that puts them in (score, rank) order.
__global__ void k_gsel_keys(const int32_t* __restrict__ vals, const int64_t* __restrict__ n_ptr,
                            const float* __restrict__ S, const int32_t* __restrict__ sa_idx,
                            uint32_t* __restrict__ keys) {
  const int64_t n = *n_ptr;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    keys[i] = cand_key(S[sa_idx[vals[i]]]);
}

// Scores by global id, at init: S_A[gid[h]] = 0 and rank_g[gid[h]] = rank of h
// for every halo node (the rest of both arrays was filled with -1).
__global__ void k_gid_init(const int32_t* __restrict__ gid, const int32_t* __restrict__ rank_of, int64_t H,
                           float* __restrict__ S, int32_t* __restrict__ rank_g) {
  for (int64_t h = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; h < H; h += (int64_t)gridDim.x * blockDim.x) {
    S[gid[h]] = 0.0f;
    rank_g[gid[h]] = rank_of[h];
  }
}

// Repeated global ids would share an S_A entry: after k_gid_init, an id whose
// rank entry is not its own halo node's rank was written twice.
__global__ void k_gid_check(const int32_t* __restrict__ gid, const int32_t* __restrict__ rank_of, int64_t H,
                            const int32_t* __restrict__ rank_g, int32_t* __restrict__ bad) {
  for (int64_t h = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; h < H; h += (int64_t)gridDim.x * blockDim.x)
    if (rank_g[gid[h]] != rank_of[h]) atomicOr(bad, 4);
}

// ------------------------------------------------------ stable radix sort
// LSD, 8 bits per pass, 2048 keys per block (256 threads x 8, striped so the
// stable order within a block is (item, wave, lane)). Digit-major block
// histograms are scanned into global offsets; ranks inside a block come from
// wave match masks (8 ballots) and per-wave digit counters in LDS.
constexpr int kSortNT = 256;
constexpr int kSortItems = 8;
constexpr int kSortTile = kSortNT * kSortItems;

__global__ __launch_bounds__(kSortNT) void k_sort_hist(const uint32_t* __restrict__ keys, const int64_t* __restrict__ n_ptr,
                                                       int64_t n_const, int64_t bound, int shift, int64_t nb,
                                                       int32_t* __restrict__ hist) {
  __shared__ int32_t h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int64_t n = min(size_of(n_ptr, n_const), bound);
  const int64_t base = (int64_t)blockIdx.x * kSortTile;
#pragma unroll
  for (int it = 0; it < kSortItems; ++it) {
    const int64_t i = base + (int64_t)it * kSortNT + threadIdx.x;
    if (i < n) atomicAdd(&h[(keys[i] >> shift) & 255u], 1);
  }
  __syncthreads();
  hist[(int64_t)threadIdx.x * nb + blockIdx.x] = h[threadIdx.x];
}

__global__ __launch_bounds__(kSortNT) void k_sort_scatter(const uint32_t* __restrict__ keys_in,
                                                          const int32_t* __restrict__ vals_in,
                                                          const int64_t* __restrict__ n_ptr, int64_t n_const,
                                                          int64_t bound, int shift, int64_t nb,
                                                          const int32_t* __restrict__ offs,
                                                          uint32_t* __restrict__ keys_out,
                                                          int32_t* __restrict__ vals_out) {
  constexpr int NW = kSortNT / MS_WAVE;
  __shared__ int32_t wcnt[NW][256];
  __shared__ int32_t running[256];
  __shared__ int32_t gbase[256];
  const int lane = lane_id(), wave = wave_id();
  for (int w = 0; w < NW; ++w) wcnt[w][threadIdx.x] = 0;
  running[threadIdx.x] = 0;
  gbase[threadIdx.x] = offs[(int64_t)threadIdx.x * nb + blockIdx.x];
  __syncthreads();
  const int64_t n = min(size_of(n_ptr, n_const), bound);
  const int64_t base = (int64_t)blockIdx.x * kSortTile;
  for (int it = 0; it < kSortItems; ++it) {
    const int64_t i = base + (int64_t)it * kSortNT + threadIdx.x;
    const bool valid = i < n;
    const uint32_t k = valid ? keys_in[i] : 0u;
    const int32_t val = valid ? vals_in[i] : 0;
    const uint32_t dgt = (k >> shift) & 255u;
    uint64_t peers = ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const uint64_t m = ballot((dgt >> b) & 1u);
      peers &= ((dgt >> b) & 1u) ? m : ~m;
    }
    const int below = lanes_below(peers);
    const bool leader = valid && ((peers >> lane) >> 1) == 0ull;  // highest lane of its digit
    if (leader) wcnt[wave][dgt] = below + 1;
    __syncthreads();
    if (valid) {
      int32_t r = running[dgt] + below;
      for (int w = 0; w < wave; ++w) r += wcnt[w][dgt];
      const int64_t dst = (int64_t)gbase[dgt] + r;
      keys_out[dst] = k;
      vals_out[dst] = val;
    }
    __syncthreads();
    {
      int32_t add = 0;
      for (int w = 0; w < NW; ++w) {
        add += wcnt[w][threadIdx.x];
        wcnt[w][threadIdx.x] = 0;
      }
      running[threadIdx.x] += add;
    }
    __syncthreads();
  }
}

// Generic exclusive scan of an int32 array with host-known length.
__global__ __launch_bounds__(kScanNT) void k_tile_reduce(const int32_t* __restrict__ a, int64_t len,
                                                         int32_t* __restrict__ partials) {
  __shared__ int32_t lds[kScanNT / MS_WAVE + 1];
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  int32_t s = 0;
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t i = base + (int64_t)it * kScanNT + threadIdx.x;
    if (i < len) s += a[i];
  }
  s = block_sum<kScanNT>(s, lds);
  if (threadIdx.x == 0) partials[blockIdx.x] = s;
}

__global__ __launch_bounds__(kScanNT) void k_tile_scan(int32_t* __restrict__ a, int64_t len,
                                                       const int32_t* __restrict__ partials) {
  __shared__ int32_t lds[kScanNT / MS_WAVE + 1];
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  int32_t v[kScanItems];
  int32_t s = 0;
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    v[it] = base + it < len ? a[base + it] : 0;
    s += v[it];
  }
  int32_t tot;
  int32_t ex = block_exclusive_scan<kScanNT>(s, lds, &tot) + partials[blockIdx.x];
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    if (base + it < len) a[base + it] = ex;
    ex += v[it];
  }
}

// ---------------------------------------------------------- key builders
// rank keys: low word = global id, high word = ~degree (degree desc).
__global__ void k_rank_keys_lo(const int32_t* __restrict__ gid, int64_t H, uint32_t* __restrict__ keys,
                               int32_t* __restrict__ vals) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < H; i += (int64_t)gridDim.x * blockDim.x) {
    keys[i] = (uint32_t)gid[i] ^ 0x80000000u;  // signed order as unsigned
    vals[i] = (int32_t)i;
  }
}
__global__ void k_rank_keys_hi(const int64_t* __restrict__ deg, const int32_t* __restrict__ vals, int64_t H,
                               uint32_t* __restrict__ keys) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < H; i += (int64_t)gridDim.x * blockDim.x) {
    int64_t d = deg[vals[i]];
    if (d < 0) d = 0;
    if (d > 0xFFFFFFFFll) d = 0xFFFFFFFFll;
    keys[i] = ~(uint32_t)d;
  }
}
__global__ void k_rank_finish(const int32_t* __restrict__ h_of_rank, int64_t H, int32_t* __restrict__ rank_of) {
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < H; r += (int64_t)gridDim.x * blockDim.x)
    rank_of[h_of_rank[r]] = (int32_t)r;
}

// Initial buffer: slot s holds the halo node of rank s.
__global__ void k_init_buffer(const int32_t* __restrict__ h_of_rank, int64_t cap, int32_t L,
                              int32_t* __restrict__ slot_id, float* __restrict__ S_E, int32_t* __restrict__ hitcnt,
                              float* __restrict__ S_A, const int32_t* __restrict__ sa_idx, int2* __restrict__ fill) {
  for (int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; s < cap; s += (int64_t)gridDim.x * blockDim.x) {
    const int32_t h = h_of_rank[s];
    slot_id[s] = h;
    S_E[s] = 1.0f;
    hitcnt[s] = 0;
    S_A[sa_idx[h]] = -1.0f;
    fill[s] = make_int2((int32_t)(L + s), h);
  }
}

// E-selection keys (only when fewer candidates than evictions):
// low = rank of the slot's node, high = fp32 bits of S_E (S_E >= 0).
__global__ void k_esel_keys_lo(const int32_t* __restrict__ E, const int64_t* __restrict__ n_ptr,
                               const int32_t* __restrict__ slot_id, const int32_t* __restrict__ rank_of,
                               uint32_t* __restrict__ keys, int32_t* __restrict__ vals) {
  const int64_t n = *n_ptr;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    keys[i] = (uint32_t)rank_of[slot_id[E[i]]];
    vals[i] = E[i];
  }
}
__global__ void k_esel_keys_hi(const int32_t* __restrict__ vals, const int64_t* __restrict__ n_ptr,
                               const float* __restrict__ S_E, uint32_t* __restrict__ keys) {
  const int64_t n = *n_ptr;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    keys[i] = __float_as_uint(S_E[vals[i]]);
}
__global__ void k_esel_keys_slot(const int32_t* __restrict__ vals, const int64_t* __restrict__ n_ptr,
                                 uint32_t* __restrict__ keys) {
  const int64_t n = *n_ptr;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    keys[i] = (uint32_t)vals[i];
}

// ------------------------------------------------------------------ swap
// Pair E[i] (ascending slot) with R[i]; every read sees pre-round values
// because the slots, the evicted nodes and the replacements are all
// distinct, so no two threads touch the same entry. S_A is reached through
// each node's S_A index (its rank, or its global id).
__global__ void k_swap(const int32_t* __restrict__ E, const int32_t* __restrict__ R, const int64_t* __restrict__ k_ptr,
                       int32_t L, int64_t cap, int32_t H, int32_t* __restrict__ slot_id, float* __restrict__ S_E,
                       float* __restrict__ S_A, const int32_t* __restrict__ sa_idx,
                       int32_t* __restrict__ out_ev, int32_t* __restrict__ out_slot,
                       int32_t* __restrict__ out_rep, int2* __restrict__ fill, int32_t* __restrict__ bad,
                       int32_t* __restrict__ slot_round, int32_t round_id) {
  const int64_t k = *k_ptr;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < k; i += (int64_t)gridDim.x * blockDim.x) {
    const int32_t s = E[i], r = R[i];
    if (s < 0 || s >= cap || r < 0 || r >= H) {  // never expected: flag, do not touch memory
      atomicOr(bad, 1);
      fill[i] = make_int2(-1, -1);
      continue;
    }
    const int32_t e = slot_id[s];
    const int32_t re = sa_idx[e], rr = sa_idx[r];
    const float se = S_E[s], sa = S_A[rr];
    S_A[re] = se;
    S_E[s] = sa;
    S_A[rr] = -1.0f;
    slot_id[s] = r;
    slot_round[s] = round_id;
    if (out_ev) out_ev[i] = e;
    if (out_slot) out_slot[i] = s;
    if (out_rep) out_rep[i] = r;
    fill[i] = make_int2((int32_t)(L + s), r);
  }
}

}  // namespace ms

namespace ms {
// G_p sanity: non-decreasing offsets, column ids inside [0, R).
__global__ void k_validate_csr(const int64_t* __restrict__ indptr, int64_t R, const int32_t* __restrict__ indices,
                               int64_t nnz, int32_t* __restrict__ bad) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < R; i += stride)
    if (indptr[i + 1] < indptr[i]) atomicOr(bad, 1);
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < nnz; e += stride) {
    const int32_t v = indices[e];
    if (v < 0 || v >= R) atomicOr(bad, 2);
  }
}
}  // namespace ms
