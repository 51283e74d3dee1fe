// sample_kernels.hpp - fanout sampling, frontier dedup and relabel (one hop
// of the NeighborSampler of Algorithm 2, DGL block convention).
#pragma once

#include "common.hpp"

namespace ms {

constexpr int kScanNT = 1024;       // threads per scan block
constexpr int kScanItems = 4;       // items per thread
constexpr int kScanTile = kScanNT * kScanItems;

__device__ __forceinline__ int64_t size_of(const int64_t* p, int64_t c) { return p ? *p : c; }

// ---------------------------------------------------------------- seeds
// F_0 = seeds; pos_of[seed] = its position. Flags out-of-range or repeated
// seeds in sz->status (the step is then abandoned by every later kernel).
__global__ void k_seed_init(const int32_t* __restrict__ seeds, int32_t n0, int32_t L,
                            int32_t* __restrict__ nodes, int32_t* __restrict__ pos_of,
                            StepSizes* sz) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) sz->n[0] = n0;
  if (i >= n0) return;
  const int32_t v = seeds[i];
  if (v < 0 || v >= L) {
    atomicOr(&sz->status, 1);
    return;
  }
  const int32_t prev = atomicCAS(&pos_of[v], -1, i);
  if (prev != -1) atomicOr(&sz->status, 2);
  nodes[i] = v;
}

// Undo k_seed_init's pos_of marks after a failed validation.
__global__ void k_seed_undo(const int32_t* __restrict__ seeds, int32_t n0, int32_t L,
                            int32_t* __restrict__ pos_of) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n0) return;
  const int32_t v = seeds[i];
  if (v >= 0 && v < L) pos_of[v] = -1;
}

// ------------------------------------------------------ per-row counts + scan
// Block b: sum over its tile of min(deg(F[i]), fo); counts go to out[i+1].
__global__ __launch_bounds__(kScanNT) void k_row_counts(const int64_t* __restrict__ csr_indptr,
                                                        const int32_t* __restrict__ nodes,
                                                        const StepSizes* sz, int hop, int32_t fo,
                                                        int32_t* __restrict__ bptr,
                                                        int32_t* __restrict__ partials) {
  __shared__ int32_t lds[kScanNT / MS_WAVE + 1];
  if (sz->status) return;
  const int64_t n = sz->n[hop - 1];
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  int32_t s = 0;
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t i = base + (int64_t)it * kScanNT + threadIdx.x;
    if (i < n) {
      const int32_t v = nodes[i];
      const int64_t d = csr_indptr[v + 1] - csr_indptr[v];
      const int32_t c = d < fo ? (int32_t)d : fo;
      bptr[i + 1] = c;
      s += c;
    }
  }
  s = block_sum<kScanNT>(s, lds);
  if (threadIdx.x == 0) partials[blockIdx.x] = s;
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

// bptr[1..n] holds counts; turn bptr[0..n] into exclusive offsets.
__global__ __launch_bounds__(kScanNT) void k_row_offsets(const StepSizes* sz, int hop,
                                                         int32_t* __restrict__ bptr,
                                                         const int32_t* __restrict__ partials) {
  __shared__ int32_t lds[kScanNT / MS_WAVE + 1];
  if (sz->status) return;
  const int64_t n = sz->n[hop - 1];
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  int32_t v[kScanItems];
  int32_t s = 0;
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t i = base + it;
    v[it] = i < n ? bptr[i + 1] : 0;
    s += v[it];
  }
  int32_t tot;
  int32_t ex = block_exclusive_scan<kScanNT>(s, lds, &tot) + partials[blockIdx.x];
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    const int64_t i = base + it;
    ex += v[it];
    if (i < n) bptr[i + 1] = ex;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) bptr[0] = 0;
}

// --------------------------------------------------------------- sampler
// One wavefront per frontier node. Rows with d <= fanout are copied. For
// longer rows the choice is the fanout positions of smallest (key, j):
//   - d <= 256: lane q draws one Philox block = keys of positions 4q..4q+3;
//   - longer rows: a threshold pass keeps (in ascending j, in LDS) every
//     position whose key is below tau, tau picked so that about 2*fanout+16
//     survive (bisection if fewer than fanout or more than 256 survive);
// then a 32-step bitwise search over ballots finds the fanout-th smallest
// key T, ties at T are broken by list order (= ascending j), and the chosen
// positions are written in ascending j.
constexpr int kSampleWaves = 4;
constexpr int kCandCap = 256;

struct SampleArgs {
  const int64_t* csr_indptr;
  const int32_t* csr_indices;
  const int32_t* nodes;
  const StepSizes* sz;
  const int32_t* bptr;
  int32_t* out;
  int32_t hop;  // 1-based
  int32_t fo;
  uint32_t t;
  uint32_t key0, key1;
  int32_t* err;  // threshold search could not isolate a candidate set
};

__global__ __launch_bounds__(kSampleWaves* MS_WAVE) void k_sample(SampleArgs a) {
  __shared__ uint64_t cand[kSampleWaves][kCandCap];
  if (a.sz->status) return;
  const int lane = lane_id(), wave = wave_id();
  const int64_t row = (int64_t)blockIdx.x * kSampleWaves + wave;
  const int64_t n = a.sz->n[a.hop - 1];
  if (row >= n) return;
  const int32_t v = a.nodes[row];
  const int64_t start = a.csr_indptr[v];
  const int64_t d = a.csr_indptr[v + 1] - start;
  const int32_t fo = a.fo;
  int32_t* out = a.out + a.bptr[row];
  const int32_t* nb = a.csr_indices + start;
  if (d <= fo) {
    for (int64_t j = lane; j < d; j += MS_WAVE) out[j] = nb[j];
    return;
  }
  const uint32_t uv = (uint32_t)v, ut = a.t, uk = (uint32_t)a.hop;
  // list element (lane, s) has list index 4*lane + s
  uint32_t key[4], pos[4];
  bool valid[4];
  if (d <= 4 * MS_WAVE) {
    const uint4 w = philox4x32_10(make_uint4((uint32_t)lane, uv, ut, uk), a.key0, a.key1);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int64_t j = 4 * lane + s;
      valid[s] = j < d;
      key[s] = word_of(w, s);
      pos[s] = (uint32_t)j;
    }
  } else {
    uint64_t* c = cand[wave];
    const uint64_t full = 1ull << 32;
    uint64_t tau = ((uint64_t)(2 * fo + 16) << 32) / (uint64_t)d + 1;
    if (tau > full) tau = full;
    uint64_t lo = 0, hi = full + 1;  // known: count(lo) < fo; count(hi) > cap (hi unknown: full+1)
    int cnt = 0;
    bool ok = false;
    for (int iter = 0; iter < 48 && !ok; ++iter) {
      cnt = 0;
      for (int64_t q0 = 0; 4 * q0 < d; q0 += MS_WAVE) {
        const int64_t q = q0 + lane;
        const uint4 w = philox4x32_10(make_uint4((uint32_t)q, uv, ut, uk), a.key0, a.key1);
        bool take[4];
        uint64_t m[4];
        int mine = 0;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          take[s] = (4 * q + s < d) && ((uint64_t)word_of(w, s) < tau);
          m[s] = ballot(take[s]);
        }
        int below = lanes_below(m[0]) + lanes_below(m[1]) + lanes_below(m[2]) + lanes_below(m[3]);
        const int total = __popcll(m[0]) + __popcll(m[1]) + __popcll(m[2]) + __popcll(m[3]);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          if (take[s]) {
            const int p = cnt + below + mine;
            if (p < kCandCap) c[p] = ((uint64_t)word_of(w, s) << 32) | (uint32_t)(4 * q + s);
            ++mine;
          }
        }
        cnt += total;
      }
      if (cnt < fo) {
        lo = tau;
        tau = (hi > full) ? (tau * 4 > full ? full : tau * 4) : (lo + hi) / 2;
      } else if (cnt > kCandCap) {
        hi = tau;
        tau = (lo + hi) / 2;
      } else {
        ok = true;
      }
      if (!ok && hi <= full && hi - lo <= 1) break;
    }
    if (!ok) {
      if (lane == 0) atomicOr(a.err, 1);
      return;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int idx = 4 * lane + s;
      valid[s] = idx < cnt;
      const uint64_t e = valid[s] ? c[idx] : 0ull;
      key[s] = (uint32_t)(e >> 32);
      pos[s] = (uint32_t)e;
    }
  }
  // T = largest x with count(key < x) < fo, i.e. the fo-th smallest key
  uint32_t T = 0;
  for (int b = 31; b >= 0; --b) {
    const uint32_t trial = T | (1u << b);
    int c = 0;
#pragma unroll
    for (int s = 0; s < 4; ++s) c += __popcll(ballot(valid[s] && key[s] < trial));
    if (c < fo) T = trial;
  }
  uint64_t lt[4], eq[4];
  int n_lt = 0;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    lt[s] = ballot(valid[s] && key[s] < T);
    eq[s] = ballot(valid[s] && key[s] == T);
    n_lt += __popcll(lt[s]);
  }
  const int need = fo - n_lt;
  // rank among ties in list order, then the selection mask
  int eq_below = lanes_below(eq[0]) + lanes_below(eq[1]) + lanes_below(eq[2]) + lanes_below(eq[3]);
  bool sel[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const bool is_eq = (eq[s] >> lane) & 1ull;
    sel[s] = ((lt[s] >> lane) & 1ull) || (is_eq && eq_below < need);
    if (is_eq) ++eq_below;
  }
  uint64_t sm[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) sm[s] = ballot(sel[s]);
  int p = lanes_below(sm[0]) + lanes_below(sm[1]) + lanes_below(sm[2]) + lanes_below(sm[3]);
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    if (sel[s]) {
      out[p] = nb[pos[s]];
      ++p;
    }
  }
}

// ------------------------------------------------------------ dedup/relabel
// Mark every sampled id not yet in the frontier in a bitmap over [0, L+H).
__global__ void k_mark_new(const int32_t* __restrict__ ids, const StepSizes* sz, int hop,
                           const int32_t* __restrict__ pos_of, uint32_t* __restrict__ bits) {
  if (sz->status) return;
  const int64_t e = sz->e[hop - 1];
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < e;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int32_t u = ids[i];
    if (pos_of[u] < 0) {
      const uint32_t bit = 1u << (u & 31);
      if (!(bits[u >> 5] & bit)) atomicOr(&bits[u >> 5], bit);
    }
  }
}

// Per-block popcount of the bitmap tile.
__global__ __launch_bounds__(kScanNT) void k_bits_count(const uint32_t* __restrict__ bits, int64_t W,
                                                        const StepSizes* sz,
                                                        int32_t* __restrict__ partials) {
  __shared__ int32_t lds[kScanNT / MS_WAVE + 1];
  if (sz->status) return;
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  int32_t s = 0;
  if (base + kScanItems <= W) {
    const uint4 w4 = *reinterpret_cast<const uint4*>(bits + base);
    s = __popc(w4.x) + __popc(w4.y) + __popc(w4.z) + __popc(w4.w);
  } else {
    for (int it = 0; it < kScanItems; ++it)
      if (base + it < W) s += __popc(bits[base + it]);
  }
  s = block_sum<kScanNT>(s, lds);
  if (threadIdx.x == 0) partials[blockIdx.x] = s;
}

// New nodes in ascending id: F[n_{k-1} + rank] = u, pos_of[u] = that
// position; the bitmap is cleared for the next hop.
__global__ __launch_bounds__(kScanNT) void k_bits_emit(uint32_t* __restrict__ bits, int64_t W,
                                                       const StepSizes* sz, int hop,
                                                       const int32_t* __restrict__ partials,
                                                       int32_t* __restrict__ nodes,
                                                       int32_t* __restrict__ pos_of) {
  __shared__ int32_t lds[kScanNT / MS_WAVE + 1];
  if (sz->status) return;
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  uint32_t w[kScanItems];
  int32_t s = 0;
#pragma unroll
  for (int it = 0; it < kScanItems; ++it) {
    w[it] = base + it < W ? bits[base + it] : 0u;
    s += __popc(w[it]);
  }
  int32_t tot;
  int64_t off = (int64_t)block_exclusive_scan<kScanNT>(s, lds, &tot) + partials[blockIdx.x] +
                sz->n[hop - 1];
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
}

// Relabel sampled ids to their frontier positions.
__global__ void k_relabel(int32_t* __restrict__ ids, const StepSizes* sz, int hop,
                          const int32_t* __restrict__ pos_of) {
  if (sz->status) return;
  const int64_t e = sz->e[hop - 1];
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < e;
       i += (int64_t)gridDim.x * blockDim.x)
    ids[i] = pos_of[ids[i]];
}

}  // namespace ms
