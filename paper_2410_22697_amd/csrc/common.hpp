// common.hpp - device utilities for libmassive (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define MS_WAVE 64

namespace ms {

__device__ __forceinline__ int lane_id() { return threadIdx.x & (MS_WAVE - 1); }
__device__ __forceinline__ int wave_id() { return threadIdx.x / MS_WAVE; }

// number of set bits of `mask` in lanes below this one
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

// A value the caller knows to be the same in every lane of the wave, moved to
// a scalar register, so that branches on it are scalar and loads through it
// are scalar loads.
__device__ __forceinline__ int32_t wave_uniform(int32_t x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ int64_t wave_uniform(int64_t x) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)(uint32_t)x);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)(uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Inclusive prefix sum over the 64 lanes of a wave.
template <typename T>
__device__ __forceinline__ T wave_inclusive_scan(T x) {
  const int lane = lane_id();
#pragma unroll
  for (int o = 1; o < MS_WAVE; o <<= 1) {
    T y = __shfl_up(x, o, MS_WAVE);
    if (lane >= o) x += y;
  }
  return x;
}

// Keeps a loaded value where it is: an empty asm that reads and writes it.
// Loads whose values are only used under a per-lane condition are otherwise
// sunk by the compiler into that condition, each behind its own wait, so the
// loads of a thread would be issued one at a time.
template <typename T>
__device__ __forceinline__ void pin(T& x) {
  asm volatile("" : "+v"(x));
}

template <typename T>
__device__ __forceinline__ T wave_sum(T x) {
#pragma unroll
  for (int o = MS_WAVE / 2; o > 0; o >>= 1) x += __shfl_xor(x, o, MS_WAVE);
  return x;
}

// Exclusive prefix sum over a block of NT threads; lds needs NT/64 + 1 slots.
// Returns this thread's exclusive prefix; *total gets the block sum.
template <int NT, typename T>
__device__ __forceinline__ T block_exclusive_scan(T v, T* lds, T* total) {
  constexpr int NW = NT / MS_WAVE;
  const int lane = lane_id(), wave = wave_id();
  T x = wave_inclusive_scan(v);
  if (lane == MS_WAVE - 1) lds[wave] = x;
  __syncthreads();
  if (wave == 0) {
    T w = lane < NW ? lds[lane] : T(0);
    T wi = wave_inclusive_scan(w);
    if (lane < NW) lds[lane] = wi - w;
    if (lane == NW - 1) lds[NW] = wi;
  }
  __syncthreads();
  T res = lds[wave] + x - v;
  *total = lds[NW];
  __syncthreads();
  return res;
}

template <int NT, typename T>
__device__ __forceinline__ T block_sum(T v, T* lds) {
  T total;
  (void)block_exclusive_scan<NT>(v, lds, &total);
  return total;
}

// a ^ b ^ key in one instruction: gfx950's three-input bitwise operation
// (truth table 0x96 = XOR of all three); key is wave-uniform (an SGPR, the
// one scalar operand the instruction may take).
__device__ __forceinline__ uint32_t xor3_key(uint32_t a, uint32_t b, uint32_t key) {
  uint32_t r;
  asm("v_bitop3_b32 %0, %1, %2, %3 bitop3:0x96" : "=v"(r) : "v"(a), "v"(b), "s"(key));
  return r;
}

// Philox4x32-10 block function (Salmon, Moraes, Dror, Shaw, SC'11): ten
// rounds; each round takes the 64-bit products of counter words 0 and 2
// with two fixed multipliers, mixes their high halves with words 1 and 3
// and the round key, and the key advances by two Weyl constants per round.
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t a = (uint64_t)0xD2511F53u * c.x;
    const uint64_t b = (uint64_t)0xCD9E8D57u * c.z;
    const uint4 n = make_uint4((uint32_t)(b >> 32) ^ c.y ^ k0, (uint32_t)b,
                               (uint32_t)(a >> 32) ^ c.w ^ k1, (uint32_t)a);
    c = n;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

__device__ __forceinline__ uint32_t word_of(const uint4& w, int s) {
  return s == 0 ? w.x : (s == 1 ? w.y : (s == 2 ? w.z : w.w));
}

// Device-side sizes of the current step (one struct in HBM per context).
struct StepSizes {
  int64_t n[9];      // frontier sizes n_0..n_K
  int64_t e[8];      // sampled edges per hop
  int64_t local, hits, misses;
  int64_t n_hbm, n_miss;  // lengths of the two gather lists
  int64_t n_big[8];       // rows longer than the big-row threshold, per hop
  int64_t n_small[8];     // the other rows, when they are listed too (one-wave-per-row sampler)
  int64_t n_local_new[8]; // new frontier nodes below L (local), per hop
  int64_t n_pending;      // hits on slots still refilling (read over the host link)
  int32_t status;    // != 0: invalid seeds; later kernels of the step skip
  int32_t blocks_done;  // blocks of the step's miss gather that have finished
};

// Eviction-round device scalars.
struct RoundState {
  int64_t nE, nC;          // |E|, |C|
  int64_t k;               // k' = min(|E|, |C|)
  int64_t need;            // ties at the threshold still to take
  uint32_t prefix, pmask;  // radix-select prefix of the threshold key (S_A word)
  uint32_t prefix_lo, pmask_lo;  // ... and of its rank word (scores by global id)
  int64_t n_lt, n_eq;      // candidates strictly before / equal to the threshold
  int64_t nE_sel, k_sel;   // |E| and k' when k' < |E| (E must be narrowed), else 0
};

// Totals over the context's life (device side).
struct Counters {
  int64_t rounds;          // rounds that evicted at least one slot
  int64_t evicted;         // slots evicted (= rows refilled)
  int32_t bad;             // some round produced inconsistent indices (never expected)
  int32_t pad;
  int64_t refilled;        // rows the refill copied over the host link (slots
                           // written through by a miss gather are not copied)
};

}  // namespace ms
