// massive.hip - libmassive: the C ABI of include/massive.h on one MI355X.
//
// Streams: a step's sampling and classify run on the caller's stream
// ("main"); its HBM gather, its miss gather from pinned host memory and its
// completion kernel follow on a side stream, so the main stream goes on to the
// next step at once; eviction rounds and their refill copies run on a copy
// stream (the refill chunks and the HBM gathers wait for each other, and the
// next classify waits for a round).
// In the staged link mode no kernel reads host memory: a worker thread of the
// context gathers each step's host rows and each refill chunk's rows into a
// pinned ring (with a pool of host threads), copies them with the DMA engines
// on a link stream, and enqueues the scatter kernels and the step's
// completion there.
// All device memory is allocated in massive_init; the per-step calls do not
// allocate.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <condition_variable>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cmath>
#include <cstring>
#include <deque>
#include <exception>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "../../include/massive.h"
#include "buffer_kernels.hpp"
#include "common.hpp"
#include "gather_pool.hpp"
#include "sample_kernels.hpp"

namespace {

thread_local std::string g_init_error;

struct TimedRange {
  hipEvent_t a, b;
  int group;
};

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline unsigned grid_for(int64_t n, int nt, int64_t cap = 16384) {
  int64_t g = cdiv(std::max<int64_t>(n, 1), nt);
  return (unsigned)std::min<int64_t>(std::max<int64_t>(g, 1), cap);
}

}  // namespace

// ------------------------------------------------------------- no-alloc path
// massive_sample_noalloc takes a step's per-step buffers (sizes, the two
// gather lists, the write-through slots, the sampler's row list, the scan flags)
// from this file-scope array instead of the context's. Layout: StepSizes
// (512 B) | hbm list int2[kNoAllocMaxRows] | miss list int2[..] | write-through
// slots int32[..] | big rows int32[..] | scan flags uint64[kNoAllocFlagWords].
// Each GPU holds its own copy (~30 MiB) while the library is loaded; its device
// address is looked up once per device, in massive_init.
constexpr int64_t kNoAllocMaxRows = 1310720;  // frontier rows (covers a 1,081,344-row bound)
constexpr int64_t kNoAllocFlagWords = (int64_t(1) << 31) / 32 / ms::kScanTile + 2;  // any L + H < 2^31
constexpr int64_t kNoAllocBytes = 512 + kNoAllocMaxRows * (8 + 8 + 4 + 4) + kNoAllocFlagWords * 8;
static_assert(sizeof(ms::StepSizes) <= 512, "sizes fit the first 512 bytes");
static __device__ __align__(256) uint8_t scratch[kNoAllocBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};  // device address of `scratch` on each device, once looked up

// The device address of `scratch` on device dev, which must be current: the
// array's name in host code is a host-side stand-in, not a device address.
hipError_t scratch_address(int dev, void** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!ptr) return hipErrorInvalidSymbol;
    g_scratch_addr[dev] = ptr;
  }
  *out = g_scratch_addr[dev];
  return hipSuccess;
}
}  // namespace

constexpr int kSlots = MASSIVE_MAX_INFLIGHT;
// host-row bytes of a step above which its miss gather takes the larger grid
// (at ~50 GB/s, ~0.5 ms of link time: about a sampling pass of the largest
// workloads)
constexpr int64_t kLinkHeavyBytes = 24ll << 20;
constexpr int kTimingGroups = 7;  // bits of MASSIVE_TIMING_ALL

struct massive_ctx {
  // configuration
  int32_t L = 0, H = 0;
  int64_t R = 0, nnz = 0, rb = 0;
  int32_t K = 0;
  int32_t fo[MASSIVE_MAX_HOPS] = {};
  int32_t pct = 0;
  float gamma = 1.0f;
  int32_t delta = 1;
  uint64_t seed = 0;
  int64_t cap = 0, hcap = 0;
  uint32_t hmask = 0;
  float alpha = 1.0f;
  int64_t W = 0;        // bitmap words
  int64_t pmax = 0;     // partials capacity
  int64_t sort_cap = 0; // radix sort capacity
  int64_t hbm_blocks = 4096;  // grid bound of the HBM gather
  // Grid of the miss gather (host link). Its reads hold memory-system
  // resources for the whole link latency and slow the sampling beside them,
  // so a step whose host-link work is light takes the smaller grid; a step
  // that may be bound by the link (a refill in flight, or many host rows in
  // the last step waited for) takes the larger one.
  int64_t host_blocks = 16;
  int64_t host_blocks_light = 12;
  int64_t host_rows_seen = -1;  // host rows of the last step waited for (-1: none yet)
  bool slot_clear[MASSIVE_MAX_INFLIGHT] = {};  // the slot's sizes were cleared by its last step's miss gather
  int64_t refill_blocks = 16; // grid of the refill (host link, off the critical path)
  double mu32[MASSIVE_MAX_HOPS] = {};    // sampler threshold targets, x 2^32
  int32_t* d_big = nullptr;             // row list of the current hop (long rows first)
  int64_t big_min = ms::kBigRow;        // rows longer than this are sampled by a whole block
  int64_t big_blocks = ms::kBigBlocks;  // blocks that walk the list of such rows
  int32_t tau_iters = ms::kTauIters;    // threshold passes per row (0 makes every long row fail)
  // streams and events
  hipStream_t s_main = nullptr, s_miss = nullptr, s_copy = nullptr;
  // Staged host link (MASSIVE_LINK_STAGED). The worker thread takes jobs in
  // order: a step's tail (its host rows gathered, copied and scattered, then
  // the completion kernel and ev_batch_done, all on s_link) or one refill
  // chunk (gathered, copied, scattered; the round's last chunk records
  // ev_fill_done). Its ring entries and pool belong to it alone; the job queue
  // and its progress are shared under lmu.
  struct LinkJob {
    bool refill = false;
    int slot = 0;
    int64_t step = 0;
    const int2* list = nullptr;     // a step: its miss list, write-through slots and output rows
    const int32_t* wslot = nullptr;
    uint8_t* feat = nullptr;
    ms::StepSizes* sz = nullptr;
    int32_t pend = -1;              // the completion kernel's landed round (-1: none)
    int64_t nbK = 0;                // frontier bound
    bool rows = false;              // the step has host rows (H > 0)
    int32_t round_id = 0, chunk = 0, nchunks = 1;  // a refill chunk
    int timing = 0;                 // timing groups on when the job was posted
  };
  static constexpr int kRing = 4;  // staging ring entries
  int64_t ring_bytes = 8 << 20;     // bytes per entry (at least one row)
  int link_mode = MASSIVE_LINK_LOADS;
  int link_threads = 8;
  hipStream_t s_link = nullptr;
  const uint8_t* h_store = nullptr;   // host address of the pinned store
  int32_t* h_rows[kSlots] = {};       // pinned [H]: host rows of each slot's miss list
  int32_t* hd_rows[kSlots] = {};      //   (device views)
  int32_t* h_fill_rows = nullptr;     // pinned [cap]: host rows of the fill list
  int32_t* hd_fill_rows = nullptr;
  int64_t* h_cnt = nullptr;           // pinned [kSlots + 1]: miss count by slot, then the fill count
  int64_t* hd_cnt = nullptr;
  uint8_t* h_ring = nullptr;          // pinned [kRing][ring_rows * rb]
  uint8_t* d_ring = nullptr;          // device [kRing][ring_rows * rb]
  int64_t ring_rows = 0;
  hipEvent_t ev_rows_ready[kSlots] = {};  // a slot's host rows are in h_rows (side stream)
  hipEvent_t ev_fill_ready = nullptr;     // the round's fill rows are in h_fill_rows (copy stream)
  hipEvent_t ev_fill_done = nullptr;      // the last refill chunk's scatter (link stream)
  hipEvent_t ev_ring[kRing] = {};         // each ring entry's last scatter
  bool ring_used[kRing] = {};
  int ring_next = 0;
  ms::GatherPool* pool = nullptr;
  std::thread worker;
  std::mutex lmu;
  std::condition_variable lcv;
  std::deque<LinkJob> ljobs;
  bool lstop = false, lbusy = false, lfailed = false;
  std::string lerr;
  int64_t tail_step = -1;        // last step whose tail the worker has enqueued
  int32_t fill_done_round = 0;   // last round whose refill chunks it has all enqueued
  std::vector<hipEvent_t> lev_pool;  // the worker's timing events
  std::vector<TimedRange> lpending;
  bool staged() const { return link_mode == MASSIVE_LINK_STAGED; }
  // per step slot (step t uses slot t % MASSIVE_MAX_INFLIGHT): classify done
  // (main), HBM gather done and miss gather + mailbox done (side)
  hipEvent_t ev_cls_done[kSlots] = {}, ev_hbm_done[kSlots] = {}, ev_batch_done[kSlots] = {};
  hipEvent_t ev_round_done = nullptr, ev_refill_done = nullptr;
  bool round_unclassified = false;  // a round was enqueued that no classify has waited for yet
  // The refill of the last round is copied in chunks, one after each of the
  // next steps' HBM gathers (host-link reads never overlap an HBM gather).
  int32_t round_id = 0;          // rounds so far, as stamped in slot_round / landed
  int32_t refill_chunks = 1;     // chunks per round: min(delta - 1, 32), one per step of the interval
  int32_t chunks_left = 0;       // chunks of round_id's refill not yet launched
  bool refill_inflight = false;  // a launched chunk may not have landed
  bool round_pending_rows = false;  // round_id's refill not fully landed (hits may need the host)
  // device memory
  int64_t* d_indptr = nullptr;
  int32_t* d_indices = nullptr;
  uint8_t* d_slab = nullptr;          // [(L + cap) * rb]: local rows, then buffer rows
  const uint8_t* d_store = nullptr;   // device view of the pinned halo store
  int32_t* d_slot_id = nullptr;
  float* d_S_E = nullptr;
  int32_t* d_hitcnt = nullptr;
  float* d_S_A = nullptr;
  int32_t* d_rank_of = nullptr;
  int32_t* d_h_of_rank = nullptr;
  // S_A layout: by rank (H entries; a node's S_A index is its rank) or by
  // global id (n_global entries; its index is its global id, and rank_g gives
  // the rank of the halo node with each id)
  int32_t layout = MASSIVE_SCORES_BY_RANK;
  int64_t n_sa = 0;                  // entries of S_A
  const int32_t* d_sa_idx = nullptr; // [H] S_A index of halo h (d_rank_of or d_gid)
  int32_t* d_gid = nullptr;          // [H] global id of halo h
  int32_t* d_rank_g = nullptr;       // [n_global] by global id: rank of that halo node, -1 elsewhere
  int32_t* d_gpart = nullptr;        // tile partials of the global-id selection
  int64_t* d_deg = nullptr;          // [H] degrees, during init only
  uint64_t* d_tab = nullptr;
  int32_t* d_pos_of = nullptr;
  uint32_t* d_bits = nullptr;
  ms::StepSizes* d_sz = nullptr;      // [kSlots], by step slot
  ms::StepSizes* h_sz = nullptr;      // [kSlots] pinned mailboxes
  int32_t* h_bad = nullptr;           // [kSlots] pinned: eviction-round consistency flag
  ms::StepSizes* hd_sz = nullptr;     // device views of the mailboxes
  int32_t* hd_bad = nullptr;
  ms::RoundState* d_rs = nullptr;
  ms::RoundState* h_rs = nullptr;     // pinned mailbox
  ms::Counters* d_ctr = nullptr;
  ms::Counters* h_ctr = nullptr;      // pinned
  int32_t* d_slot_round = nullptr;    // [cap] round whose swap last filled the slot
  int32_t* d_landed = nullptr;        // [cap] round whose refill row has landed
  int32_t* d_part = nullptr;
  int32_t* d_part2 = nullptr;
  uint64_t* d_scan_flags = nullptr;  // the sampler's single-pass scans (rounds use d_part, d_part2)
  int64_t scan_tiles = 0;
  uint32_t scan_epoch = 0;           // of the last scan launched
  // gather lists by step slot (written by classify, read by the side stream)
  int2* d_hbm_list[kSlots] = {};
  int2* d_miss_list[kSlots] = {};
  int32_t* d_miss_slot[kSlots] = {};  // per miss-list entry: write-through slot or -1
  uint8_t* d_dummy = nullptr;         // [row_bytes] row that idle copy lanes move onto itself
  int32_t* d_E = nullptr;
  int32_t* d_R = nullptr;
  int2* d_fill = nullptr;
  uint32_t* d_k0 = nullptr;
  uint32_t* d_k1 = nullptr;
  int32_t* d_v0 = nullptr;
  int32_t* d_v1 = nullptr;
  int32_t* d_hist = nullptr;
  uint32_t* d_ghist = nullptr;
  // host-side step state
  int64_t t = 0;        // steps sampled
  int64_t mat_t = 0;    // S_E materialised through this many steps
  bool pending_round = false;
  bool broken = false;
  int64_t failed_step = -1;  // earliest step whose batch failed on the device (-1: none)
  int device = -1;            // the device current at init (its streams and memory)
  uint8_t* d_scratch = nullptr;  // device address of the no-alloc scratch array on that device
  struct InFlight {
    massive_batch* io = nullptr;
    int64_t step = -1;
    const int32_t* seeds = nullptr;
    int32_t n0 = 0;
  } infl[kSlots];
  // timing
  int timing = 0;  // bit g: group g is timed
  std::vector<hipEvent_t> ev_pool;
  std::vector<TimedRange> pending;
  double tms[kTimingGroups] = {};
  int64_t tcalls[kTimingGroups] = {};
  std::string err;

  int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    err = buf;
    return code;
  }
  hipEvent_t ev_get() {
    if (ev_pool.empty()) {
      hipEvent_t e;
      // timing only: no system-scope fence
      if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
      return e;
    }
    hipEvent_t e = ev_pool.back();
    ev_pool.pop_back();
    return e;
  }
  // brackets a launch group on stream s when timing is on
  struct Range {
    massive_ctx* c;
    hipStream_t s;
    int group;
    hipEvent_t a = nullptr;
    Range(massive_ctx* c_, hipStream_t s_, int g) : c(c_), s(s_), group(g) {
      if (((c->timing >> g) & 1) && (a = c->ev_get())) (void)hipEventRecord(a, s);
    }
    ~Range() {
      if (!a) return;
      hipEvent_t b = c->ev_get();
      if (!b) return;
      (void)hipEventRecord(b, s);
      c->pending.push_back({a, b, group});
    }
  };
  // a start/stop pair that hipExtLaunchKernelGGL stamps around one dispatch
  bool kernel_pair(int group, hipEvent_t* a, hipEvent_t* b) {
    *a = *b = nullptr;
    if (!((timing >> group) & 1)) return false;
    *a = ev_get();
    *b = ev_get();
    if (!*a || !*b) return false;
    return true;
  }
  void resolve_timing() {
    for (auto& r : pending) {
      add_range(r);
      ev_pool.push_back(r.a);
      ev_pool.push_back(r.b);
    }
    pending.clear();
    // the worker's ranges (its events go back to its own pool)
    std::lock_guard<std::mutex> lk(lmu);
    for (auto& r : lpending) {
      add_range(r);
      lev_pool.push_back(r.a);
      lev_pool.push_back(r.b);
    }
    lpending.clear();
  }
  void add_range(const TimedRange& r) {
    float ms = 0.f;
    if (hipEventSynchronize(r.b) == hipSuccess && hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
      tms[r.group] += ms;
      tcalls[r.group] += 1;
    }
  }
};

#define CK(call)                                                                          \
  do {                                                                                    \
    hipError_t e_ = (call);                                                               \
    if (e_ != hipSuccess) return c->fail(MASSIVE_EHIP, "%s: %s", #call, hipGetErrorString(e_)); \
  } while (0)

#define CKA(ptr, bytes)                                                                   \
  do {                                                                                    \
    size_t b_ = (size_t)(bytes);                                                          \
    if (hipMalloc((void**)&(ptr), b_ ? b_ : 16) != hipSuccess)                            \
      return c->fail(MASSIVE_ENOMEM, "hipMalloc of %zu bytes for %s failed", b_, #ptr);   \
  } while (0)

namespace {

// one stable LSD pass: (kin, vin) -> (kout, vout) by 8-bit digit at `shift`
int sort_pass(massive_ctx* c, hipStream_t s, const uint32_t* kin, const int32_t* vin, const int64_t* n_ptr,
              int64_t n_const, int64_t bound, int shift, uint32_t* kout, int32_t* vout) {
  const int64_t nb = std::max<int64_t>(1, cdiv(bound, ms::kSortTile));
  ms::k_sort_hist<<<(unsigned)nb, ms::kSortNT, 0, s>>>(kin, n_ptr, n_const, bound, shift, nb, c->d_hist);
  const int64_t len = 256 * nb, nb2 = std::max<int64_t>(1, cdiv(len, ms::kScanTile));
  ms::k_tile_reduce<<<(unsigned)nb2, ms::kScanNT, 0, s>>>(c->d_hist, len, c->d_part);
  ms::k_scan_partials<<<1, ms::kScanNT, 0, s>>>(c->d_part, nb2, nullptr, nullptr);
  ms::k_tile_scan<<<(unsigned)nb2, ms::kScanNT, 0, s>>>(c->d_hist, len, c->d_part);
  ms::k_sort_scatter<<<(unsigned)nb, ms::kSortNT, 0, s>>>(kin, vin, n_ptr, n_const, bound, shift, nb, c->d_hist, kout,
                                                          vout);
  return MASSIVE_OK;
}

// four passes of 8 bits; the result lands in (k0, v0), or its values in
// `vals_final` if given.
int sort_u32(massive_ctx* c, hipStream_t s, const int64_t* n_ptr, int64_t n_const, int64_t bound,
             int32_t* vals_final) {
  sort_pass(c, s, c->d_k0, c->d_v0, n_ptr, n_const, bound, 0, c->d_k1, c->d_v1);
  sort_pass(c, s, c->d_k1, c->d_v1, n_ptr, n_const, bound, 8, c->d_k0, c->d_v0);
  sort_pass(c, s, c->d_k0, c->d_v0, n_ptr, n_const, bound, 16, c->d_k1, c->d_v1);
  sort_pass(c, s, c->d_k1, c->d_v1, n_ptr, n_const, bound, 24, c->d_k0, vals_final ? vals_final : c->d_v0);
  return MASSIVE_OK;
}

bool device_visible(const void* p) {
  hipPointerAttribute_t at;
  if (hipPointerGetAttributes(&at, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return at.type == hipMemoryTypeDevice || at.type == hipMemoryTypeManaged || at.type == hipMemoryTypeHost ||
         at.devicePointer != nullptr;
}

// the flattened gather, specialised on the widest vector the row allows
enum GatherKind { kHbm, kMiss };

// The flattened row gather, specialised on the widest vector the row and
// both base pointers allow. max_blocks bounds the grid: host-link gathers
// use a few CUs (16 blocks reach the link's rate; more only congest the
// fabric that HBM traffic also needs).
// With timing on, the dispatch itself is bracketed by hipExtLaunchKernelGGL's
// start/stop events (no launch latency in the measured time).
// The miss gather also takes the write-through slots (wslot) and the buffer
// rows (buf) of the hits on slots still refilling.
void launch_gather(massive_ctx* c, int group, GatherKind kind, hipStream_t s, const int2* list,
                   const int64_t* count, const uint8_t* src, uint8_t* dst, int64_t rb, int64_t max_rows,
                   int64_t max_blocks, const int32_t* wslot = nullptr, uint8_t* buf = nullptr,
                   const ms::StepTail* tail = nullptr) {
  hipEvent_t ea = nullptr, eb = nullptr;
  const bool timed = c->kernel_pair(group, &ea, &eb);
  int vec = 4;
  const uintptr_t al = (uintptr_t)src | (uintptr_t)dst | (uintptr_t)buf;
  if (rb % 16 == 0 && al % 16 == 0)
    vec = 16;
  else if (rb % 8 == 0 && al % 8 == 0)
    vec = 8;
  const uint32_t cpr = (uint32_t)(rb / vec);
  const uint64_t magic = cpr > 1 ? (~0ull) / cpr + 1 : 0;
  const int64_t chunks = std::max<int64_t>(max_rows, 1) * cpr;
  const unsigned grid = grid_for(chunks / 4, 256, max_blocks);
#define MS_ONE(V, ONE)                                                                                         \
  do {                                                                                                         \
    if (kind == kHbm) {                                                                                        \
      if (timed)                                                                                               \
        hipExtLaunchKernelGGL(ms::k_gather_hbm<V, ONE>, dim3(grid), dim3(256), 0, s, ea, eb, 0, list, count, src, \
                              dst, rb, cpr, magic);                                                            \
      else                                                                                                     \
        ms::k_gather_hbm<V, ONE><<<grid, 256, 0, s>>>(list, count, src, dst, rb, cpr, magic);                  \
    } else {                                                                                                   \
      if (timed)                                                                                               \
        hipExtLaunchKernelGGL(ms::k_gather_miss<V, ONE>, dim3(grid), dim3(256), 0, s, ea, eb, 0, list, wslot,  \
                              count, src, dst, buf, c->d_dummy, rb, cpr, magic, *tail);                       \
      else                                                                                                     \
        ms::k_gather_miss<V, ONE><<<grid, 256, 0, s>>>(list, wslot, count, src, dst, buf, c->d_dummy, rb, cpr, \
                                                       magic, *tail);                                          \
    }                                                                                                          \
  } while (0)
#define MS_KIND(V)          \
  do {                      \
    if (cpr == 1)           \
      MS_ONE(V, true);      \
    else                    \
      MS_ONE(V, false);     \
  } while (0)
  if (vec == 16)
    MS_KIND(ms::v4u);
  else if (vec == 8)
    MS_KIND(ms::v2u);
  else
    MS_KIND(unsigned int);
#undef MS_KIND
#undef MS_ONE
  if (timed) c->pending.push_back({ea, eb, group});
}

// The refill: rows of the fill list copied from the host store into buffer
// slots, each slot published in landed[] once its row is written.
void launch_refill(massive_ctx* c, hipStream_t s, const int64_t* count, int64_t max_rows, int32_t round_id,
                   int32_t chunk, int32_t nchunks) {
  hipEvent_t ea = nullptr, eb = nullptr;
  const bool timed = c->kernel_pair(5, &ea, &eb);
  const uint8_t* src = c->d_store;
  uint8_t* dst = c->d_slab;
  const int64_t rb = c->rb;
  int vec = 4;
  if (rb % 16 == 0 && ((uintptr_t)src % 16) == 0 && ((uintptr_t)dst % 16) == 0)
    vec = 16;
  else if (rb % 8 == 0 && ((uintptr_t)src % 8) == 0 && ((uintptr_t)dst % 8) == 0)
    vec = 8;
  const uint32_t cpr = (uint32_t)(rb / vec);
  uint32_t G = 1;
  while (G < cpr && G < MS_WAVE) G <<= 1;
  const int64_t rows_per_block = (256 / MS_WAVE) * ms::kRefillRows * (MS_WAVE / G);
  const unsigned grid = grid_for(std::max<int64_t>(max_rows / nchunks + 1, 1), (int)rows_per_block, c->refill_blocks);
#define MS_RF(V)                                                                                              \
  do {                                                                                                        \
    if (timed)                                                                                                \
      hipExtLaunchKernelGGL(ms::k_refill<V>, dim3(grid), dim3(256), 0, s, ea, eb, 0, (const int2*)c->d_fill, count, \
                            src, dst, c->d_dummy, rb, cpr, G, c->L, c->d_landed, round_id, chunk, nchunks, c->d_ctr); \
    else                                                                                                      \
      ms::k_refill<V><<<grid, 256, 0, s>>>(c->d_fill, count, src, dst, c->d_dummy, rb, cpr, G, c->L, c->d_landed, round_id, \
                                           chunk, nchunks, c->d_ctr);                                        \
  } while (0)
  if (vec == 16)
    MS_RF(ms::v4u);
  else if (vec == 8)
    MS_RF(ms::v2u);
  else
    MS_RF(unsigned int);
#undef MS_RF
  if (timed) c->pending.push_back({ea, eb, 5});
}

// Launches the next `count` pending refill chunks on the copy stream, after
// event `after` (the HBM gather they must not overlap).
int launch_refill_chunks(massive_ctx* c, int count, hipEvent_t after) {
  while (count-- > 0 && c->chunks_left > 0) {
    if (after) {
      hipError_t e = hipStreamWaitEvent(c->s_copy, after, 0);
      if (e != hipSuccess) return c->fail(MASSIVE_EHIP, "hipStreamWaitEvent: %s", hipGetErrorString(e));
    }
    const int32_t chunk = c->refill_chunks - c->chunks_left;
    launch_refill(c, c->s_copy, &c->d_rs->k, c->cap, c->round_id, chunk, c->refill_chunks);
    c->chunks_left -= 1;
    hipError_t e = hipEventRecord(c->ev_refill_done, c->s_copy);
    if (e != hipSuccess) return c->fail(MASSIVE_EHIP, "hipEventRecord: %s", hipGetErrorString(e));
    c->refill_inflight = true;
  }
  return MASSIVE_OK;
}

// ------------------------------------------------------------ staged host link
#define HW(call)                                                                     \
  do {                                                                               \
    hipError_t e_ = (call);                                                          \
    if (e_ != hipSuccess) return std::string(#call) + ": " + hipGetErrorString(e_); \
  } while (0)

int vec_for(int64_t rb, uintptr_t al) {
  if (rb % 16 == 0 && al % 16 == 0) return 16;
  if (rb % 8 == 0 && al % 8 == 0) return 8;
  return 4;
}

// A timing event pair of the worker for group g, or nullptrs when g was off
// when the job was posted.
void link_timing(massive_ctx* c, int timing, int g, hipEvent_t* a, hipEvent_t* b) {
  *a = *b = nullptr;
  if (!((timing >> g) & 1)) return;
  std::lock_guard<std::mutex> lk(c->lmu);
  for (hipEvent_t* e : {a, b}) {
    if (!c->lev_pool.empty()) {
      *e = c->lev_pool.back();
      c->lev_pool.pop_back();
    } else if (hipEventCreateWithFlags(e, hipEventDisableSystemFence) != hipSuccess) {  // timing only
      *e = nullptr;
    }
  }
  if (!*a || !*b) {
    for (hipEvent_t e : {*a, *b})
      if (e) c->lev_pool.push_back(e);
    *a = *b = nullptr;
  }
}

void link_timing_end(massive_ctx* c, hipEvent_t a, hipEvent_t b, int g) {
  std::lock_guard<std::mutex> lk(c->lmu);
  c->lpending.push_back({a, b, g});
}

// Store rows rows[0..n) through the ring, ring_rows at a time: an entry is
// gathered on the host once its last scatter has run, copied to the device on
// the link stream, then handed to scatter(stage, lo, m), which enqueues the
// kernel that consumes staged rows lo..lo+m.
template <class F>
std::string link_rows(massive_ctx* c, const int32_t* rows, int64_t n, F&& scatter) {
  hipStream_t s = c->s_link;
  const int64_t eb = c->ring_rows * c->rb;
  for (int64_t lo = 0; lo < n; lo += c->ring_rows) {
    const int64_t m = std::min(c->ring_rows, n - lo);
    const int e = c->ring_next;
    c->ring_next = (e + 1) % massive_ctx::kRing;
    if (c->ring_used[e]) HW(hipEventSynchronize(c->ev_ring[e]));
    uint8_t* h = c->h_ring + e * eb;
    uint8_t* d = c->d_ring + e * eb;
    c->pool->gather(c->h_store, c->H, c->rb, rows + lo, m, h);
    HW(hipMemcpyAsync(d, h, (size_t)(m * c->rb), hipMemcpyHostToDevice, s));
    scatter(d, lo, m);
    HW(hipGetLastError());
    HW(hipEventRecord(c->ev_ring[e], s));
    c->ring_used[e] = true;
  }
  return std::string();
}

template <typename V>
void scatter_rows(hipStream_t s, const massive_ctx::LinkJob& j, const uint8_t* st, int64_t lo, int64_t m,
                  uint8_t* buf, int64_t rb, uint32_t cpr, uint64_t magic) {
  const unsigned grid = grid_for(m * cpr, 256, 4096);
  if (cpr == 1)
    ms::k_scatter_rows<V, true><<<grid, 256, 0, s>>>(st, j.list, j.wslot, lo, m, j.feat, buf, rb, cpr, magic);
  else
    ms::k_scatter_rows<V, false><<<grid, 256, 0, s>>>(st, j.list, j.wslot, lo, m, j.feat, buf, rb, cpr, magic);
}

template <typename V>
void refill_scatter(massive_ctx* c, hipStream_t s, const uint8_t* st, int64_t lo, int64_t m, uint32_t cpr,
                    uint32_t G, int32_t round_id) {
  const int rows_per_block = (256 / MS_WAVE) * (MS_WAVE / (int)G);
  const unsigned grid = grid_for(m, rows_per_block, 4096);
  ms::k_refill_scatter<V><<<grid, 256, 0, s>>>(st, c->d_fill, lo, m, c->d_slab, c->rb, cpr, G, c->L, c->d_landed,
                                              round_id, c->d_ctr);
}

// A step's tail: its host rows (misses and hits on refilling slots) through
// the ring into their output rows (and write-through slots), then, after the
// step's HBM gather, the completion kernel and the batch's event.
std::string link_step(massive_ctx* c, const massive_ctx::LinkJob& j) {
  hipStream_t s = c->s_link;
  int64_t n = 0;
  if (j.rows) {
    HW(hipEventSynchronize(c->ev_rows_ready[j.slot]));
    n = std::min<int64_t>(std::max<int64_t>(c->h_cnt[j.slot], 0), c->H);
  }
  if (n > 0) {
    hipEvent_t ta, tb;
    link_timing(c, j.timing, 3, &ta, &tb);
    if (ta) HW(hipEventRecord(ta, s));
    const int64_t rb = c->rb;
    uint8_t* buf = c->d_slab + (int64_t)c->L * rb;
    const int vec = vec_for(rb, (uintptr_t)j.feat | (uintptr_t)buf | (uintptr_t)c->d_ring);
    const uint32_t cpr = (uint32_t)(rb / vec);
    const uint64_t magic = cpr > 1 ? (~0ull) / cpr + 1 : 0;
    std::string e = link_rows(c, c->h_rows[j.slot], n, [&](const uint8_t* st, int64_t lo, int64_t m) {
      if (vec == 16)
        scatter_rows<ms::v4u>(s, j, st, lo, m, buf, rb, cpr, magic);
      else if (vec == 8)
        scatter_rows<ms::v2u>(s, j, st, lo, m, buf, rb, cpr, magic);
      else
        scatter_rows<unsigned int>(s, j, st, lo, m, buf, rb, cpr, magic);
    });
    if (!e.empty()) return e;
    if (ta) {
      HW(hipEventRecord(tb, s));
      link_timing_end(c, ta, tb, 3);
    }
  }
  HW(hipStreamWaitEvent(s, c->ev_hbm_done[j.slot], 0));
  const bool publish = j.pend >= 0;
  ms::k_step_done<<<publish ? grid_for(j.nbK, 256, 1024) : 1, 256, 0, s>>>(
      j.wslot, &j.sz->n_miss, c->d_landed, c->cap, j.pend, j.sz, c->K, &c->d_ctr->bad, c->hd_sz + j.slot,
      c->hd_bad + j.slot);
  HW(hipGetLastError());
  HW(hipEventRecord(c->ev_batch_done[j.slot], s));
  return std::string();
}

// One refill chunk of the current round: fill-list entries of the chunk
// through the ring into their slots; the round's last chunk records
// ev_fill_done.
std::string link_refill(massive_ctx* c, const massive_ctx::LinkJob& j) {
  hipStream_t s = c->s_link;
  HW(hipEventSynchronize(c->ev_fill_ready));
  const int64_t k = std::min<int64_t>(std::max<int64_t>(c->h_cnt[kSlots], 0), c->cap);
  const int64_t lo = k * j.chunk / j.nchunks, hi = k * (j.chunk + 1) / j.nchunks;
  if (hi > lo) {
    hipEvent_t ta, tb;
    link_timing(c, j.timing, 5, &ta, &tb);
    if (ta) HW(hipEventRecord(ta, s));
    const int vec = vec_for(c->rb, (uintptr_t)c->d_slab | (uintptr_t)c->d_ring);
    const uint32_t cpr = (uint32_t)(c->rb / vec);
    uint32_t G = 1;
    while (G < cpr && G < MS_WAVE) G <<= 1;
    std::string e = link_rows(c, c->h_fill_rows + lo, hi - lo, [&](const uint8_t* st, int64_t off, int64_t m) {
      if (vec == 16)
        refill_scatter<ms::v4u>(c, s, st, lo + off, m, cpr, G, j.round_id);
      else if (vec == 8)
        refill_scatter<ms::v2u>(c, s, st, lo + off, m, cpr, G, j.round_id);
      else
        refill_scatter<unsigned int>(c, s, st, lo + off, m, cpr, G, j.round_id);
    });
    if (!e.empty()) return e;
    if (ta) {
      HW(hipEventRecord(tb, s));
      link_timing_end(c, ta, tb, 5);
    }
  }
  if (j.chunk == j.nchunks - 1) HW(hipEventRecord(c->ev_fill_done, s));
  return std::string();
}
#undef HW

// The worker: jobs in posting order until the context ends. After a failure
// it takes the remaining jobs without running them, so that every wait for
// its progress ends; the failure is reported by the next call that waits.
void link_loop(massive_ctx* c) {
  const hipError_t de = hipSetDevice(c->device);
  for (;;) {
    massive_ctx::LinkJob j;
    bool skip;
    {
      std::unique_lock<std::mutex> lk(c->lmu);
      c->lcv.wait(lk, [c] { return c->lstop || !c->ljobs.empty(); });
      if (c->ljobs.empty()) return;  // stopped, every job taken
      j = c->ljobs.front();
      c->ljobs.pop_front();
      c->lbusy = true;
      skip = c->lfailed;
    }
    std::string err;
    if (de != hipSuccess)
      err = std::string("hipSetDevice: ") + hipGetErrorString(de);
    else if (!skip)
      err = j.refill ? link_refill(c, j) : link_step(c, j);
    {
      std::lock_guard<std::mutex> lk(c->lmu);
      if (!err.empty() && !c->lfailed) {
        c->lfailed = true;
        c->lerr = err;
      }
      if (!j.refill)
        c->tail_step = j.step;
      else if (j.chunk == j.nchunks - 1)
        c->fill_done_round = j.round_id;
      c->lbusy = false;
    }
    c->lcv.notify_all();
  }
}

void link_post(massive_ctx* c, const massive_ctx::LinkJob& j) {
  {
    std::lock_guard<std::mutex> lk(c->lmu);
    c->ljobs.push_back(j);
  }
  c->lcv.notify_all();
}

// Waits until done() holds (under the worker's lock) or the worker has failed.
template <class P>
int link_wait(massive_ctx* c, P done) {
  std::string e;
  {
    std::unique_lock<std::mutex> lk(c->lmu);
    c->lcv.wait(lk, [&] { return c->lfailed || done(); });
    if (!c->lfailed) return MASSIVE_OK;
    e = c->lerr;
  }
  c->broken = true;
  return c->fail(MASSIVE_EHIP, "host-link worker: %s", e.c_str());
}

// Every posted job enqueued and the link stream idle (nothing to do in the
// loads mode).
int link_drain(massive_ctx* c) {
  if (!c->staged()) return MASSIVE_OK;
  const int rc = link_wait(c, [c] { return c->ljobs.empty() && !c->lbusy; });
  if (rc != MASSIVE_OK) return rc;
  CK(hipStreamSynchronize(c->s_link));
  return MASSIVE_OK;
}

// Posts the next `count` refill chunks of the current round.
void link_post_chunks(massive_ctx* c, int count) {
  while (count-- > 0 && c->chunks_left > 0) {
    massive_ctx::LinkJob j;
    j.refill = true;
    j.round_id = c->round_id;
    j.chunk = c->refill_chunks - c->chunks_left;
    j.nchunks = c->refill_chunks;
    j.timing = c->timing;
    link_post(c, j);
    c->chunks_left -= 1;
  }
}

void free_ctx(massive_ctx* c) {
  if (!c) return;
  // the worker finishes the jobs already posted, then ends
  if (c->worker.joinable()) {
    {
      std::lock_guard<std::mutex> lk(c->lmu);
      c->lstop = true;
    }
    c->lcv.notify_all();
    c->worker.join();
  }
  delete c->pool;
  (void)hipDeviceSynchronize();
  void* dev[] = {c->d_indptr, c->d_indices, c->d_slab, c->d_slot_id, c->d_S_E, c->d_hitcnt, c->d_S_A,
                 c->d_rank_of, c->d_h_of_rank, c->d_tab, c->d_pos_of, c->d_bits, c->d_sz, c->d_rs,
                 c->d_part, c->d_part2, c->d_scan_flags, c->d_dummy, c->d_E, c->d_R,
                 c->d_fill, c->d_ctr, c->d_slot_round, c->d_landed,
                 c->d_k0, c->d_k1, c->d_v0, c->d_v1, c->d_hist, c->d_ghist, c->d_big,
                 c->d_gid, c->d_rank_g, c->d_gpart, c->d_deg};
  for (void* p : dev)
    if (p) (void)hipFree(p);
  for (int i = 0; i < kSlots; ++i)
    for (void* p : {(void*)c->d_hbm_list[i], (void*)c->d_miss_list[i], (void*)c->d_miss_slot[i]})
      if (p) (void)hipFree(p);
  if (c->h_sz) (void)hipHostFree(c->h_sz);
  if (c->h_rs) (void)hipHostFree(c->h_rs);
  if (c->h_bad) (void)hipHostFree(c->h_bad);
  if (c->h_ctr) (void)hipHostFree(c->h_ctr);
  for (int i = 0; i < kSlots; ++i)
    if (c->h_rows[i]) (void)hipHostFree(c->h_rows[i]);
  for (void* p : {(void*)c->h_fill_rows, (void*)c->h_cnt, (void*)c->h_ring})
    if (p) (void)hipHostFree(p);
  if (c->d_ring) (void)hipFree(c->d_ring);
  for (int i = 0; i < kSlots; ++i)
    for (hipEvent_t e : {c->ev_cls_done[i], c->ev_hbm_done[i], c->ev_batch_done[i], c->ev_rows_ready[i]})
      if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : c->ev_ring)
    if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : {c->ev_fill_ready, c->ev_fill_done})
    if (e) (void)hipEventDestroy(e);
  for (auto& r : c->lpending) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (hipEvent_t e : c->lev_pool) (void)hipEventDestroy(e);
  for (hipEvent_t e : {c->ev_round_done, c->ev_refill_done})
    if (e) (void)hipEventDestroy(e);
  for (auto& r : c->pending) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (hipEvent_t e : c->ev_pool) (void)hipEventDestroy(e);
  if (c->s_miss) (void)hipStreamDestroy(c->s_miss);
  if (c->s_copy) (void)hipStreamDestroy(c->s_copy);
  if (c->s_link) (void)hipStreamDestroy(c->s_link);
  delete c;
}

int init_impl(massive_ctx* c, const massive_init_args* a) {
  c->L = a->L;
  c->H = a->H;
  c->R = (int64_t)a->L + a->H;
  c->rb = a->row_bytes;
  c->K = a->K;
  for (int k = 0; k < a->K; ++k) c->fo[k] = a->fanout[k];
  c->pct = a->buffer_pct;
  c->gamma = a->gamma;
  c->delta = a->delta;
  c->seed = a->seed;
  c->nnz = a->indptr[c->R];
  c->cap = (int64_t)a->H * a->buffer_pct / 100;
  c->layout = a->score_layout;
  c->n_sa = c->layout == MASSIVE_SCORES_BY_GID ? a->n_global : a->H;
  c->hcap = 64;
  while (c->hcap < 2 * c->cap) c->hcap <<= 1;
  c->hmask = (uint32_t)(c->hcap - 1);
  c->W = cdiv(c->R, 32);
  c->sort_cap = std::max<int64_t>(std::max<int64_t>(c->H, c->cap), 1);
  c->pmax = std::max(cdiv(c->R, ms::kScanTile), cdiv(256 * cdiv(c->sort_cap, ms::kSortTile), ms::kScanTile));
  c->pmax = std::max<int64_t>(c->pmax, cdiv(c->W, ms::kScanTile)) + 8;
  // Eq. 1 with S_E at its initial value 1: alpha = gamma^delta in fp32 products
  // (once a product no longer changes the value, e.g. at 0, the rest cannot)
  float al = 1.0f;
  for (int32_t i = 0; i < a->delta; ++i) {
    const float next = al * a->gamma;
    if (next == al) break;
    al = next;
  }
  c->alpha = al;
  // sampler: about fo + 3 sqrt(fo) + 3 keys survive the first threshold
  for (int k = 0; k < a->K; ++k) {
    const double fo = a->fanout[k];
    const double mu = std::min(fo + 3.0 * std::sqrt(fo) + 3.0, 0.5 * (fo + ms::kCandCap));
    c->mu32[k] = mu * 4294967296.0;
  }

  if (const char* e = getenv("MASSIVE_HBM_BLOCKS")) c->hbm_blocks = std::max(1, atoi(e));
  if (const char* e = getenv("MASSIVE_HOST_BLOCKS")) c->host_blocks = c->host_blocks_light = std::max(1, atoi(e));
  if (const char* e = getenv("MASSIVE_REFILL_BLOCKS")) c->refill_blocks = std::max(1, atoi(e));
  // one chunk after each of the next steps' HBM gathers, all launched before
  // the step of the next round, so that round never waits for a chunk in flight
  c->refill_chunks = std::max<int32_t>(1, std::min<int32_t>(a->delta - 1, 32));
  if (const char* e = getenv("MASSIVE_REFILL_CHUNKS")) c->refill_chunks = std::max(1, atoi(e));
  if (const char* e = getenv("MASSIVE_BIG_ROW")) c->big_min = std::max<int64_t>(256, atoll(e));
  if (const char* e = getenv("MASSIVE_BIG_BLOCKS")) c->big_blocks = std::max<int64_t>(1, atoll(e));
  if (const char* e = getenv("MASSIVE_TAU_ITERS")) c->tau_iters = std::min(std::max(0, atoi(e)), ms::kTauIters);
  if (const char* e = getenv("MASSIVE_RING_BYTES")) c->ring_bytes = std::max<int64_t>(1, atoll(e));
  c->s_main = (hipStream_t)a->stream;
  c->link_mode = a->link_mode;
  c->link_threads = a->link_threads > 0 ? a->link_threads : 8;
  CK(hipGetDevice(&c->device));
  if (c->device < 0 || c->device >= kMaxDevices) return c->fail(MASSIVE_EHIP, "device %d out of range", c->device);
  {
    void* p = nullptr;
    CK(scratch_address(c->device, &p));
    c->d_scratch = static_cast<uint8_t*>(p);
  }
  CK(hipStreamCreateWithFlags(&c->s_miss, hipStreamNonBlocking));
  CK(hipStreamCreateWithFlags(&c->s_copy, hipStreamNonBlocking));
  // Events that only order work between this device's streams (classify ->
  // gathers, HBM gather -> refill and round) skip the system-scope fence:
  // their kernels' writes are visible on the device without it. The batch's
  // completion event keeps it: after it the host reads the step's sizes and
  // the caller its outputs (the next round also follows it).
  for (int i = 0; i < kSlots; ++i) {
    for (hipEvent_t* e : {&c->ev_cls_done[i], &c->ev_hbm_done[i]})
      CK(hipEventCreateWithFlags(e, hipEventDisableTiming | hipEventDisableSystemFence));
    CK(hipEventCreateWithFlags(&c->ev_batch_done[i], hipEventDisableTiming));
  }
  for (hipEvent_t* e : {&c->ev_round_done, &c->ev_refill_done})
    CK(hipEventCreateWithFlags(e, hipEventDisableTiming));
  if (c->staged()) {
    CK(hipStreamCreateWithFlags(&c->s_link, hipStreamNonBlocking));
    for (int i = 0; i < kSlots; ++i) CK(hipEventCreateWithFlags(&c->ev_rows_ready[i], hipEventDisableTiming));
    for (hipEvent_t* e : {&c->ev_fill_ready, &c->ev_fill_done}) CK(hipEventCreateWithFlags(e, hipEventDisableTiming));
    for (hipEvent_t& e : c->ev_ring) CK(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  }

  // the pinned store must be mapped into the device address space
  {
    void* dp = nullptr;
    if (c->H > 0) {
      if (hipHostGetDevicePointer(&dp, const_cast<void*>(a->halo_store), 0) != hipSuccess || !dp)
        return c->fail(MASSIVE_EINVAL, "halo_store is not pinned host memory (allocate it with hipHostMalloc / "
                                       "torch pin_memory=True)");
    }
    c->d_store = (const uint8_t*)dp;
  }

  const int64_t R = c->R, H = c->H, cap = c->cap, rb = c->rb;
  CKA(c->d_indptr, (R + 1) * 8);
  CKA(c->d_indices, c->nnz * 4);
  CKA(c->d_slab, (c->L + cap) * rb);
  CKA(c->d_slot_id, cap * 4);
  CKA(c->d_S_E, cap * 4);
  CKA(c->d_hitcnt, cap * 4);
  CKA(c->d_S_A, c->n_sa * 4);
  CKA(c->d_gid, H * 4);
  if (c->layout == MASSIVE_SCORES_BY_GID) {
    CKA(c->d_rank_g, c->n_sa * 4);
    CKA(c->d_gpart, (cdiv(c->n_sa, ms::kScanTile) + 8) * 4);
  }
  CKA(c->d_rank_of, H * 4);
  CKA(c->d_h_of_rank, H * 4);
  // a node's S_A index: its global id or its rank (classify reads entry 0 of
  // this array for rows that are not misses, so it is set whatever H is)
  c->d_sa_idx = c->layout == MASSIVE_SCORES_BY_GID ? c->d_gid : c->d_rank_of;
  if (!c->d_sa_idx) return c->fail(MASSIVE_EHIP, "no S_A index array");
  CKA(c->d_tab, c->hcap * 8);
  CKA(c->d_pos_of, R * 4);
  CKA(c->d_big, R * 4);
  CKA(c->d_bits, (c->W + 4) * 4);
  CKA(c->d_sz, kSlots * sizeof(ms::StepSizes));
  CKA(c->d_rs, sizeof(ms::RoundState));
  CKA(c->d_ctr, sizeof(ms::Counters));
  CKA(c->d_slot_round, cap * 4);
  CKA(c->d_landed, cap * 4);
  CKA(c->d_part, c->pmax * 4);
  CKA(c->d_part2, c->pmax * 4);
  c->scan_tiles = std::max(cdiv(R, ms::kScanTile), cdiv(c->W, ms::kScanTile)) + 1;
  CKA(c->d_scan_flags, c->scan_tiles * 8);
  for (int i = 0; i < kSlots; ++i) {
    CKA(c->d_hbm_list[i], R * 8);
    CKA(c->d_miss_list[i], R * 8);
    CKA(c->d_miss_slot[i], R * 4);
  }
  CKA(c->d_dummy, std::max<int64_t>(c->rb, 16));
  CKA(c->d_E, cap * 4);
  CKA(c->d_R, cap * 4);
  CKA(c->d_fill, cap * 8);
  CKA(c->d_k0, c->sort_cap * 4);
  CKA(c->d_k1, c->sort_cap * 4);
  CKA(c->d_v0, c->sort_cap * 4);
  CKA(c->d_v1, c->sort_cap * 4);
  CKA(c->d_hist, 256 * cdiv(c->sort_cap, ms::kSortTile) * 4);
  CKA(c->d_ghist, 256 * 4);
  if (hipHostMalloc((void**)&c->h_sz, kSlots * sizeof(ms::StepSizes), hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc((void**)&c->h_rs, sizeof(ms::RoundState), hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc((void**)&c->h_bad, kSlots * sizeof(int32_t), hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc((void**)&c->h_ctr, sizeof(ms::Counters), hipHostMallocDefault) != hipSuccess)
    return c->fail(MASSIVE_ENOMEM, "hipHostMalloc of the size mailboxes failed");
  if (hipHostGetDevicePointer((void**)&c->hd_sz, c->h_sz, 0) != hipSuccess || !c->hd_sz ||
      hipHostGetDevicePointer((void**)&c->hd_bad, c->h_bad, 0) != hipSuccess || !c->hd_bad)
    return c->fail(MASSIVE_EHIP, "the size mailboxes have no device view");
  if (c->staged()) {
    // host rows of each slot's misses (at most H per step), of a round's fill
    // list (at most cap), their counts, and the staging ring
    c->h_store = static_cast<const uint8_t*>(a->halo_store);
    c->ring_rows = std::max<int64_t>(1, c->ring_bytes / rb);
    const int64_t ring_bytes = massive_ctx::kRing * c->ring_rows * rb;
    auto pinned = [](void** p, int64_t bytes) {
      return hipHostMalloc(p, (size_t)std::max<int64_t>(bytes, 16), hipHostMallocDefault) == hipSuccess;
    };
    bool ok = true;
    for (int i = 0; i < kSlots; ++i) ok = ok && pinned((void**)&c->h_rows[i], H * 4);
    ok = ok && pinned((void**)&c->h_fill_rows, cap * 4) && pinned((void**)&c->h_cnt, (kSlots + 1) * 8) &&
         pinned((void**)&c->h_ring, ring_bytes);
    if (!ok) return c->fail(MASSIVE_ENOMEM, "hipHostMalloc of the staged link's buffers failed");
    for (int i = 0; i < kSlots; ++i)
      ok = ok && hipHostGetDevicePointer((void**)&c->hd_rows[i], c->h_rows[i], 0) == hipSuccess && c->hd_rows[i];
    ok = ok && hipHostGetDevicePointer((void**)&c->hd_fill_rows, c->h_fill_rows, 0) == hipSuccess &&
         c->hd_fill_rows && hipHostGetDevicePointer((void**)&c->hd_cnt, c->h_cnt, 0) == hipSuccess && c->hd_cnt;
    if (!ok) return c->fail(MASSIVE_EHIP, "the staged link's row lists have no device view");
    std::memset(c->h_cnt, 0, (kSlots + 1) * 8);
    CKA(c->d_ring, ring_bytes);
    c->pool = new ms::GatherPool(c->link_threads);
    c->worker = std::thread(link_loop, c);
  }

  hipStream_t s = c->s_main;
  CK(hipMemcpyAsync(c->d_indptr, a->indptr, (R + 1) * 8, hipMemcpyHostToDevice, s));
  if (c->nnz) CK(hipMemcpyAsync(c->d_indices, a->indices, c->nnz * 4, hipMemcpyHostToDevice, s));
  if (c->L) CK(hipMemcpyAsync(c->d_slab, a->local_feat, (int64_t)c->L * rb, hipMemcpyHostToDevice, s));
  {
    CK(hipMemsetAsync(c->d_ctr, 0, sizeof(ms::Counters), s));
    ms::k_validate_csr<<<grid_for(std::max(R, c->nnz), 256, 8192), 256, 0, s>>>(c->d_indptr, R, c->d_indices, c->nnz,
                                                                                &c->d_ctr->bad);
    CK(hipMemcpyAsync(c->h_ctr, c->d_ctr, sizeof(ms::Counters), hipMemcpyDeviceToHost, s));
    CK(hipStreamSynchronize(s));
    if (c->h_ctr->bad)
      return c->fail(MASSIVE_EINVAL, (c->h_ctr->bad & 2) ? "indices has ids outside [0, L+H)"
                                                          : "indptr is not non-decreasing");
  }
  CK(hipMemsetAsync(c->d_pos_of, 0xFF, R * 4, s));
  CK(hipMemsetAsync(c->d_bits, 0, (c->W + 4) * 4, s));
  CK(hipMemsetAsync(c->d_ghist, 0, 256 * 4, s));
  CK(hipMemsetAsync(c->d_scan_flags, 0, c->scan_tiles * 8, s));
  CK(hipMemsetAsync(c->d_ctr, 0, sizeof(ms::Counters), s));
  CK(hipMemsetAsync(c->d_slot_round, 0xFF, cap * 4, s));
  CK(hipMemsetAsync(c->d_landed, 0xFF, cap * 4, s));

  if (H > 0) {
    // halo rank: (degree desc, global id asc) by two stable radix sorts
    CKA(c->d_deg, H * 8);
    CK(hipMemcpyAsync(c->d_gid, a->halo_gid, H * 4, hipMemcpyHostToDevice, s));
    CK(hipMemcpyAsync(c->d_deg, a->halo_degree, H * 8, hipMemcpyHostToDevice, s));
    ms::k_rank_keys_lo<<<grid_for(H, 256), 256, 0, s>>>(c->d_gid, H, c->d_k0, c->d_v0);
    sort_u32(c, s, nullptr, H, H, nullptr);
    ms::k_rank_keys_hi<<<grid_for(H, 256), 256, 0, s>>>(c->d_deg, c->d_v0, H, c->d_k0);
    sort_u32(c, s, nullptr, H, H, c->d_h_of_rank);
    ms::k_rank_finish<<<grid_for(H, 256), 256, 0, s>>>(c->d_h_of_rank, H, c->d_rank_of);
    if (c->layout == MASSIVE_SCORES_BY_GID) {
      // S_A and the rank of every global id: -1 except at halo ids
      ms::k_fill<float><<<grid_for(c->n_sa, 256), 256, 0, s>>>(c->d_S_A, c->n_sa, -1.0f);
      ms::k_fill<int32_t><<<grid_for(c->n_sa, 256), 256, 0, s>>>(c->d_rank_g, c->n_sa, -1);
      ms::k_gid_init<<<grid_for(H, 256), 256, 0, s>>>(c->d_gid, c->d_rank_of, H, c->d_S_A, c->d_rank_g);
      CK(hipMemsetAsync(c->d_ctr, 0, sizeof(ms::Counters), s));
      ms::k_gid_check<<<grid_for(H, 256), 256, 0, s>>>(c->d_gid, c->d_rank_of, H, c->d_rank_g, &c->d_ctr->bad);
      CK(hipMemcpyAsync(c->h_ctr, c->d_ctr, sizeof(ms::Counters), hipMemcpyDeviceToHost, s));
      CK(hipStreamSynchronize(s));
      if (c->h_ctr->bad) return c->fail(MASSIVE_EINVAL, "halo_gid repeats a global id");
      CK(hipMemsetAsync(c->d_ctr, 0, sizeof(ms::Counters), s));
    } else {
      ms::k_fill<float><<<grid_for(H, 256), 256, 0, s>>>(c->d_S_A, H, 0.0f);
    }
    CK(hipStreamSynchronize(s));
    (void)hipFree(c->d_deg);
    c->d_deg = nullptr;
  }
  ms::k_fill<uint64_t><<<grid_for(c->hcap, 256), 256, 0, s>>>(c->d_tab, c->hcap, ms::kEmpty);
  if (cap > 0) {
    ms::k_init_buffer<<<grid_for(cap, 256), 256, 0, s>>>(c->d_h_of_rank, cap, c->L, c->d_slot_id, c->d_S_E,
                                                         c->d_hitcnt, c->d_S_A, c->d_sa_idx, c->d_fill);
    ms::k_hash_insert<<<grid_for(cap, 256), 256, 0, s>>>(c->d_tab, c->hmask, c->d_slot_id, cap, nullptr);
    // the cap best-ranked rows arrive over the host link
    c->h_rs->k = cap;
    CK(hipMemcpyAsync(&c->d_rs->k, &c->h_rs->k, 8, hipMemcpyHostToDevice, s));
    launch_refill(c, s, &c->d_rs->k, cap, 0, 0, 1);
  }
  // the step-slot events start out complete
  for (int i = 0; i < kSlots; ++i) {
    CK(hipEventRecord(c->ev_cls_done[i], s));
    CK(hipEventRecord(c->ev_hbm_done[i], c->s_miss));
    CK(hipEventRecord(c->ev_batch_done[i], c->s_miss));
  }
  CK(hipGetLastError());
  CK(hipStreamSynchronize(s));
  CK(hipStreamSynchronize(c->s_miss));
  return MASSIVE_OK;
}

}  // namespace

extern "C" {

int massive_init(const massive_init_args* a, massive_ctx** out) {
  g_init_error.clear();
  if (!out) {
    g_init_error = "out is NULL";
    return MASSIVE_EINVAL;
  }
  *out = nullptr;
  auto bad = [](const char* m) {
    g_init_error = m;
    return MASSIVE_EINVAL;
  };
  if (!a) return bad("args is NULL");
  if (a->L < 0 || a->H < 0 || (int64_t)a->L + a->H <= 0) return bad("need L >= 0, H >= 0, L + H > 0");
  if (!a->indptr || !a->indices) return bad("indptr / indices are NULL");
  if (a->L > 0 && !a->local_feat) return bad("local_feat is NULL");
  if (a->H > 0 && (!a->halo_store || !a->halo_gid || !a->halo_degree)) return bad("halo arrays are NULL");
  // (at most 1 MiB keeps the copy kernels' division by chunks per row, a
  // multiply by a rounded-up reciprocal, exact for every chunk index that fits
  // in device memory)
  if (a->row_bytes <= 0 || a->row_bytes % 4 || a->row_bytes > (1 << 20))
    return bad("row_bytes must be a positive multiple of 4, at most 1 MiB");
  if (a->K < 1 || a->K > MASSIVE_MAX_HOPS) return bad("K must be in 1..8");
  for (int k = 0; k < a->K; ++k)
    if (a->fanout[k] < 1 || a->fanout[k] > 256) return bad("every fanout must be in 1..256");
  if (a->buffer_pct < 0 || a->buffer_pct > 100) return bad("buffer_pct must be in 0..100");
  if (!(a->gamma > 0.0f && a->gamma <= 1.0f)) return bad("gamma must be in (0, 1]");
  if (a->delta < 1) return bad("delta must be >= 1");
  if (a->score_layout != MASSIVE_SCORES_BY_RANK && a->score_layout != MASSIVE_SCORES_BY_GID)
    return bad("score_layout must be MASSIVE_SCORES_BY_RANK or MASSIVE_SCORES_BY_GID");
  if (a->score_layout == MASSIVE_SCORES_BY_GID) {
    if (a->n_global < 1 || a->n_global > (int64_t(1) << 31)) return bad("n_global must be in 1..2^31");
    for (int32_t h = 0; h < a->H; ++h)
      if (a->halo_gid[h] < 0 || a->halo_gid[h] >= a->n_global) return bad("a halo_gid lies outside [0, n_global)");
  }
  if (a->link_mode != MASSIVE_LINK_LOADS && a->link_mode != MASSIVE_LINK_STAGED)
    return bad("link_mode must be MASSIVE_LINK_LOADS or MASSIVE_LINK_STAGED");
  if (a->link_threads < 0 || a->link_threads > 64) return bad("link_threads must be in 0..64");
  const int64_t R = (int64_t)a->L + a->H;
  if (a->indptr[0] != 0 || a->indptr[R] < 0) return bad("indptr must start at 0");
  massive_ctx* c = new (std::nothrow) massive_ctx();
  if (!c) return bad("out of host memory");
  int rc;
  try {
    rc = init_impl(c, a);
  } catch (const std::exception& e) {  // host threads or memory of the staged link
    rc = c->fail(MASSIVE_ENOMEM, "massive_init: %s", e.what());
  }
  if (rc != MASSIVE_OK) {
    g_init_error = c->err;
    free_ctx(c);
    return rc;
  }
  *out = c;
  return MASSIVE_OK;
}

int massive_output_bounds(const massive_ctx* c, int32_t n_seeds, int64_t* n_bound, int64_t* e_bound) {
  if (!c || !n_bound || !e_bound || n_seeds < 0) return MASSIVE_EINVAL;
  n_bound[0] = std::min<int64_t>(n_seeds, c->L);
  for (int k = 0; k < c->K; ++k) {
    e_bound[k] = n_bound[k] * c->fo[k];
    n_bound[k + 1] = std::min<int64_t>(c->R, n_bound[k] + e_bound[k]);
  }
  return MASSIVE_OK;
}

}  // extern "C"

namespace {

// Per-step buffers of one enqueued step: those of the context's step slot,
// or the no-alloc scratch array (then its scan flags are cleared per call,
// fill kernels clear it, and nothing is timed).
struct StepBufs {
  ms::StepSizes* sz;
  int2* hbm_list;
  int2* miss_list;
  int32_t* miss_slot;
  int32_t* big;
  uint64_t* flags;
  bool from_scratch;
};

// The epoch of the next single-pass scan (flags of earlier epochs are stale
// by their tag); the flags are cleared before the tags could wrap around.
uint32_t next_scan_epoch(massive_ctx* c, hipStream_t s) {
  if (c->scan_epoch >= (1u << 30)) {
    ms::k_fill<uint64_t><<<grid_for(c->scan_tiles, 256), 256, 0, s>>>(c->d_scan_flags, c->scan_tiles, 0ull);
    c->scan_epoch = 0;
  }
  return ++c->scan_epoch;
}

// Argument checks shared by the entry points that enqueue a step; nb and eb
// receive the output bounds of the batch.
int check_step_args(massive_ctx* c, const int32_t* seeds, int32_t n0, massive_batch* io, int64_t* nb, int64_t* eb) {
  if (c->broken) return c->fail(MASSIVE_ESTATE, "context is unusable after an earlier failure");
  if (!io || n0 < 0 || (n0 > 0 && !seeds)) return c->fail(MASSIVE_EINVAL, "bad seeds / batch arguments");
  if (c->pending_round) return c->fail(MASSIVE_ESTATE, "massive_evict_step was not called after the last step");
  if (n0 > c->L) return c->fail(MASSIVE_EINVAL, "more seeds than local nodes");
  for (int i = 0; i < kSlots; ++i)
    if (c->infl[i].io == io) return c->fail(MASSIVE_ESTATE, "this batch is still in flight");
  massive_output_bounds(c, n0, nb, eb);
  if (!io->nodes || !io->mask || !io->feat) return c->fail(MASSIVE_EINVAL, "nodes / mask / feat are NULL");
  if (io->nodes_cap < nb[c->K]) return c->fail(MASSIVE_ECAPACITY, "nodes_cap %lld < bound %lld",
                                               (long long)io->nodes_cap, (long long)nb[c->K]);
  for (int k = 0; k < c->K; ++k) {
    if (!io->indptr[k] || !io->indices[k]) return c->fail(MASSIVE_EINVAL, "hop %d buffers are NULL", k + 1);
    if (io->indptr_cap[k] < nb[k] + 1 || io->indices_cap[k] < eb[k])
      return c->fail(MASSIVE_ECAPACITY, "hop %d buffers below the bound (%lld, %lld)", k + 1, (long long)(nb[k] + 1),
                     (long long)eb[k]);
    if (eb[k] >= (1ll << 31)) return c->fail(MASSIVE_EINVAL, "hop %d may emit 2^31 edges or more", k + 1);
  }
  if (c->t >= 0xFFFFFFFFll) return c->fail(MASSIVE_ESTATE, "step counter exhausted");
  // every pointer the kernels dereference must be visible to the device:
  // nodes, mask, feat, the seeds and two arrays per hop (K <= MASSIVE_MAX_HOPS)
  if (!device_visible(io->nodes) || !device_visible(io->mask) || !device_visible(io->feat))
    return c->fail(MASSIVE_EINVAL, "nodes / mask / feat are not HIP-visible memory");
  if (n0 > 0 && !device_visible(seeds)) return c->fail(MASSIVE_EINVAL, "seeds are not HIP-visible memory");
  for (int k = 0; k < c->K; ++k)
    if (!device_visible(io->indptr[k]) || !device_visible(io->indices[k]))
      return c->fail(MASSIVE_EINVAL, "hop %d buffers are not HIP-visible memory", k + 1);

  return MASSIVE_OK;
}

// Enqueues one step (sampling and classify on the main stream, the gathers
// and the step's completion on the side stream) with the per-step buffers sb.
int enqueue_step(massive_ctx* c, const int32_t* seeds, int32_t n0, massive_batch* io, const int64_t* nb,
                 const int64_t* eb, const StepBufs& sb) {
  hipStream_t s = c->s_main;
  const int slot = (int)(c->t % kSlots);
  ms::StepSizes* sz = sb.sz;
  int2* miss_list = sb.miss_list;
  const uint32_t key0 = (uint32_t)c->seed, key1 = (uint32_t)(c->seed >> 32);
  // this slot's sizes and lists were last used by the side stream kSlots
  // steps ago (complete: that batch was waited for)
  CK(hipStreamWaitEvent(s, c->ev_batch_done[slot], 0));
  // the scratch array may be shared with other contexts on this device: its
  // scan flags are cleared here (any epoch from 1 on is then fresh), and it is
  // cleared by fill kernels (nothing that a captured graph would replay wrongly)
  uint32_t scratch_epoch = 0;
  auto epoch = [&]() { return sb.from_scratch ? ++scratch_epoch : next_scan_epoch(c, s); };
  if (sb.from_scratch) {
    ms::k_fill<int32_t><<<1, 256, 0, s>>>(reinterpret_cast<int32_t*>(sz), (int64_t)(sizeof(ms::StepSizes) / 4), 0);
    const int64_t words = std::max(cdiv(nb[c->K], ms::kScanTile), cdiv(c->W, ms::kScanTile)) + 1;
    ms::k_fill<uint64_t><<<grid_for(words, 256, 64), 256, 0, s>>>(sb.flags, words, 0ull);
  } else if (!c->slot_clear[slot]) {
    // (a slot's sizes are cleared by the miss gather of the step that last
    // used it; the staged link and a context without halo nodes end a step
    // with k_step_done, which does not clear them)
    CK(hipMemsetAsync(sz, 0, sizeof(ms::StepSizes), s));
  }
  if (!sb.from_scratch) c->slot_clear[slot] = false;
  {
    massive_ctx::Range tr(c, s, 0);
    for (int k = 1; k <= c->K; ++k) {
      const int64_t nprev = nb[k - 1];
      const int64_t nbk = std::max<int64_t>(1, cdiv(nprev, ms::kScanTile));
      // the previous hop's relabel shares the launch
      const int64_t nrel = k > 1 ? (int64_t)grid_for(eb[k - 2], ms::kScanTile, 1024) : 0;
      // a large frontier lists every row for the one-wave-per-row sampler
      const bool by_waves = nprev > ms::kBlockRowsMax;
      ms::k_row_scan<<<(unsigned)(nbk + nrel), ms::kScanNT, 0, s>>>(
          c->d_indptr, io->nodes, sz, k, c->fo[k - 1], io->indptr[k - 1], sb.flags, epoch(),
          sb.big, c->big_min, nbk, k > 1 ? io->indices[k - 2] : nullptr, c->d_pos_of, by_waves ? nprev : 0,
          k == 1 ? seeds : nullptr, n0, c->L);
      ms::SampleArgs sa;
      sa.csr_indptr = c->d_indptr;
      sa.csr_indices = c->d_indices;
      sa.nodes = io->nodes;
      sa.sz = sz;
      sa.bptr = io->indptr[k - 1];
      sa.out = io->indices[k - 1];
      sa.hop = k;
      sa.fo = c->fo[k - 1];
      sa.t = (uint32_t)c->t;
      sa.key0 = key0;
      sa.key1 = key1;
      sa.err = &sz->status;
      sa.mu32 = c->mu32[k - 1];
      sa.big_min = c->big_min;
      sa.big_rows = sb.big;
      sa.pos_of = c->d_pos_of;
      sa.bits = c->d_bits;
      sa.tau_iters = c->tau_iters;
      // a small frontier is bound by its longest rows: a block each; a large
      // one keeps the chip busy: a wave each, longest first. The last hop's
      // dispatch can carry its own start/stop events (timing group 6).
      hipEvent_t hop_a = nullptr, hop_b = nullptr;
      const bool timed = k == c->K && c->kernel_pair(6, &hop_a, &hop_b);
      if (!by_waves) {
        sa.row_waves = 0;
        sa.big_blocks = std::max<int64_t>(1, std::min<int64_t>(nprev, c->big_blocks));
        const dim3 grid((unsigned)(sa.big_blocks + std::max<int64_t>(1, cdiv(nprev, ms::kSampleWaves))));
        if (timed)
          hipExtLaunchKernelGGL(ms::k_sample_blocks, grid, dim3(ms::kSampleWaves * MS_WAVE), 0, s, hop_a, hop_b, 0, sa);
        else
          ms::k_sample_blocks<<<grid, ms::kSampleWaves * MS_WAVE, 0, s>>>(sa);
      } else {
        sa.row_waves = nprev;  // the row list (nprev entries at most) ends there
        sa.big_blocks = 0;
        const dim3 grid((unsigned)std::max<int64_t>(1, cdiv(nprev, ms::kRowWaves)));
        if (timed)
          hipExtLaunchKernelGGL(ms::k_sample_waves, grid, dim3(ms::kRowWaves * MS_WAVE), 0, s, hop_a, hop_b, 0, sa);
        else
          ms::k_sample_waves<<<grid, ms::kRowWaves * MS_WAVE, 0, s>>>(sa);
      }
      if (timed) c->pending.push_back({hop_a, hop_b, 6});
      const int64_t nbw = std::max<int64_t>(1, cdiv(c->W, ms::kScanTile));
      ms::k_bits_scan<<<(unsigned)nbw, ms::kScanNT, 0, s>>>(c->d_bits, c->W, c->L, sz, k, sb.flags,
                                                             epoch(), io->nodes, c->d_pos_of);
      if (k == c->K)
        ms::k_relabel<<<grid_for(eb[k - 1], ms::kScanTile, 1024), ms::kScanNT, 0, s>>>(io->indices[k - 1], sz, k,
                                                                                     c->d_pos_of);
    }
  }
  // A refill that may still be in flight: hits on its slots read the host
  // store instead (same bytes); once it has landed the buffer serves them.
  int32_t pend = -1;
  if (c->round_pending_rows && c->staged()) {
    // the worker has enqueued the round's last chunk and that has run
    bool enq = false;
    if (c->chunks_left == 0) {
      std::lock_guard<std::mutex> lk(c->lmu);
      enq = c->fill_done_round == c->round_id && !c->lfailed;
    }
    if (enq && hipEventQuery(c->ev_fill_done) == hipSuccess) {
      c->round_pending_rows = false;
      CK(hipStreamWaitEvent(s, c->ev_fill_done, 0));
    } else {
      (void)hipGetLastError();
      pend = c->round_id;
    }
  } else if (c->round_pending_rows) {
    if (c->chunks_left == 0 && (!c->refill_inflight || hipEventQuery(c->ev_refill_done) == hipSuccess)) {
      c->round_pending_rows = false;
      if (c->refill_inflight) CK(hipStreamWaitEvent(s, c->ev_refill_done, 0));
      c->refill_inflight = false;
    } else {
      (void)hipGetLastError();
      pend = c->round_id;
    }
  }
  // the round owed by the previous step ran on the copy stream beside this
  // step's sampling; classify reads the buffer it rebuilt
  if (c->round_unclassified) {
    CK(hipStreamWaitEvent(s, c->ev_round_done, 0));
    c->round_unclassified = false;
  }
  {
    massive_ctx::Range tr(c, s, 1);
    ms::ClassifyArgs ca;
    ca.nodes = io->nodes;
    ca.sz = sz;
    ca.K = c->K;
    ca.L = c->L;
    ca.tab = c->d_tab;
    ca.tmask = c->hmask;
    ca.hitcnt = c->d_hitcnt;
    ca.S_A = c->d_S_A;
    ca.sa_idx = c->d_sa_idx;
    ca.pos_of = c->d_pos_of;
    ca.mask = io->mask;
    ca.hbm_list = sb.hbm_list;
    ca.miss_list = miss_list;
    ca.miss_slot = sb.miss_slot;
    ca.slot_round = c->d_slot_round;
    ca.landed = c->d_landed;
    ca.pend_round = pend;
    ca.seeds = seeds;
    ca.n0 = n0;
    // the frontier's size is known on the device only: at most kClsBlocks
    // blocks stride over it (a frontier far below the bound leaves the blocks
    // past its end idle, not a long tail of dispatches)
    ms::k_classify<<<grid_for(nb[c->K], ms::kClsNT * ms::kClsItems, ms::kClsBlocks), ms::kClsNT, 0, s>>>(ca);
  }
  CK(hipEventRecord(c->ev_cls_done[slot], s));
  // The gathers run on the side stream, so the main stream goes on to the
  // next step's sampling at once. HBM rows first, at full bandwidth: after the
  // previous step's miss gather (stream order) and the last refill chunk, as
  // concurrent host-link reads would throttle them; then the host-link rows,
  // beside the refill chunk launched after the HBM gather.
  hipStream_t sm = c->s_miss;
  CK(hipStreamWaitEvent(sm, c->ev_cls_done[slot], 0));
  if (c->refill_inflight) CK(hipStreamWaitEvent(sm, c->ev_refill_done, 0));
  launch_gather(c, 2, kHbm, sm, sb.hbm_list, &sz->n_hbm, c->d_slab, (uint8_t*)io->feat, c->rb, nb[c->K],
                c->hbm_blocks);
  CK(hipEventRecord(c->ev_hbm_done[slot], sm));
  if (c->staged()) {
    // the host rows go to the worker, which enqueues the rest of the step
    // (and then one refill chunk) on the link stream
    if (c->H > 0) {
      ms::k_rows_out<<<grid_for(std::min<int64_t>(nb[c->K], c->H), 256, 1024), 256, 0, sm>>>(
          miss_list, &sz->n_miss, c->H, c->hd_rows[slot], c->hd_cnt + slot);
      CK(hipEventRecord(c->ev_rows_ready[slot], sm));
    }
    CK(hipGetLastError());
    massive_ctx::LinkJob j;
    j.slot = slot;
    j.step = c->t;
    j.list = miss_list;
    j.wslot = sb.miss_slot;
    j.feat = (uint8_t*)io->feat;
    j.sz = sz;
    j.pend = pend >= 0 && c->H > 0 ? pend : -1;
    j.nbK = nb[c->K];
    j.rows = c->H > 0;
    j.timing = c->timing;
    link_post(c, j);
    link_post_chunks(c, 1);
    c->infl[slot].io = io;
    c->infl[slot].step = c->t;
    c->infl[slot].seeds = seeds;
    c->infl[slot].n0 = n0;
    c->t += 1;
    c->pending_round = true;
    return MASSIVE_OK;
  }
  {
    int rc = launch_refill_chunks(c, 1, c->ev_hbm_done[slot]);
    if (rc != MASSIVE_OK) return rc;
  }
  // the miss gather ends the step: it stamps the slots it writes through as
  // landed and publishes the step's sizes to the host mailbox (a context
  // without halo nodes publishes them with a kernel of its own)
  const ms::StepTail tail{sz, c->K, &c->d_ctr->bad, c->hd_sz + slot, c->hd_bad + slot, c->d_landed, c->cap,
                          pend, 1};
  if (c->H > 0) {
    const bool heavy = c->round_pending_rows || c->host_rows_seen < 0 || c->host_rows_seen * c->rb > kLinkHeavyBytes;
    launch_gather(c, 3, kMiss, sm, miss_list, &sz->n_miss, c->d_store, (uint8_t*)io->feat, c->rb, nb[c->K],
                  heavy ? c->host_blocks : c->host_blocks_light, sb.miss_slot, c->d_slab + (int64_t)c->L * c->rb,
                  &tail);
    if (!sb.from_scratch) c->slot_clear[slot] = true;
  }
  else
    ms::k_step_done<<<1, 256, 0, sm>>>(sb.miss_slot, &sz->n_miss, c->d_landed, c->cap, -1, sz, c->K,
                                       &c->d_ctr->bad, c->hd_sz + slot, c->hd_bad + slot);
  // (also the miss gather's completion, which the next round's refill follows)
  CK(hipEventRecord(c->ev_batch_done[slot], sm));
  CK(hipGetLastError());
  c->infl[slot].io = io;
  c->infl[slot].step = c->t;
  c->infl[slot].seeds = seeds;
  c->infl[slot].n0 = n0;
  c->t += 1;
  c->pending_round = true;
  return MASSIVE_OK;
}

}  // namespace

extern "C" {

int massive_sample_async(massive_ctx* c, const int32_t* seeds, int32_t n0, massive_batch* io) {
  if (!c) return MASSIVE_EINVAL;
  int64_t nb[MASSIVE_MAX_HOPS + 1], eb[MASSIVE_MAX_HOPS];
  int rc = check_step_args(c, seeds, n0, io, nb, eb);
  if (rc != MASSIVE_OK) return rc;
  const int slot = (int)(c->t % kSlots);
  if (c->infl[slot].io)
    return c->fail(MASSIVE_ESTATE, "%d batches in flight: wait for the oldest one first", kSlots);
  const StepBufs sb{c->d_sz + slot, c->d_hbm_list[slot], c->d_miss_list[slot], c->d_miss_slot[slot], c->d_big,
                    c->d_scan_flags, false};
  rc = enqueue_step(c, seeds, n0, io, nb, eb, sb);
  // a HIP call that failed part-way left work on the queues that no batch
  // tracks: the context takes no further work
  if (rc == MASSIVE_EHIP) c->broken = true;
  return rc;
}

int massive_batch_wait(massive_ctx* c, massive_batch* io) {
  if (!c || !io) return MASSIVE_EINVAL;
  int slot = -1;
  for (int i = 0; i < kSlots; ++i)
    if (c->infl[i].io == io) slot = i;
  if (slot < 0) return c->fail(MASSIVE_EINVAL, "this batch is not in flight");
  const massive_ctx::InFlight f = c->infl[slot];
  c->infl[slot] = massive_ctx::InFlight();
  if (c->staged()) {  // the worker has enqueued the tails of this step and the earlier ones
    const int64_t st = f.step;
    const int rc = link_wait(c, [c, st] { return c->tail_step >= st; });
    if (rc != MASSIVE_OK) return rc;
  }
  CK(hipEventSynchronize(c->ev_batch_done[slot]));
  // Steps issued before this one and still in flight decide whether it is
  // valid: a step that failed on the device skipped its dedup scan and its
  // classify, so its bitmap marks and frontier positions stayed set, and every
  // later step sampled against them.
  for (int i = 0; i < kSlots; ++i)
    if (c->infl[i].io && c->infl[i].step < f.step) {
      CK(hipEventSynchronize(c->ev_batch_done[i]));
      if ((c->h_sz[i].status || c->h_bad[i]) && (c->failed_step < 0 || c->infl[i].step < c->failed_step))
        c->failed_step = c->infl[i].step;
    }
  if (c->failed_step >= 0 && f.step > c->failed_step) {
    c->broken = true;
    return c->fail(MASSIVE_ESTATE, "step %lld failed before this batch (step %lld) was complete: its outputs are "
                                   "not valid and the context is unusable",
                   (long long)c->failed_step, (long long)f.step);
  }
  const ms::StepSizes& z = c->h_sz[slot];
  if (c->h_bad[slot]) {
    c->broken = true;
    c->failed_step = f.step;
    return c->fail(MASSIVE_EHIP, "an eviction round produced inconsistent indices");
  }
  if (z.status & 3) {
    // the step left no trace on the device; it can be taken back if nothing
    // was issued after it
    const char* why = (z.status & 1) ? "a seed is not a local node id" : "a seed is repeated";
    bool alone = true;
    for (int i = 0; i < kSlots; ++i) alone = alone && !c->infl[i].io;
    if (f.step == c->t - 1 && c->pending_round && alone) {
      c->t -= 1;
      c->pending_round = false;
      return c->fail(MASSIVE_EINVAL, "%s", why);
    }
    c->broken = true;
    c->failed_step = f.step;
    return c->fail(MASSIVE_EINVAL, "%s (later work was already issued: context unusable)", why);
  }
  if (z.status) {
    c->broken = true;
    c->failed_step = f.step;
    return c->fail(MASSIVE_EHIP, "%s (status %d)",
                   (z.status & 8) ? "a single-pass scan waited past its bound" : "sampler could not isolate a candidate set",
                   z.status);
  }
  for (int k = 0; k <= c->K; ++k) io->n[k] = z.n[k];
  for (int k = 0; k < c->K; ++k) io->e[k] = z.e[k];
  io->local = z.local;
  io->hits = z.hits;
  io->misses = z.misses;
  io->host_rows = z.n_miss;
  c->host_rows_seen = z.n_miss;
  return MASSIVE_OK;
}

int massive_sample(massive_ctx* c, const int32_t* seeds, int32_t n0, massive_batch* io) {
  int rc = massive_sample_async(c, seeds, n0, io);
  if (rc != MASSIVE_OK) return rc;
  return massive_batch_wait(c, io);
}

int massive_sample_noalloc(massive_ctx* c, const int32_t* seeds, int32_t n0, massive_batch* io) {
  if (!c) return MASSIVE_EINVAL;
  int64_t nb[MASSIVE_MAX_HOPS + 1], eb[MASSIVE_MAX_HOPS];
  int rc = check_step_args(c, seeds, n0, io, nb, eb);
  if (rc != MASSIVE_OK) return rc;
  for (int i = 0; i < kSlots; ++i)
    if (c->infl[i].io) return c->fail(MASSIVE_ESTATE, "a batch is in flight: wait for it before a no-alloc step");
  if (nb[c->K] > kNoAllocMaxRows)
    return c->fail(MASSIVE_ECAPACITY, "the no-alloc scratch holds %lld frontier rows, this batch's bound is %lld "
                                      "(massive_sample has no such limit)",
                   (long long)kNoAllocMaxRows, (long long)nb[c->K]);
  const int64_t words = std::max(cdiv(nb[c->K], ms::kScanTile), cdiv(c->W, ms::kScanTile)) + 1;
  if (words > kNoAllocFlagWords)
    return c->fail(MASSIVE_ECAPACITY, "the no-alloc scratch holds %lld scan flags, this step needs %lld",
                   (long long)kNoAllocFlagWords, (long long)words);
  if (!c->d_scratch) return c->fail(MASSIVE_EHIP, "the no-alloc scratch has no device address");
  uint8_t* base = c->d_scratch;
  StepBufs sb;
  sb.sz = reinterpret_cast<ms::StepSizes*>(base);
  sb.hbm_list = reinterpret_cast<int2*>(base + 512);
  sb.miss_list = sb.hbm_list + kNoAllocMaxRows;
  sb.miss_slot = reinterpret_cast<int32_t*>(sb.miss_list + kNoAllocMaxRows);
  sb.big = sb.miss_slot + kNoAllocMaxRows;
  sb.flags = reinterpret_cast<uint64_t*>(sb.big + kNoAllocMaxRows);
  sb.from_scratch = true;
  // timing events are created on demand: this path records none
  const int timing = c->timing;
  c->timing = 0;
  rc = enqueue_step(c, seeds, n0, io, nb, eb, sb);
  c->timing = timing;
  if (rc == MASSIVE_EHIP) c->broken = true;  // as in massive_sample_async
  if (rc != MASSIVE_OK) return rc;
  return massive_batch_wait(c, io);
}

}  // extern "C"

namespace {

int evict_step_impl(massive_ctx* c, int32_t* evicted, int32_t* slots, int32_t* replaced, int64_t* k_out) {
  if (c->broken) return c->fail(MASSIVE_ESTATE, "context is unusable after an earlier failure");
  if (!c->pending_round) return c->fail(MASSIVE_ESTATE, "no sampled step owes an eviction round");
  if (k_out) *k_out = 0;
  const int64_t tl = c->t - 1;
  if (!(tl > 0 && tl % c->delta == 0) || c->cap == 0) {
    c->pending_round = false;
    return MASSIVE_OK;
  }
  for (const void* p : {(const void*)evicted, (const void*)slots, (const void*)replaced})
    if (p && !device_visible(p)) return c->fail(MASSIVE_EINVAL, "an eviction output is not HIP-visible memory");
  c->pending_round = false;
  // The round runs on the copy stream, beside the next step's sampling on
  // the main stream (the next classify waits for it). It follows, in stream
  // order, the previous round's refill chunks, which read the fill list, the
  // round state and the slot stamps that it rewrites; it starts after this
  // step's classify and HBM gather (hit counts, scores; the gather runs alone).
  hipStream_t s = c->s_copy;
  const int64_t cap = c->cap, H = c->H;
  ms::RoundState* rs = c->d_rs;
  if (c->staged()) {
    // The previous round's refill has landed before this round reassigns
    // slots and rewrites the fill list and its host rows: its chunks are
    // posted, the worker has enqueued the last one, and the round waits for it.
    link_post_chunks(c, c->chunks_left);
    if (c->round_id > 0) {
      const int32_t prev = c->round_id;
      const int rc = link_wait(c, [c, prev] { return c->fill_done_round >= prev; });
      if (rc != MASSIVE_OK) return rc;
      CK(hipStreamWaitEvent(s, c->ev_fill_done, 0));
    }
  } else {
    int rc = launch_refill_chunks(c, c->chunks_left, nullptr);
    if (rc != MASSIVE_OK) return rc;
  }
  c->round_pending_rows = false;
  CK(hipStreamWaitEvent(s, c->ev_hbm_done[tl % kSlots], 0));
  {
    massive_ctx::Range tr(c, s, 4);
    ms::k_materialize<<<grid_for(cap, 256), 256, 0, s>>>(c->d_S_E, c->d_hitcnt, cap, (int32_t)(c->t - c->mat_t),
                                                          c->gamma);
    c->mat_t = c->t;
    CK(hipMemsetAsync(rs, 0, sizeof(ms::RoundState), s));
    const int64_t nbe = std::max<int64_t>(1, cdiv(cap, ms::kScanTile));
    ms::k_evict_count<<<(unsigned)nbe, ms::kScanNT, 0, s>>>(c->d_S_E, cap, c->alpha, c->d_part, &rs->nE);
    ms::k_evict_emit<<<(unsigned)nbe, ms::kScanNT, 0, s>>>(c->d_S_E, cap, c->alpha, c->d_part, c->d_E);
    ms::k_round_setup<<<1, 1, 0, s>>>(rs, c->d_ctr, H - cap);
    // fewer candidates than evictions: keep the k' slots of smallest (S_E,
    // rank). With |C| = H - cap >= cap >= |E| (f <= 50%) it cannot happen and
    // the narrowing is not launched; otherwise its kernels see zero elements
    // in rounds where it does not happen.
    if (cap > H - cap) {
      ms::k_esel_keys_lo<<<grid_for(cap, 256), 256, 0, s>>>(c->d_E, &rs->nE_sel, c->d_slot_id, c->d_rank_of,
                                                            c->d_k0, c->d_v0);
      sort_u32(c, s, &rs->nE_sel, 0, cap, nullptr);
      ms::k_esel_keys_hi<<<grid_for(cap, 256), 256, 0, s>>>(c->d_v0, &rs->nE_sel, c->d_S_E, c->d_k0);
      sort_u32(c, s, &rs->nE_sel, 0, cap, nullptr);
      ms::k_esel_keys_slot<<<grid_for(cap, 256), 256, 0, s>>>(c->d_v0, &rs->k_sel, c->d_k0);
      sort_u32(c, s, &rs->k_sel, 0, cap, c->d_E);
    }
    ms::k_fill_gated<int32_t><<<grid_for(cap, 256), 256, 0, s>>>(c->d_R, cap, -1, &rs->k);
    if (c->layout == MASSIVE_SCORES_BY_GID) {
      // S_A over every global id, scanned in id order: an exact radix select
      // over the 64-bit key (score word, rank), then the k' keys below or at
      // it, sorted by rank and then stably by score
      const int64_t n = c->n_sa;
      for (int word = 0; word < 2; ++word)
        for (int shift = 24; shift >= 0; shift -= 8) {
          ms::k_gselect_hist<<<grid_for(cdiv(n, 4), 256, 4096), 256, 0, s>>>(c->d_S_A, c->d_rank_g, n, rs, word,
                                                                           shift, c->d_ghist);
          ms::k_select_pick<<<1, 256, 0, s>>>(rs, c->d_ghist, shift, &c->d_ctr->bad, word);
        }
      const int64_t nbg = std::max<int64_t>(1, cdiv(n, ms::kScanTile));
      ms::k_gsel_count<<<(unsigned)nbg, ms::kScanNT, 0, s>>>(c->d_S_A, c->d_rank_g, n, rs, c->d_gpart);
      ms::k_scan_partials<<<1, ms::kScanNT, 0, s>>>(c->d_gpart, nbg, nullptr, nullptr);
      ms::k_gsel_emit<<<(unsigned)nbg, ms::kScanNT, 0, s>>>(c->d_S_A, c->d_rank_g, c->d_h_of_rank, n, rs,
                                                            c->d_gpart, c->d_k0, c->d_v0);
      sort_u32(c, s, &rs->k, 0, cap, nullptr);
      ms::k_gsel_keys<<<grid_for(cap, 256), 256, 0, s>>>(c->d_v0, &rs->k, c->d_S_A, c->d_sa_idx, c->d_k0);
      sort_u32(c, s, &rs->k, 0, cap, c->d_R);
    } else {
      // radix select of the k'-th candidate key, 8 bits per pass
      for (int shift = 24; shift >= 0; shift -= 8) {
        ms::k_select_hist<<<grid_for(H, 256, 2048), 256, 0, s>>>(c->d_S_A, H, rs, shift, c->d_ghist);
        ms::k_select_pick<<<1, 256, 0, s>>>(rs, c->d_ghist, shift, &c->d_ctr->bad);
      }
      const int64_t nbh = std::max<int64_t>(1, cdiv(H, ms::kScanTile));
      ms::k_rank_count<<<(unsigned)nbh, ms::kScanNT, 0, s>>>(c->d_S_A, H, rs, c->d_part, c->d_part2);
      ms::k_rank_emit<<<(unsigned)nbh, ms::kScanNT, 0, s>>>(c->d_S_A, c->d_h_of_rank, H, rs, c->d_part, c->d_part2,
                                                            c->d_k0, c->d_v0, c->d_R);
      // candidates before the threshold: stable sort by key (S_A desc), rank order kept for ties
      sort_u32(c, s, &rs->n_lt, 0, cap, c->d_R);
    }
    c->round_id += 1;
    ms::k_swap<<<grid_for(cap, 256), 256, 0, s>>>(c->d_E, c->d_R, &rs->k, c->L, cap, c->H, c->d_slot_id, c->d_S_E,
                                                  c->d_S_A, c->d_sa_idx, evicted, slots, replaced, c->d_fill, &c->d_ctr->bad,
                                                  c->d_slot_round, c->round_id);
    ms::k_fill_gated<uint64_t><<<grid_for(c->hcap, 256), 256, 0, s>>>(c->d_tab, c->hcap, ms::kEmpty, &rs->k);
    ms::k_hash_insert<<<grid_for(cap, 256), 256, 0, s>>>(c->d_tab, c->hmask, c->d_slot_id, cap, &rs->k);
  }
  if (c->staged()) {  // the fill list's host rows, for the worker's refill chunks
    ms::k_rows_out<<<grid_for(cap, 256, 1024), 256, 0, s>>>(c->d_fill, &rs->k, cap, c->hd_fill_rows,
                                                            c->hd_cnt + kSlots);
    CK(hipEventRecord(c->ev_fill_ready, s));
  }
  if (k_out) {
    CK(hipMemcpyAsync(&c->h_rs->k, &rs->k, 8, hipMemcpyDeviceToHost, s));
    CK(hipMemcpyAsync(c->h_ctr, c->d_ctr, sizeof(ms::Counters), hipMemcpyDeviceToHost, s));
  }
  CK(hipEventRecord(c->ev_round_done, s));
  c->round_unclassified = true;
  // the refill is copied in chunks after the next steps' HBM gathers; the last
  // step's miss gather may still write rows of the previous round's
  // replacements into slots this round reassigns, so the new refill comes after
  // it (in the staged mode the link stream orders them: the worker enqueues
  // the new chunks after that step's tail)
  if (!c->staged()) CK(hipStreamWaitEvent(s, c->ev_batch_done[tl % kSlots], 0));
  c->chunks_left = c->refill_chunks;
  c->round_pending_rows = true;
  CK(hipGetLastError());
  if (k_out) {
    CK(hipEventSynchronize(c->ev_round_done));
    if (c->h_ctr->bad) {
      c->broken = true;
      return c->fail(MASSIVE_EHIP, "eviction round produced inconsistent indices");
    }
    *k_out = c->h_rs->k;
  }
  return MASSIVE_OK;
}

}  // namespace

extern "C" {

int massive_evict_step(massive_ctx* c, int32_t* evicted, int32_t* slots, int32_t* replaced, int64_t* k_out) {
  if (!c) return MASSIVE_EINVAL;
  const int rc = evict_step_impl(c, evicted, slots, replaced, k_out);
  // a round that failed part-way on a HIP call leaves the buffer state
  // undefined: the context takes no further work
  if (rc == MASSIVE_EHIP) c->broken = true;
  return rc;
}

int massive_get_counters(massive_ctx* c, int64_t* rounds, int64_t* evicted, int64_t* refilled) {
  if (!c) return MASSIVE_EINVAL;
  {
    const int rc = link_drain(c);  // staged refill chunks posted so far
    if (rc != MASSIVE_OK) return rc;
  }
  CK(hipStreamSynchronize(c->s_copy));  // refill chunks launched so far
  CK(hipMemcpyAsync(c->h_ctr, c->d_ctr, sizeof(ms::Counters), hipMemcpyDeviceToHost, c->s_main));
  CK(hipStreamSynchronize(c->s_main));
  if (rounds) *rounds = c->h_ctr->rounds;
  if (evicted) *evicted = c->h_ctr->evicted;
  if (refilled) *refilled = c->h_ctr->refilled;
  return MASSIVE_OK;
}

int massive_get_state(massive_ctx* c, int32_t* slot_id, float* S_E, float* S_A, int64_t* t) {
  if (!c) return MASSIVE_EINVAL;
  {
    const int rc = link_drain(c);
    if (rc != MASSIVE_OK) return rc;
  }
  hipStream_t s = c->s_main;
  CK(hipStreamSynchronize(c->s_miss));
  if (c->round_unclassified) CK(hipStreamWaitEvent(s, c->ev_round_done, 0));
  if (c->cap > 0 && c->t > c->mat_t) {
    ms::k_materialize<<<grid_for(c->cap, 256), 256, 0, s>>>(c->d_S_E, c->d_hitcnt, c->cap,
                                                             (int32_t)(c->t - c->mat_t), c->gamma);
    c->mat_t = c->t;
  }
  if (slot_id && c->cap) CK(hipMemcpyAsync(slot_id, c->d_slot_id, c->cap * 4, hipMemcpyDeviceToHost, s));
  if (S_E && c->cap) CK(hipMemcpyAsync(S_E, c->d_S_E, c->cap * 4, hipMemcpyDeviceToHost, s));
  if (S_A && c->H) {
    // S_A is kept by halo rank or by global id; export it by halo id (through
    // a sort buffer, free once the last round has completed)
    float* by_id = reinterpret_cast<float*>(c->d_v1);
    ms::k_scores_by_id<<<grid_for(c->H, 256), 256, 0, s>>>(c->d_S_A, c->d_sa_idx, c->H, by_id);
    CK(hipMemcpyAsync(S_A, by_id, (int64_t)c->H * 4, hipMemcpyDeviceToHost, s));
  }
  CK(hipStreamSynchronize(s));
  if (t) *t = c->t;
  return MASSIVE_OK;
}

int massive_get_buffer_rows(massive_ctx* c, void* out) {
  if (!c || (!out && c->cap)) return MASSIVE_EINVAL;
  if (c->staged()) {  // every chunk of the round, through the worker
    link_post_chunks(c, c->chunks_left);
    const int rc = link_drain(c);
    if (rc != MASSIVE_OK) return rc;
  } else {
    int rc = launch_refill_chunks(c, c->chunks_left, nullptr);
    if (rc != MASSIVE_OK) return rc;
  }
  if (c->refill_inflight) CK(hipStreamWaitEvent(c->s_main, c->ev_refill_done, 0));
  CK(hipStreamSynchronize(c->s_miss));  // rows written through by miss gathers
  if (c->cap)
    CK(hipMemcpyAsync(out, c->d_slab + (int64_t)c->L * c->rb, c->cap * c->rb, hipMemcpyDeviceToHost, c->s_main));
  CK(hipStreamSynchronize(c->s_main));
  return MASSIVE_OK;
}

int massive_info(const massive_ctx* c, int64_t* cap, float* alpha) {
  if (!c) return MASSIVE_EINVAL;
  if (cap) *cap = c->cap;
  if (alpha) *alpha = c->alpha;
  return MASSIVE_OK;
}

int massive_set_timing(massive_ctx* c, int groups) {
  if (!c) return MASSIVE_EINVAL;
  if (groups & ~MASSIVE_TIMING_ALL) return c->fail(MASSIVE_EINVAL, "timing groups 0x%x outside 0x%x", groups,
                                                   MASSIVE_TIMING_ALL);
  {
    const int rc = link_drain(c);
    if (rc != MASSIVE_OK) return rc;
  }
  CK(hipDeviceSynchronize());
  c->resolve_timing();
  c->timing = groups;
  for (int i = 0; i < kTimingGroups; ++i) {
    c->tms[i] = 0.0;
    c->tcalls[i] = 0;
  }
  return MASSIVE_OK;
}

int massive_get_timing(massive_ctx* c, double* out_ms, int64_t* out_calls) {
  if (!c) return MASSIVE_EINVAL;
  {
    const int rc = link_drain(c);
    if (rc != MASSIVE_OK) return rc;
  }
  CK(hipStreamSynchronize(c->s_main));
  CK(hipStreamSynchronize(c->s_miss));
  CK(hipStreamSynchronize(c->s_copy));
  c->resolve_timing();
  for (int i = 0; i < kTimingGroups; ++i) {
    if (out_ms) out_ms[i] = c->tms[i];
    if (out_calls) out_calls[i] = c->tcalls[i];
  }
  return MASSIVE_OK;
}

int massive_destroy(massive_ctx* c) {
  free_ctx(c);
  return MASSIVE_OK;
}

const char* massive_last_error(const massive_ctx* c) {
  if (!c) return g_init_error.c_str();
  return c->err.c_str();
}

}  // extern "C"
