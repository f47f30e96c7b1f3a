// Fused MoE GEMM2 + combine for gfx950 (MI355X), and its C ABI.
//
// One persistent kernel, two workgroup roles (paper: Background,
// "Fine-Grained Overlap and GPU Residency"; Method, "Split-level
// dependency"):
//
//  * compute workgroups walk the global tile sequence (split-major, then
//    expert, then m-tile, then n-tile; compute workgroup b takes tiles b,
//    b+P, b+2P, ...), run one 256x256 tile of Y = x_perm @ W2[e] on bf16
//    MFMA with LDS double buffering and store it to the bf16 staging
//    buffer; after its last tile of a split a workgroup publishes all its
//    tiles of that split (one agent-scope release, then their flags);
//  * consumer workgroups wait until every tile of a split is published
//    (agent-scope acquire), then, per task of 64 tokens x 1024 columns,
//    gather each token's rows, weight them by the gates and write the
//    token's output once, summing the rows in ascending row order so the
//    result does not depend on the partition.
//
// Every workgroup first adds its share of rows to the token->rows inverse
// map.  Flags and counters carry the launch's epoch, so nothing has to be
// cleared between launches and a stale value can never satisfy a wait.
// Compute workgroups never wait while they hold tiles.  With C = 0 they
// serve consumer tasks afterwards, and then wait on other workgroups' tiles:
// they do so only once every workgroup of the grid has started (a started
// counter), else they leave the tasks to the workgroups started later, so a
// launch that shares the GPU with another never waits on workgroups that
// cannot get a CU.  Every consumer wait is bounded.
#include <hip/hip_runtime.h>

#include <atomic>
#include <chrono>
#include <cstddef>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <random>
#include <unordered_map>

#include "moe_gemm2.h"

namespace {

constexpr int kThreads = 512;           // 8 waves of 64, two per SIMD
constexpr int kBM = 256;                // compute tile rows (routed rows)
constexpr int kBN = 256;                // compute tile columns (hidden)
constexpr int kBK = 64;                 // reduction step of one LDS stage
constexpr int kStages = 2;              // LDS ring depth
constexpr int kResidentPerCu = 1;       // one workgroup (eight waves, 256 registers each) per CU
constexpr int kCommTM = 64;             // consumer task: tokens (at most; fewer for small batches)
constexpr int kCommTMMin = 16;          // consumer task: tokens (at least)
constexpr int kTaskTarget = 512;        // owner-write tasks wanted per launch (two per CU)
constexpr int kCommTN = 1024;           // consumer task: columns (at most)
constexpr int kMaxE = 1024;
constexpr int kMaxSplits = 16;
constexpr int kMaxBandTab = 2048;       // (E + 1) * L entries of the token-band tables
constexpr int kMaxTopk = 64;
constexpr int kMaxGrid = 4096;
constexpr int kRotMinRounds = 16;   // launches this long rotate their rounds

// Y rows are padded by 128 bytes: with a power-of-two pitch (H = 2048: 4 KB)
// the rows of a tile fall on few memory channels, which cost ~18% of the
// write bandwidth of row-strided stores in a microbenchmark.
constexpr int kYPad = 64;     // Y row padding, elements
// Every 128-byte line of Y is written by exactly one compute tile: rows
// start on a line, and so does each column split's segment of a row.  (Two
// workgroups writing disjoint parts of one line was measured to lose data
// now and then, when they ran on different XCDs.)
constexpr int kYLine = 64;    // elements per 128-byte line
__host__ __device__ inline int round_up_line(int n) { return (n + kYLine - 1) / kYLine * kYLine; }
constexpr uint32_t kStBadRouting = 1u;
constexpr uint32_t kStTimeout = 2u;

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned long long u64;

struct KArgs {
  const uint16_t* x;          // [rows, I] bf16
  const uint16_t* w2;         // [E, I, H] bf16
  const int32_t* offsets;     // [E+1]
  const int32_t* token_ids;   // [rows]
  const float* gate_w;        // [rows]
  float* out;                 // [T, H]
  uint16_t* Y;                // [rows, ypitch] bf16 staging
  uint32_t* tile_flags;       // [max_tiles]: epoch once tile g is published
  uint32_t* wg_flags;         // [kMaxGrid]: epoch once workgroup b added its inverse-map rows
  u64* tok_cnt;               // [T]: launch-tagged count of each token's rows
  int32_t* inv;               // [T, topk]
  uint32_t* status;           // [1]
  u64* trace;                 // optional
  long long rows;             // capacity of x / Y / token_ids / gate_w
  long long max_tiles;        // capacity of tile_flags
  long long spin_limit;
  int T, H, I, E, topk, L;
  int ypitch;                 // row pitch of Y in elements: L ysplit + kYPad
  int ysplit;                 // elements of a row's segment for one split (nsplit rounded up
                              // to a line); column c of split s is at s ysplit + c - s nsplit
  int nsplit;                 // columns per split (H / L)
  int ntps;                   // compute n-tiles per split
  int C, P;                   // consumer and compute workgroups
  int drain;                  // compute workgroups also take consumer tasks
  int comm_tm;                // consumer task tokens (<= kCommTM)
  int comm_tn;                // consumer task width (<= kCommTN)
  int cb_per_split;           // consumer column blocks per split
  int tasks_per_split;
  int comm_tm_last;           // owner-write (column splits): tokens of the last split's
  int tasks_last;             //   tasks (finer, so that the launch ends evenly) and their count
  u64* epoch_word;            // the workspace's last completed launch epoch
  uint32_t* done_ctr;         // workgroups of this launch that have finished
  uint32_t* start_ctr;        // workgroups of this launch that have started
  int delay_mod;              // debug: compute workgroups c % delay_mod == 0 delay
  long long delay_ticks;      //   each split publish by delay_ticks (100 MHz), else 0
  uint32_t* task_ctr;         // [kMaxSplits]: next consumer task of each split (reset by
                              // workgroup 0 each launch)
  uint32_t* split_flags;      // [L, kMaxGrid]: epoch once compute workgroup c has published
                              // all its tiles of split s (or has none there); column splits
  int mode;                   // 0 owner-write, 1 fp32 atomic scatter, 2 owner-write over
                              // token bands (splits along the routed rows)
};

// Arguments of the up-projection stage (grouped GEMM1 with the SwiGLU
// activation): x_perm[r, c] = silu(h_r . Wg[e(r)][:, c]) * (h_r . Wu[e(r)][:, c])
// with h_r = hidden[token_ids[r]], the tokens gathered by the loads.
struct G1Args {
  const uint16_t* hidden;     // [T, H] bf16
  const uint16_t* w1;         // [E, H, 2I] bf16, gate and up interleaved in 16-column blocks
  const int32_t* offsets;     // [E+1]
  const int32_t* token_ids;   // [rows]
  uint16_t* xout;             // [rows, I] bf16
  uint32_t* status;           // [1]
  long long rows;             // capacity of token_ids / xout
  int T, H, I, E;
  int ntps;                   // n-tiles of the packed 2I columns
  int nsplit;                 // = 2I (one split)
};

// The grouped GEMM core below serves two stages through these accessors:
// its reduction length, the row length of its B operand, B of expert e, and
// where the A rows of a tile live: the base its loads address, the bytes
// readable from there, and the byte offset of the tile's row `row`.
__device__ __forceinline__ int gemm_k(const KArgs& a) { return a.I; }
__device__ __forceinline__ int gemm_ldb(const KArgs& a) { return a.H; }
__device__ __forceinline__ const uint16_t* gemm_b(const KArgs& a, int e) {
  return a.w2 + (size_t)e * a.I * a.H;
}
__device__ __forceinline__ const uint16_t* gemm_a_base(const KArgs& a, long long r0) {
  return a.x + (size_t)r0 * a.I;
}
__device__ __forceinline__ long long gemm_a_bytes(const KArgs& a, long long r0) {
  return (a.rows - r0) * a.I * 2;
}
__device__ __forceinline__ uint32_t gemm_a_off(const int* rowtok, const KArgs& a, int row) {
  return (uint32_t)row * (uint32_t)a.I * 2u;
}
__device__ __forceinline__ int gemm_k(const G1Args& a) { return a.H; }
__device__ __forceinline__ int gemm_ldb(const G1Args& a) { return 2 * a.I; }
__device__ __forceinline__ const uint16_t* gemm_b(const G1Args& a, int e) {
  return a.w1 + (size_t)e * a.H * (2 * a.I);
}
// the A rows are gathered: row `row` is hidden[token], the token staged in LDS
__device__ __forceinline__ const uint16_t* gemm_a_base(const G1Args& a, long long r0) {
  return a.hidden;
}
__device__ __forceinline__ long long gemm_a_bytes(const G1Args& a, long long r0) {
  return (long long)a.T * a.H * 2;
}
__device__ __forceinline__ uint32_t gemm_a_off(const int* rowtok, const G1Args& a, int row) {
  return (uint32_t)rowtok[row] * (uint32_t)a.H * 2u;
}
template <class Args> struct RowGather { static constexpr bool on = false; };
template <> struct RowGather<G1Args> { static constexpr bool on = true; };

struct Smem {
  uint16_t a[kStages][kBM * kBK];  // x tile: row m = kBK/8 chunks of 8 k (swizzled)
  uint16_t b[kStages][kBK * kBN];  // W2 tile: row k = 32 chunks of 8 n (swizzled)
  int start[kMaxE];           // sanitized first row of each expert
  int count[kMaxE];           // sanitized row count of each expert
  int tile_prefix[kMaxE + 1]; // exclusive prefix of ceil(count/kBM)
  int scan[kThreads / 64];   // per-wave totals of the expert scan
  int rowtok[kBM];            // gathering stages: token of each row of the staged tile
  int band_pre[kMaxBandTab];  // token bands: [b (E+1) + e] exclusive prefix over experts of
                              // band b's m-tile counts
  int band_start[kMaxSplits + 1];  // token bands: first global tile of each band
  int flag;
  int task;                   // consumer task claimed by the workgroup
  int task_band;              // token bands: last band holding a row of the staged task
  int prefix_end;             // end of the published prefix found by wait_prefix
  int split_seen;             // a split's workgroup flags all set, seen with the claim
  u64 epoch;                  // this launch's epoch, read once at the start
};

// ---- memory-model helpers ----------------------------------------------------
__device__ __forceinline__ u64 ld_relaxed(u64* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Per-token row counters: the launch counter (mod 2^40) in the high 40
// bits, the count in the low 24; a counter from an older launch counts as
// zero.  Launch counters only grow, so an atomic max opens a launch's count.
constexpr int kCntBits = 24;
constexpr u64 kCntMask = (1ull << kCntBits) - 1;

__device__ __forceinline__ uint32_t epoch_count(u64 v, u64 cnt_epoch) {
  return (v & ~kCntMask) == cnt_epoch ? (uint32_t)(v & kCntMask) : 0u;
}

// The launch's epoch: one more than the workspace's last completed launch,
// whose last workgroup to finish stored it.  Stream order makes that store
// visible to the next launch, also when both are replays of one captured
// graph (whose kernel arguments cannot change), and no workgroup of this
// launch changes it before every workgroup is done.  Readiness flags hold
// its low 32 bits (never 0, the cleared state); per-token counters hold it
// mod 2^40 above a 24-bit count.
// The epoch is read once per workgroup at the start, into LDS (a global
// load later would be waited for together with the ring loads in flight).
__device__ __forceinline__ u64 launch_epoch(const KArgs& a) {
  return __hip_atomic_load(a.epoch_word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1;
}
// Agent-scope release and acquire with the wait for the cache operation
// itself.  The release writes back the L2 (buffer_wbl2) and the acquire
// invalidates it (buffer_inv); both are vector memory operations counted in
// vmcnt.  The compiler places its wait after them only while it tracks some
// other vector memory operation in flight, and here the callers have waited
// for everything already, so it drops the wait: a flag store could then
// become visible before the written-back lines, or the barrier could let the
// workgroup's other waves read before the invalidate has finished.  The
// explicit wait closes both.
__device__ __forceinline__ void release_agent() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}
__device__ __forceinline__ void acquire_agent() {
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

__device__ __forceinline__ uint32_t flag_epoch(const Smem& sm) { return (uint32_t)sm.epoch; }
__device__ __forceinline__ u64 count_epoch(const Smem& sm) {
  return (sm.epoch & ((1ull << (64 - kCntBits)) - 1)) << kCntBits;
}

__device__ __forceinline__ u64 now_100mhz() { return __builtin_amdgcn_s_memrealtime(); }

// threadIdx.x, opaque to the compiler: per-lane addresses derived from it
// are then recomputed where used instead of being hoisted out of the tile
// loop, where the register budget would spill them (and a spill reload's
// wait would also wait for the ring loads in flight).
__device__ __forceinline__ int opaque_tid() {
  int t = threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}

// Wave 0 polls flags[0..n) until every flag equals the epoch (bounded),
// advancing past the leading run of set flags; then, with `acquire`, the
// whole workgroup acquires (without it, a later acquire must precede any
// read of the data these flags publish).  Returns false (and records a
// timeout) if the bound expired.
// One polling round trip of wave 0 over flags [i, min(i + kPollSpan, n)):
// every lane loads kPollPerLane flags (64 apart, so each load instruction
// reads 64 consecutive flags) before any is tested, so a split of ~1600
// flags takes a few round trips of the agent-coherent loads instead of 25.
// Returns the offset from i of the first flag not yet published, or
// kPollSpan when all of them are (flags past n count as published).
constexpr int kPollPerLane = 8;
constexpr int kPollSpan = 64 * kPollPerLane;
__device__ __forceinline__ int first_unpublished(uint32_t* flags, long long i, long long n,
                                                 uint32_t epoch, int lane) {
  uint32_t v[kPollPerLane];
#pragma unroll
  for (int j = 0; j < kPollPerLane; ++j) {
    const long long idx = i + 64 * j + lane;
    v[j] = idx < n ? __hip_atomic_load(&flags[idx], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                   : epoch;
  }
#pragma unroll
  for (int j = 0; j < kPollPerLane; ++j) {
    const u64 ready = __ballot(v[j] == epoch);
    if (ready != ~0ull) return 64 * j + (int)__builtin_ctzll(~ready);
  }
  return kPollSpan;
}

__device__ bool wait_flags(Smem& sm, uint32_t* flags, long long n, const KArgs& a,
                           bool acquire = true) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    const uint32_t epoch = flag_epoch(sm);
    long long i = 0, spins = 0;
    int ok = 1;
    while (i < n) {
      const int first = first_unpublished(flags, i, n, epoch, lane);
      if (first == kPollSpan) {
        i += kPollSpan;
        continue;
      }
      i += first;   // leading set flags stay set
      if (++spins > a.spin_limit) {
        ok = 0;
        if (lane == 0)
          __hip_atomic_fetch_or(a.status, kStTimeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
      __builtin_amdgcn_s_sleep(8);
    }
    if (lane == 0) sm.flag = ok;
  }
  __syncthreads();
  const bool ok = sm.flag != 0;
  // One agent-scope acquire per workgroup, by the wave that saw the flags:
  // it invalidates the CU's L1 and the XCD's L2, which every wave of the
  // workgroup shares, and the barrier orders the other waves' reads after
  // it.  (An acquire in every wave made eight L2 invalidates per workgroup;
  // with all workgroups acquiring at once they queued for microseconds.)
  if (acquire && threadIdx.x < 64) acquire_agent();
  __syncthreads();  // sm.flag may be rewritten by the next wait
  return ok;
}

// The acquire of wait_flags alone, for flags already seen published.
__device__ __forceinline__ void acquire_workgroup() {
  if (threadIdx.x < 64) acquire_agent();
  __syncthreads();
}

// Waits until flags [from, need) are published, then extends the prefix over
// the flags that are already published up to `limit` (without waiting), and
// acquires once for the whole prefix (wave 0 polls; the same bound as
// wait_flags).  Returns the end of the published prefix (>= need), or -1 if
// the bound expired.  A consumer that keeps the returned end needs no wait
// and no acquire for the tiles before it, so it acquires once per catch-up
// with the compute workgroups rather than once per task.
__device__ long long wait_prefix(Smem& sm, uint32_t* flags, long long from, long long need,
                                 long long limit, const KArgs& a) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    const uint32_t epoch = flag_epoch(sm);
    long long i = from, spins = 0;
    int ok = 1;
    while (i < need) {
      const int first = first_unpublished(flags, i, need, epoch, lane);
      if (first == kPollSpan) {
        i += kPollSpan;
        continue;
      }
      i += first;
      if (++spins > a.spin_limit) {
        ok = 0;
        if (lane == 0)
          __hip_atomic_fetch_or(a.status, kStTimeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
      __builtin_amdgcn_s_sleep(8);
    }
    if (ok) {
      if (i > need) i = need;
      while (i < limit) {
        // flags past limit must stop the prefix: test them as unpublished
        const int first = first_unpublished(flags, i, limit, epoch, lane);
        const long long room = limit - i;
        if (first == kPollSpan && room > kPollSpan) {
          i += kPollSpan;
          continue;
        }
        i += first < room ? first : room;
        break;
      }
    }
    if (lane == 0) {
      sm.flag = ok;
      sm.prefix_end = (int)i;
    }
  }
  __syncthreads();
  const bool ok = sm.flag != 0;
  const long long end = sm.prefix_end;
  if (ok && threadIdx.x < 64) acquire_agent();
  __syncthreads();  // sm.flag and sm.prefix_end may be rewritten by the next wait
  return ok ? end : -1;
}

// ---- prologue: expert ranges and the routed-tile prefix ----------------------
// Each expert's row range is clamped into [0, rows] with end >= start, so
// every row range stays inside the buffers even for bad input (which is
// flagged); overlapping ranges from bad input compute some rows twice (with
// meaningless values), and a tile count past the workspace's capacity makes
// the compute workgroups stop (flagged) instead of indexing past it.
template <class Args>
__device__ void load_experts(Smem& sm, const Args& a) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  // each thread takes a contiguous chunk of experts for both passes
  const int chunk = (a.E + kThreads - 1) / kThreads;
  const int lo = min(a.E, tid * chunk), hi = min(a.E, lo + chunk);
  bool bad = false;
  int local = 0;   // m-tiles of the chunk
  for (int e = lo; e < hi; ++e) {
    long long s = a.offsets[e], en = a.offsets[e + 1];
    if (e == 0 && s != 0) bad = true;
    if (en < s || en > a.rows) bad = true;
    s = s < 0 ? 0 : (s > a.rows ? a.rows : s);
    en = en < s ? s : (en > a.rows ? a.rows : en);
    sm.start[e] = (int)s;
    sm.count[e] = (int)(en - s);
    local += (int)((en - s + kBM - 1) / kBM);
  }
  if (bad && a.status)
    __hip_atomic_fetch_or(a.status, kStBadRouting, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // exclusive scan of the chunks' m-tiles: inclusive within each wave by
  // shuffles, then the totals of the waves before (two barriers in all)
  int v = local;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int u = __shfl_up(v, d);
    if (lane >= d) v += u;
  }
  if (lane == 63) sm.scan[wave] = v;
  __syncthreads();
  int before = 0;
  for (int w = 0; w < wave; ++w) before += sm.scan[w];
  int run = before + v - local;
  for (int e = lo; e < hi; ++e) {
    sm.tile_prefix[e] = run;
    run += (sm.count[e] + kBM - 1) / kBM;
  }
  if (tid == kThreads - 1) sm.tile_prefix[a.E] = before + v;
  __syncthreads();
}

// What the consumers need before their first task, built by every
// workgroup for its share: for the owner-write combine, the rows of each
// token (the inverse map); for the atomic scatter, a zeroed output.  With
// `publish`, the workgroup's share is published at once (release + its
// workgroup flag); otherwise the caller publishes it later, with its first
// split's tiles (one L2 write-back for both).
__device__ void consumer_prologue(const Smem& sm, const KArgs& a, long long rows_dev, bool publish) {
  const long long stride = (long long)gridDim.x * kThreads;
  if (a.mode == 1) {
    // out as 16-byte words, split into one contiguous range per workgroup
    const long long words = (long long)a.T * a.H / 4;
    const long long per = (words + gridDim.x - 1) / gridDim.x;
    const long long lo = (long long)blockIdx.x * per;
    const long long hi = min(words, lo + per);
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    for (long long i = lo + threadIdx.x; i < hi; i += kThreads)
      __builtin_nontemporal_store(z, (f32x4*)a.out + i);
    rows_dev = 0;   // no inverse map
  }
  const u64 cnt_epoch = count_epoch(sm);
  for (long long r = (long long)blockIdx.x * kThreads + threadIdx.x; r < rows_dev; r += stride) {
    const int t = a.token_ids[r];
    if (t < 0 || t >= a.T) {
      __hip_atomic_fetch_or(a.status, kStBadRouting, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      continue;
    }
    // Open this launch's count (a counter from an older launch holds a
    // smaller epoch in its high word), then take a slot.  The two atomics
    // of a thread on one address are performed in order, so the add always
    // sees this epoch; no compare-and-swap, no dependent round trip.
    __hip_atomic_fetch_max(&a.tok_cnt[t], cnt_epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const u64 old = __hip_atomic_fetch_add(&a.tok_cnt[t], 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t slot =
        (old & ~kCntMask) == cnt_epoch ? (uint32_t)(old & kCntMask) : 0xffffffffu;
    if (slot >= (uint32_t)a.topk) {
      __hip_atomic_fetch_or(a.status, kStBadRouting, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      continue;
    }
    a.inv[(long long)t * a.topk + slot] = (int32_t)r;
  }
  // workgroup 0 resets the consumer task counters; every claim of split s
  // comes after the claimer has seen workgroup 0's release (its inverse-map
  // flag, or its publish of split s), so after these stores
  if (blockIdx.x == 0 && threadIdx.x < a.L)
    __hip_atomic_store(&a.task_ctr[threadIdx.x], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (!publish) return;
  // as for a split: per-wave vmcnt(0), barrier, one release by thread 0
  __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (0 << 8));
  __syncthreads();
  if (threadIdx.x == 0) {
    release_agent();
    __hip_atomic_store(&a.wg_flags[blockIdx.x], flag_epoch(sm), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  }
}

// ---- compute role: one 256x256 tile ------------------------------------------
// The MFMA computes D = Y^T for the tile: its A operand is W2^T (rows n) and
// its B operand is x (columns m), 8 consecutive k per lane.  Eight waves (two
// per SIMD, 4 along n x 2 along m) each own 64 n x 128 m as 2 x 4 blocks of
// v_mfma_f32_32x32x16_bf16: with two waves per SIMD one wave's MFMAs run
// while the other waits for its LDS fragments, and the wave tile keeps the
// costly transposing reads (W2) at one 16 KB pass per K=16 step per CU.
//
// Operands reach LDS by direct buffer->LDS loads (no registers) through a
// ring of kStages stages of kBK reduction steps, kStages - 1 stages ahead of
// the MFMAs:
//  * x stage: 256 rows of 2 kBK bytes (kBK/8 chunks of 8 k); chunk c of row
//    m sits at chunk c ^ ((m / r) % (kBK/8)), r = rows per 256-byte bank
//    line, so the 16 rows one 16-lane group of a 16-byte read touches fill
//    all 64 banks;
//  * W2 stage: kBK rows (k) of 512 bytes (32 chunks of 8 n); chunk c of row
//    k sits at chunk c ^ 4(k & 3), so the 32 lanes of a transposing read
//    (4 rows x 64 bytes) hit 64 distinct banks.
// x fragments are plain 16-byte LDS reads.  W2 is stored as in memory (n
// contiguous) and read with ds_read_b64_tr_b16: in each group of 16 lanes,
// lane i receives element i%4 of the 8-byte reads of lanes 4p + i/4
// (p = 0..3), so pointing lane j at row k0 + j/4, columns c(j%4)..+3 hands
// lane i the 4 consecutive k of column c(i/4) + i%4.
// MFMA row rho = 8q + 4h + r (q < 4, h < 2, r < 4) of an n-block is mapped
// to column 16(q/2) + 8h + 4(q%2) + r, so a lane's accumulators 8c..8c+7
// are 8 consecutive columns of one row of Y (one 16-byte store).
constexpr int kWaves = kThreads / 64;
constexpr int kWN = 64;              // wave tile: n
constexpr int kWM = 128;             // wave tile: m
constexpr int kWavesN = kBN / kWN;
constexpr int kNB = kWN / 32;
constexpr int kMB = kWM / 32;
constexpr int kKS = kBK / 16;                          // MFMA K steps per stage
constexpr int kStageElems = kBM * kBK;                 // == kBK * kBN
constexpr int kLoadsPerOperand = kStageElems * 2 / 1024 / kWaves;   // 1 KB loads per wave
constexpr int kLoadsPerStage = 2 * kLoadsPerOperand;
constexpr int kXRowsPerLoad = 1024 / (2 * kBK);
constexpr int kXChunks = kBK / 8;
constexpr int kXRowsPerLine = 256 / (2 * kBK);
static_assert((kBN / kWN) * (kBM / kWM) == kWaves, "wave grid");
static_assert(kBM * kBK == kBK * kBN, "stage sizes");
static_assert(kKS % 2 == 0, "fragment double buffer parity must carry across stages");
static_assert(kStages >= 2 && (kStages - 1) * kLoadsPerStage <= 63, "vmcnt range");

typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// One 16-byte-per-lane buffer -> LDS load: lane L's 16 bytes, at byte
// offset voff of the buffer rsrc describes, land at lds_base + 16 L; an
// offset at or past the buffer's extent reads zeros.  Issued as asm so the
// compiler does not serialise later LDS reads behind it; completion is
// tracked with explicit vmcnt waits.  (Buffer addressing, a 32-bit offset
// per lane against a base in scalar registers, keeps the texture
// addresser's work per load lower than 64-bit global addresses: measured,
// the same ring with global_load_lds_dwordx4 spends up to a third more
// time per stage.)
typedef int i32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void dma16(i32x4 rsrc, uint32_t voff, uint32_t lds_base) {
  // (the resource is wave-uniform; readfirstlane keeps it in scalar
  // registers also where the compiler cannot prove that)
  i32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) r[i] = __builtin_amdgcn_readfirstlane(rsrc[i]);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(__builtin_amdgcn_readfirstlane(lds_base)), "v"(voff), "s"(r)
               : "memory", "m0");
}

// A raw buffer resource: base address, no stride, `bytes` readable (at most
// 2^31 - 1, so that kOutOfRange is always past it), wave-uniform.
constexpr uint32_t kOutOfRange = 0x80000000u;
__device__ __forceinline__ i32x4 buffer_rsrc(const void* base, long long bytes) {
  const uint64_t b = (uint64_t)(uintptr_t)base;
  const long long n = bytes < 0 ? 0 : (bytes > 0x7fffffffLL ? 0x7fffffffLL : bytes);
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)b);
  r[1] = __builtin_amdgcn_readfirstlane((int)(uint32_t)((b >> 32) & 0xffffu));
  r[2] = __builtin_amdgcn_readfirstlane((int)n);
  r[3] = 0x00020000;   // raw 32-bit data format (gfx9 family)
  return r;
}

// Stores issued as asm, like the ring loads: the compiler then does not
// track them, and so does not wait for them (a wait that, vmcnt being in
// order, would also wait for the next tile's ring stages issued after
// them) before it reuses their source registers at the next tile's start.
// The data registers are read shortly after issue; the s_nop covers the
// hazard of overwriting them in the next instructions.  Completion is
// ordered by the explicit vmcnt waits before a publish.
__device__ __forceinline__ void store16_nt(void* p, u32x4 v) {
  asm volatile("global_store_dwordx4 %0, %1, off nt\n\ts_nop 1" : : "v"(p), "v"(v) : "memory");
}
__device__ __forceinline__ void store8(void* p, u64 v) {
  asm volatile("global_store_dwordx2 %0, %1, off\n\ts_nop 1" : : "v"(p), "v"(v) : "memory");
}

template <int N>
__device__ __forceinline__ void waitcnt_vm() {
  // s_waitcnt encoding: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt_hi[15:14]
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
}

// Waits until the stage that is `newer` stages older than the newest one
// issued has landed for this wave (all its LDS operations done as well).
__device__ __forceinline__ void wait_stage(int newer) {
  static_assert(kStages <= 4, "extend wait_stage");
  if (newer >= 3) waitcnt_vm<3 * kLoadsPerStage>();
  else if (newer == 2) waitcnt_vm<2 * kLoadsPerStage>();
  else if (newer == 1) waitcnt_vm<kLoadsPerStage>();
  else waitcnt_vm<0>();
}

__device__ __forceinline__ void block_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

struct TileCtx {
  i32x4 ra, rb;                           // buffers of the tile's A rows and B columns
  uint32_t xo[kLoadsPerOperand];          // this lane's A chunk for its loads (bytes, k offset 0)
  uint32_t wo[kLoadsPerOperand];          // this lane's B chunk for its loads (bytes, k offset 0)
  int xk[kLoadsPerOperand];               // k offset of the chunk each x load fetches
  int wk[kLoadsPerOperand];               // k row (within a stage) each W2 load fetches
  uint32_t lds_a, lds_b;                  // LDS addresses of stage 0
};

// Issue load q (q < kLoadsPerOperand) of each operand of reduction stage kt
// into ring slot `slot`.  Every load is issued, so each stage adds exactly
// kLoadsPerStage to vmcnt; lanes whose chunk lies past the reduction
// (k >= I) read past the buffer's extent, which loads zeros into both
// operands there.
template <class Args>
__device__ __forceinline__ void issue_load(const Args& a, const TileCtx& t, int kt, int slot,
                                           int wave, int q) {
  const int k0 = kt * kBK;
  const uint32_t blk = (uint32_t)(slot * kStageElems + (kLoadsPerOperand * wave + q) * 512) * 2;
  const int kx = k0 + t.xk[q];
  dma16(t.ra, kx < gemm_k(a) ? t.xo[q] + 2u * (uint32_t)k0 : kOutOfRange, t.lds_a + blk);
  const int kw = k0 + t.wk[q];
  dma16(t.rb, kw < gemm_k(a) ? t.wo[q] + 2u * (uint32_t)k0 * (uint32_t)gemm_ldb(a) : kOutOfRange,
        t.lds_b + blk);
}

template <class Args>
__device__ __forceinline__ void issue_stage(const Args& a, const TileCtx& t, int kt, int slot,
                                            int wave) {
#pragma unroll
  for (int q = 0; q < kLoadsPerOperand; ++q) issue_load(a, t, kt, slot, wave, q);
}

// One operand's half of a stage: the B (W2) loads, or the A (x) loads.
template <class Args>
__device__ __forceinline__ void issue_stage_b(const Args& a, const TileCtx& t, int kt, int slot,
                                              int wave) {
  const int k0 = kt * kBK;
#pragma unroll
  for (int q = 0; q < kLoadsPerOperand; ++q) {
    const uint32_t blk = (uint32_t)(slot * kStageElems + (kLoadsPerOperand * wave + q) * 512) * 2;
    const int kw = k0 + t.wk[q];
    dma16(t.rb, kw < gemm_k(a) ? t.wo[q] + 2u * (uint32_t)k0 * (uint32_t)gemm_ldb(a) : kOutOfRange,
          t.lds_b + blk);
  }
}
template <class Args>
__device__ __forceinline__ void issue_stage_a(const Args& a, const TileCtx& t, int kt, int slot,
                                              int wave) {
  const int k0 = kt * kBK;
#pragma unroll
  for (int q = 0; q < kLoadsPerOperand; ++q) {
    const uint32_t blk = (uint32_t)(slot * kStageElems + (kLoadsPerOperand * wave + q) * 512) * 2;
    const int kx = k0 + t.xk[q];
    dma16(t.ra, kx < gemm_k(a) ? t.xo[q] + 2u * (uint32_t)k0 : kOutOfRange, t.lds_a + blk);
  }
}

typedef const __attribute__((address_space(3))) uint16_t lds_u16;

// MFMA operands of K=16 step ks of a ring slot: W2^T blocks by two
// transposing 8-byte reads, x blocks by one 16-byte read.
__device__ __forceinline__ void load_frags(lds_u16* As, lds_u16* Bs, const int (&offA)[kNB],
                                           const int (&offB)[kKS], int ks,
                                           bf16x8 (&af)[kNB], bf16x8 (&bm)[kMB]) {
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(Bs + offA[nb] + ks * 16 * kBN));
    const i16x4 hi =
        __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(Bs + offA[nb] + ks * 16 * kBN + 4 * kBN));
    const i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    af[nb] = __builtin_bit_cast(bf16x8, v);
  }
#pragma unroll
  for (int mb = 0; mb < kMB; ++mb)
    bm[mb] = *(const __attribute__((address_space(3))) bf16x8*)(As + offB[ks] + mb * 32 * kBK);
}

// The 16 MFMAs of one K=16 step of the wave's 128 x 128 block.
__device__ __forceinline__ void mfma_step(f32x16 (&acc)[kNB][kMB], const bf16x8 (&af)[kNB],
                                          const bf16x8 (&bm)[kMB]) {
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
    for (int mb = 0; mb < kMB; ++mb)
      acc[nb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[nb], bm[mb], acc[nb][mb], 0, 0, 0);
}

// The first K=16 step of a tile: every accumulator from zero (an inline
// zero operand, so no register clearing before it).
__device__ __forceinline__ void mfma_step_zero(f32x16 (&acc)[kNB][kMB], const bf16x8 (&af)[kNB],
                                               const bf16x8 (&bm)[kMB]) {
  const f32x16 z = {};
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
    for (int mb = 0; mb < kMB; ++mb)
      acc[nb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[nb], bm[mb], z, 0, 0, 0);
}

// mfma_step with loads q0 .. q0+kNB-1 of stage kt issued one after each
// n-block of MFMAs: spread out, the loads never hold the wave's in-order
// issue long enough to starve the matrix core.
template <class Args>
__device__ __forceinline__ void mfma_step_loads(f32x16 (&acc)[kNB][kMB], const bf16x8 (&af)[kNB],
                                                const bf16x8 (&bm)[kMB], const Args& a,
                                                const TileCtx& t, int kt, int slot, int wave,
                                                int q0, bool on) {
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
#pragma unroll
    for (int mb = 0; mb < kMB; ++mb)
      acc[nb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[nb], bm[mb], acc[nb][mb], 0, 0, 0);
    if (on) issue_load(a, t, kt, slot, wave, q0 + nb);
  }
}

// One compute tile: expert e, rows r0 .. r0+rows_valid-1 of x_perm,
// columns n0 .. n0+cols_valid-1 of Y.
struct TileInfo {
  int e, r0, rows_valid, n0, cols_valid;
  int ny0;   // Y column of the tile's first column (the split's line-aligned segment)
};

// Gathering stages: the token of tile row threadIdx.x (rows past the
// expert repeat its last row), loaded from token_ids.  The id is checked
// only when it is staged (gather_commit, after a wait that covers the load
// anyway): an id outside [0, T) is flagged and replaced by 0, so that every
// load of the hidden rows stays in bounds.
__device__ __forceinline__ int gather_load(const G1Args& a, const TileInfo& ti) {
  const int i = threadIdx.x;
  if (i >= kBM) return 0;
  const long long r = (long long)ti.r0 + (i < ti.rows_valid ? i : ti.rows_valid - 1);
  return a.token_ids[r];
}
__device__ __forceinline__ void gather_commit(Smem& sm, const G1Args& a, int t) {
  if (threadIdx.x < kBM) {
    if (t < 0 || t >= a.T) {
      __hip_atomic_fetch_or(a.status, kStBadRouting, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      t = 0;
    }
    sm.rowtok[threadIdx.x] = t;
  }
}

__device__ __forceinline__ int y_split_pitch(const KArgs& a) { return a.ysplit; }
__device__ __forceinline__ int y_split_pitch(const G1Args& a) { return a.nsplit; }

// The last index i in [0, n) with pre[i] <= v, for a non-decreasing pre with
// pre[0] <= v, found by the whole wave: each round tests 64 evenly spaced
// candidates at once (one LDS read per lane) and keeps the gap after the
// last one that passes, so E <= 64 experts take one round trip instead of
// log2(E) dependent ones.  Every lane of the wave must take part.
__device__ __forceinline__ int wave_last_le(const int* pre, int n, int v) {
  const int lane = threadIdx.x & 63;
  int lo = 0, len = n;   // the answer lies in [lo, lo + len); pre[lo] <= v
  while (len > 64) {
    const int step = (len + 63) >> 6;
    const int i = lo + lane * step;
    const u64 m = __ballot(lane * step < len && pre[i] <= v);
    const int j = 63 - __builtin_clzll(m);   // lane 0 always passes
    lo += j * step;
    len = min(step, len - j * step);
  }
  const u64 m = __ballot(lane < len && pre[lo + lane] <= v);
  return lo + 63 - __builtin_clzll(m);
}

// Tile g of the global sequence (split-major, then expert, m-tile, n-tile).
// Every tile count fits in 32 bits (checked on the host for the worst case
// of overlapping expert ranges).
template <class Args>
__device__ TileInfo decode_tile(const Smem& sm, const Args& a, int W_comp, int g) {
  const int s = g / W_comp;
  const int idx = g - s * W_comp;
  const int mt = idx / a.ntps;
  const int nt = idx - mt * a.ntps;
  // expert owning m-tile mt: last e with tile_prefix[e] <= mt
  const int lo = wave_last_le(sm.tile_prefix, a.E, mt);
  TileInfo ti;
  ti.e = lo;
  ti.r0 = sm.start[lo] + (mt - sm.tile_prefix[lo]) * kBM;
  ti.rows_valid = min(kBM, sm.start[lo] + sm.count[lo] - ti.r0);
  ti.n0 = s * a.nsplit + nt * kBN;
  ti.cols_valid = min(kBN, (s + 1) * a.nsplit - ti.n0);
  ti.ny0 = s * y_split_pitch(a) + nt * kBN;
  return ti;
}

// ---- token bands (mode 2) ------------------------------------------------------
// The pipeline splits run along the routed rows instead of the columns: each
// expert's n_e = ceil(count_e / kBM) m-tiles are cut into L consecutive runs,
// band b holding m-tiles [b n_e / L, (b+1) n_e / L), and every band covers
// the full width H.  The global tile sequence is band -> expert -> m-tile ->
// n-tile, so the n-tiles of an m-tile stay together (its x rows are read once
// for all of H) and, with rows sorted by token inside each expert, band b
// holds about the tokens [b T / L, (b+1) T / L).  A consumer task waits for
// the bands that hold its rows (computed from the rows themselves, so any
// row order is correct).
__device__ __forceinline__ int band_lo(int n, int b, int L) { return (int)((long long)b * n / L); }

// band_pre and band_start from the expert table (wave w scans bands w, w+8..)
__device__ void load_bands(Smem& sm, const KArgs& a) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int E1 = a.E + 1;
  for (int b = wave; b < a.L; b += kThreads / 64) {
    int carry = 0;
    for (int e0 = 0; e0 < a.E; e0 += 64) {
      const int e = e0 + lane;
      int c = 0;
      if (e < a.E) {
        const int n = (sm.count[e] + kBM - 1) / kBM;
        c = band_lo(n, b + 1, a.L) - band_lo(n, b, a.L);
      }
      int v = c;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int u = __shfl_up(v, d);
        if (lane >= d) v += u;
      }
      if (e < a.E) sm.band_pre[b * E1 + e] = carry + v - c;
      carry += __shfl(v, 63);
    }
    if (lane == 0) sm.band_pre[b * E1 + a.E] = carry;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int b = 0; b < a.L; ++b) {
      sm.band_start[b] = run;
      run += sm.band_pre[b * E1 + a.E] * a.ntps;
    }
    sm.band_start[a.L] = run;
  }
  __syncthreads();
}

__device__ __forceinline__ int band_of_tile(const Smem& sm, const KArgs& a, int g) {
  int b = 0;
  while (b + 1 < a.L && sm.band_start[b + 1] <= g) ++b;
  return b;
}

// Tile g of the band sequence.
__device__ TileInfo decode_band_tile(const Smem& sm, const KArgs& a, int g) {
  const int b = band_of_tile(sm, a, g);
  const int idx = g - sm.band_start[b];
  const int mt = idx / a.ntps;
  const int nt = idx - mt * a.ntps;
  const int* pre = sm.band_pre + b * (a.E + 1);
  // last expert whose band-b run starts at or before mt
  const int lo = wave_last_le(pre, a.E, mt);
  const int n_e = (sm.count[lo] + kBM - 1) / kBM;
  const int i = band_lo(n_e, b, a.L) + (mt - pre[lo]);
  TileInfo ti;
  ti.e = lo;
  ti.r0 = sm.start[lo] + i * kBM;
  ti.rows_valid = min(kBM, sm.count[lo] - i * kBM);
  ti.n0 = nt * kBN;
  ti.cols_valid = min(kBN, a.H - ti.n0);
  ti.ny0 = ti.n0;
  return ti;
}

// The band of the m-tile holding permuted row r (L - 1 for a row outside
// every expert's range, possible only with bad offsets: such a task then
// waits for every band).
__device__ __forceinline__ int band_of_row(const Smem& sm, const KArgs& a, int r) {
  int lo = 0, hi = a.E - 1;
  while (lo < hi) {   // last expert starting at or before r
    const int mid = (lo + hi + 1) >> 1;
    if (sm.start[mid] <= r) lo = mid; else hi = mid - 1;
  }
  const int off = r - sm.start[lo];
  if (off < 0 || off >= sm.count[lo]) return a.L - 1;
  const int n_e = (sm.count[lo] + kBM - 1) / kBM;
  const int i = off / kBM;
  return (int)(((long long)(i + 1) * a.L + n_e - 1) / n_e) - 1;
}

// This lane's global addresses for its loads of a tile's stages.
template <class Args>
__device__ __forceinline__ TileCtx make_ctx(Smem& sm, const Args& a, const TileInfo& ti, int wave) {
  const int lane = threadIdx.x & 63;
  const int e = ti.e, r0 = ti.r0, rows_valid = ti.rows_valid, n0 = ti.n0, cols_valid = ti.cols_valid;
  TileCtx t;
  t.lds_a = lds_addr(&sm.a[0][0]);
  t.lds_b = lds_addr(&sm.b[0][0]);
  {
    const int ldb = gemm_ldb(a);
    t.ra = buffer_rsrc(gemm_a_base(a, r0), gemm_a_bytes(a, r0));
    t.rb = buffer_rsrc(gemm_b(a, e) + n0, ((long long)gemm_k(a) * ldb - n0) * 2);
#pragma unroll
    for (int q = 0; q < kLoadsPerOperand; ++q) {
      const int i = kLoadsPerOperand * wave + q;   // 1 KB block of the stage
      // x: rows kXRowsPerLoad i + L / kXChunks, physical chunk L % kXChunks
      const int row = kXRowsPerLoad * i + lane / kXChunks;
      const int lc = (lane % kXChunks) ^ ((row / kXRowsPerLine) % kXChunks);
      // rows past the expert and columns past the tile are never stored:
      // their loads take an offset past the buffer (zeros, no memory request)
      const int grow = row < rows_valid ? row : rows_valid - 1;
      t.xk[q] = 8 * lc;
      t.xo[q] = row < rows_valid ? gemm_a_off(sm.rowtok, a, grow) + 2u * (uint32_t)t.xk[q]
                                 : kOutOfRange;
      // W2: rows 2i + L/32, physical chunk L%32
      const int krow = 2 * i + (lane >> 5);
      const int wc = (lane & 31) ^ (4 * (krow & 3));
      t.wk[q] = krow;
      t.wo[q] = 8 * wc < cols_valid ? 16u * (uint32_t)wc + 2u * (uint32_t)krow * (uint32_t)ldb
                                    : kOutOfRange;
    }
  }
  return t;
}

// The loads of a tile's first min(kStages, nk) stages (its ring fill), the
// tile's stage 0 going into ring slot `base`.
template <class Args>
__device__ __forceinline__ void issue_prologue(const Args& a, const TileCtx& t, int nk, int base,
                                               int wave) {
#pragma unroll
  for (int s = 0; s < kStages; ++s)
    if (s < nk) issue_stage(a, t, s, (base + s) % kStages, wave);
}

// The K=16 steps of one stage boundary: the last step of stage kt (MFMAs on
// fragments read before the boundary) and the other steps of stage kt+1
// (slot s1), with the loads of stage `ls` of the tile `tl` into slot `lslot`
// spread over the first kLoadSteps steps.
template <class Args>
__device__ __forceinline__ void boundary_steps(f32x16 (&acc)[kNB][kMB], bf16x8 (&af)[2][kNB],
                                               bf16x8 (&bm)[2][kMB], const Args& a,
                                               lds_u16* As1, lds_u16* Bs1, const int (&offA)[kNB],
                                               const int (&offB)[kKS], const TileCtx& tl, int ls,
                                               int lslot, int wave, bool on) {
  constexpr int kLoadSteps = kLoadsPerOperand / kNB;   // steps that carry a stage's loads
  load_frags(As1, Bs1, offA, offB, 0, af[0], bm[0]);
  __builtin_amdgcn_sched_barrier(0);
  mfma_step_loads(acc, af[(kKS - 1) & 1], bm[(kKS - 1) & 1], a, tl, ls, lslot, wave, 0, on);
#pragma unroll
  for (int ks = 0; ks + 1 < kKS; ++ks) {
    load_frags(As1, Bs1, offA, offB, ks + 1, af[(ks + 1) & 1], bm[(ks + 1) & 1]);
    __builtin_amdgcn_sched_barrier(0);
    if (ks + 1 < kLoadSteps)
      mfma_step_loads(acc, af[ks & 1], bm[ks & 1], a, tl, ls, lslot, wave, (ks + 1) * kNB, on);
    else
      mfma_step(acc, af[ks & 1], bm[ks & 1]);
  }
}

// The tile's Y rows: bf16 through the LDS slot `eslot` to whole-line stores.
__device__ __forceinline__ void epilogue_store(Smem& sm, const KArgs& a, f32x16 (&acc)[kNB][kMB],
                                               int eslot, int lane, int wave, int wn0, int wm0,
                                               const TileInfo& ti) {
  const int rows_valid = ti.rows_valid, cols_valid = ti.cols_valid, r0 = ti.r0;
  // The wave's kWM x kWN block goes through LDS one 32-row m-block at a
  // time (4 KB per wave, all eight in the x part of slot eslot, so that its
  // W2 part can take the next tile's stage already) as bf16 rows of 2 kWN
  // bytes, 16-byte chunk j of row r at chunk j ^ ((r / r1) % c), c = chunks
  // per row, r1 = rows per 256-byte bank line (so 16 consecutive rows hit
  // 16 distinct bank groups), then leaves as whole rows of 2 kWN bytes (full
  // 128-byte lines).  A wave's LDS operations run in order, so each pass may
  // overwrite the previous one once its reads were issued.
  constexpr int kEpChunks = kWN / 8;
  constexpr int kEpRowsPerLine = 256 / (2 * kWN);
  constexpr int kEpRowsPerStore = 64 / kEpChunks;
  constexpr int kEpRows = 32;                       // rows per pass: one m-block
  static_assert(kWaves * kEpRows * kWN <= kStageElems,
                "one pass of every wave fits in the x part of a slot");
  const int h = lane >> 5;
  __attribute__((address_space(3))) uint16_t* ep =
      (__attribute__((address_space(3))) uint16_t*)(uintptr_t)lds_addr(&sm.a[eslot][0]) +
      wave * (kEpRows * kWN);
  const int j = lane % kEpChunks;
  const int n = wn0 + 8 * j;
  const bool n_ok = n < cols_valid;
#pragma unroll
  for (int mb = 0; mb < kMB; ++mb) {
    {
      const int row = lane & 31;
      const int sw = (row / kEpRowsPerLine) % kEpChunks;
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          bf16x8 v;
#pragma unroll
          for (int i = 0; i < 8; ++i) v[i] = (__bf16)acc[nb][mb][8 * c + i];
          const int chunk = 4 * nb + 2 * c + h;
          *(__attribute__((address_space(3))) bf16x8*)(ep + row * kWN + ((chunk ^ sw) << 3)) = v;
        }
    }
#pragma unroll
    for (int it = 0; it < kEpRows / kEpRowsPerStore; ++it) {
      const int row = kEpRowsPerStore * it + lane / kEpChunks;
      const int m = wm0 + kEpRows * mb + row;
      const int sw = (row / kEpRowsPerLine) % kEpChunks;
      const bf16x8 v =
          *(const __attribute__((address_space(3))) bf16x8*)(ep + row * kWN + ((j ^ sw) << 3));
      if (n_ok && m < rows_valid)
        store16_nt(a.Y + (size_t)(r0 + m) * a.ypitch + ti.ny0 + n, __builtin_bit_cast(u32x4, v));
    }
  }
}

// The up-projection tile's outputs.  In the packed W1 a 32-column block is
// 16 gate columns followed by the up columns of the same 16 outputs, and the
// MFMA row remap gives lane half h the accumulators 8c..8c+7 = 8 consecutive
// columns 32nb + 16c + 8h.., so a lane holds the gate (c = 0) and the up
// (c = 1) values of the same 8 outputs: act = silu(gate) * up in fp32,
// rounded once to bf16.  The workgroup's 256 x 128 outputs go through the
// LDS slot eslot (rows 0..127 in its x part, 128..255 in its W part; 16-byte
// chunk c of row r at c ^ (r % 16), so 16 rows' chunks hit 16 distinct bank
// groups) and leave as whole 256-byte row pieces of x_perm.
__device__ __forceinline__ void epilogue_store(Smem& sm, const G1Args& a, f32x16 (&acc)[kNB][kMB],
                                               int eslot, int lane, int wave, int wn0, int wm0,
                                               const TileInfo& ti) {
  constexpr int kOut = kBN / 2;           // output columns per tile
  constexpr int kChunks = kOut / 8;       // 16-byte chunks per output row
  static_assert(kChunks == 16 && (kBM / 2) * kOut <= kStageElems, "activation epilogue layout");
  const int h = lane >> 5;
  auto row_ptr = [&](int row) {
    return (__attribute__((address_space(3))) uint16_t*)(uintptr_t)(
               row < kBM / 2 ? lds_addr(&sm.a[eslot][0]) : lds_addr(&sm.b[eslot][0])) +
           (row & (kBM / 2 - 1)) * kOut;
  };
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
    for (int mb = 0; mb < kMB; ++mb) {
      const int row = wm0 + 32 * mb + (lane & 31);
      const int chunk = wn0 / 16 + 2 * nb + h;
      bf16x8 v;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float g = acc[nb][mb][i];
        const float u = acc[nb][mb][8 + i];
        v[i] = (__bf16)(g / (1.f + __expf(-g)) * u);
      }
      *(__attribute__((address_space(3))) bf16x8*)(row_ptr(row) + ((chunk ^ (row & 15)) << 3)) = v;
    }
  block_barrier();   // every wave's outputs are in the slot
  const int c0 = ti.n0 / 2, cvalid = ti.cols_valid / 2;
  for (int idx = threadIdx.x; idx < kBM * kChunks; idx += kThreads) {
    const int row = idx / kChunks, ch = idx % kChunks;
    const bf16x8 v =
        *(const __attribute__((address_space(3))) bf16x8*)(row_ptr(row) + ((ch ^ (row & 15)) << 3));
    if (row < ti.rows_valid && 8 * ch < cvalid)
      store16_nt(a.xout + (size_t)(ti.r0 + row) * a.I + c0 + 8 * ch, __builtin_bit_cast(u32x4, v));
  }
}

// Computes tile `ti` and stores it to Y.  The ring continues across tiles:
// stage kt of this tile sits in slot (base + kt) % kStages, and the next
// tile's stages follow this tile's last one.  Its ring fill was issued
// already if `filled`; with `next`, the next tile `nt` gets its stage 0
// from this tile's last stage boundary (the slot freed there, while this
// tile's last stage computes) and its stage 1 after this tile's Y stores
// (the slot of this tile's last stage, which carries the epilogue).
// tctx: on entry the tile's load addresses when it is `filled` (its caller
// made them for its ring fill), on return the next tile's.
template <class Args>
__device__ void compute_tile(Smem& sm, const Args& a, const TileInfo& ti, bool filled, bool next,
                             const TileInfo& nt, int base, u64* t_mid, TileCtx& tctx,
                             bool defer_stage1 = false) {
  // The lane's LDS offsets are recomputed for every tile (a few VALU
  // operations) rather than kept across the tile loop.
  const int lane = opaque_tid() & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nk = (gemm_k(a) + kBK - 1) / kBK;
  if constexpr (RowGather<Args>::on) {
    // the tile's gathered rows: staged by the previous tile when it loaded
    // this tile's first stage, else now
    if (!filled) {
      gather_commit(sm, a, gather_load(a, ti));
      block_barrier();
    }
  }
  if (!filled) tctx = make_ctx(sm, a, ti, wave);
  const TileCtx t = tctx;

  // per-lane LDS element offsets of the MFMA fragments (stage 0, step 0)
  const int wn0 = (wave % kWavesN) * kWN;
  const int wm0 = (wave / kWavesN) * kWM;
  int offA[kNB];
  {
    const int j = lane & 15;
    const int krow = 8 * (lane >> 5) + (j >> 2);
    const int u = j & 3;
    const int rg = (lane >> 4) & 1;
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) {
      const int col = wn0 + 32 * nb + 16 * rg + 8 * (u & 1) + 4 * (u >> 1);
      offA[nb] = krow * kBN + (((col >> 3) ^ (4 * (krow & 3))) << 3) + (col & 7);
    }
  }
  int offB[kKS];
  {
    const int m = wm0 + (lane & 31);
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) {
      const int c = 2 * ks + (lane >> 5);
      offB[ks] = m * kBK + ((c ^ ((m / kXRowsPerLine) % kXChunks)) << 3);
    }
  }

  // (the first K=16 step writes every accumulator from zero)
  f32x16 acc[kNB][kMB];

  // prologue: fill the ring (unless done during the previous tile's
  // publish), then wait for stage 0 (every wave's share)
  if (!filled) issue_prologue(a, t, nk, base, wave);
  wait_stage(min(kStages - 1, nk - 1));
  block_barrier();
  // gathering stages: the next tile's tokens load now and are staged at the
  // last stage boundary (after its wait, so waiting for them costs nothing)
  int next_tok = 0;
  if constexpr (RowGather<Args>::on) {
    if (next) next_tok = gather_load(a, nt);
  }

  // One flat pipeline over the K=16 steps: the fragments of step g+1 are
  // read while the MFMAs of step g run, also across stage boundaries.  The
  // stage boundary (stage kt+1 landed for every wave, every wave done
  // reading the slot of stage kt) is one barrier, after which that slot is
  // refilled with stage kt + kStages (of the next tile past the last one).
  bf16x8 af[2][kNB], bm[2][kMB];
  auto slot_of = [&](int kt) { return (base + kt) % kStages; };
  auto slot_a = [&](int kt) { return (lds_u16*)(uintptr_t)(t.lds_a + slot_of(kt) * kStageElems * 2); };
  auto slot_b = [&](int kt) { return (lds_u16*)(uintptr_t)(t.lds_b + slot_of(kt) * kStageElems * 2); };
  // Steps are grouped so that the loop starts at a stage boundary (which
  // waits for all LDS reads anyway) and every MFMA group follows the reads
  // of the next step in straight-line code: the compiler's LDS waits before
  // each group then cover only that group's own fragments.
  load_frags(slot_a(0), slot_b(0), offA, offB, 0, af[0], bm[0]);
#pragma unroll
  for (int ks = 0; ks + 1 < kKS; ++ks) {
    load_frags(slot_a(0), slot_b(0), offA, offB, ks + 1, af[(ks + 1) & 1], bm[(ks + 1) & 1]);
    __builtin_amdgcn_sched_barrier(0);   // keep the next step's reads ahead of these MFMAs
    if (ks == 0)
      mfma_step_zero(acc, af[0], bm[0]);
    else
      mfma_step(acc, af[ks & 1], bm[ks & 1]);
  }
  static_assert(kLoadsPerOperand % kNB == 0 && kLoadsPerOperand / kNB <= kKS, "load spread");
  static_assert(kStages == 2, "the boundary loop refills one stage ahead");
  // boundaries whose freed slot takes a stage of this tile
  for (int kt = 0; kt + kStages < nk; ++kt) {
    wait_stage(kStages - 2);
    block_barrier();
    boundary_steps(acc, af, bm, a, slot_a(kt + 1), slot_b(kt + 1), offA, offB, t, kt + kStages,
                   slot_of(kt), wave, true);
  }
  // The next tile's load addresses (nt is a valid tile, == ti, without a
  // next one), made once for its stage 0 and 1 here and kept for it; a
  // gathering stage makes them after the next tile's rows are staged.
  // The last boundary: its freed slot takes the next tile's stage 0.
  if (nk >= 2) {
    wait_stage(0);
    if constexpr (RowGather<Args>::on) {
      if (next) gather_commit(sm, a, next_tok);   // this tile's rows are in t already
    }
    block_barrier();
    tctx = make_ctx(sm, a, nt, wave);
    boundary_steps(acc, af, bm, a, slot_a(nk - 1), slot_b(nk - 1), offA, offB, tctx, 0,
                   slot_of(nk), wave, next);
  }
  mfma_step(acc, af[(kKS - 1) & 1], bm[(kKS - 1) & 1]);
  if constexpr (RowGather<Args>::on) {
    if (next && nk == 1) gather_commit(sm, a, next_tok);
  }
  // every wave is done with the slot of the last stage, which carries the
  // epilogue
  block_barrier();
  t_mid[0] = now_100mhz();
  const int eslot = slot_of(nk - 1);
  // with a single stage there was no boundary: the next tile's stage 0 goes
  // into the other slot now, ahead of the Y stores
  if (nk == 1) tctx = make_ctx(sm, a, nt, wave);
  if (next && nk == 1) issue_stage(a, tctx, 0, slot_of(nk), wave);

  // The down-projection's epilogue uses only the x part of the slot, so the
  // W2 half of the next tile's stage 1 loads during it.
  constexpr bool kEarlyB = !RowGather<Args>::on;
  // (Also before a split's publish: those loads are older than the Y
  // stores, so the publish's wait for the stores covers them at no cost.)
  const bool stage1_now = next && nk >= 2 && !defer_stage1;
  if (kEarlyB && next && nk >= 2) issue_stage_b(a, tctx, 1, eslot, wave);
  epilogue_store(sm, a, acc, eslot, lane, wave, wn0, wm0, ti);
  if (stage1_now) {
    // every wave has read its block back (its stores carry the data), so
    // the slot may take the rest of the next tile's stage 1
    block_barrier();
    if (kEarlyB)
      issue_stage_a(a, tctx, 1, eslot, wave);
    else
      issue_stage(a, tctx, 1, eslot, wave);
  }
  t_mid[1] = now_100mhz();
}

// The x half of the next tile's stage 1 into its slot, when the tile
// before deferred it past its split's publish (after every wave has read
// its epilogue block back); the W2 half went in before the epilogue.
__device__ __forceinline__ void issue_stage1_a(const KArgs& a, const TileCtx& tn, int base) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  issue_stage_a(a, tn, 1, (base + 1) % kStages, wave);
}

// ---- consumer role: one task --------------------------------------------------
__device__ __forceinline__ float bf16lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

// Metadata of one consumer task, staged in LDS (over the idle operand ring):
// per token of the task, its row count and its rows and gate weights sorted
// by row.  One pass for all tokens turns the dependent chain count/inverse
// map -> gate into two dependent loads per task instead of per token pair.
struct TaskMeta {
  int n[kCommTM];
  int row[kCommTM * kMaxTopk];
  float gate[kCommTM * kMaxTopk];
  int unsorted[kCommTM * kMaxTopk];   // the rows in inverse-map order, while they are ranked
};

static_assert(sizeof(TaskMeta) <= sizeof(Smem::a) + sizeof(Smem::b) &&
                  offsetof(Smem, b) == offsetof(Smem, a) + sizeof(Smem::a),
              "task metadata overlays the operand ring");
__device__ TaskMeta& task_meta(Smem& sm) { return *reinterpret_cast<TaskMeta*>(&sm.a[0][0]); }

__device__ void load_task_meta(Smem& sm, TaskMeta& m, const KArgs& a, u64 cnt_epoch, int t0,
                               int ntok) {
  const int K = a.topk;
  const bool bands = a.mode == 2;
  if (bands) {
    if (threadIdx.x == 0) sm.task_band = 0;
    __syncthreads();
  }
  // One thread per (token, slot): the token's count and the slot's inverse-
  // map entry in one round trip (the entry is in bounds; past the count it
  // is stale and ignored), then the row's gate in a second.  The rows of a
  // token are distinct, so each takes the position of its rank among them
  // (ascending row order), counted over the unsorted copy in LDS.
  for (int i = opaque_tid(); i < ntok * K; i += kThreads) {
    const int t = i / K;
    const int j = i - t * K;
    const u64 cv = ld_relaxed(&a.tok_cnt[t0 + t]);
    const int r = a.inv[(long long)(t0 + t) * K + j];
    const uint32_t have = epoch_count(cv, cnt_epoch);
    const int n = (int)(have < (uint32_t)K ? have : (uint32_t)K);
    m.unsorted[i] = j < n ? r : 0;
    if (j == 0) m.n[t] = n;
  }
  __syncthreads();
  for (int i = opaque_tid(); i < ntok * K; i += kThreads) {
    const int t = i / K;
    const int j = i - t * K;
    const int n = m.n[t];
    if (j < n) {
      const int r = m.unsorted[i];
      const float g = a.gate_w[r];
      int rank = 0;
      for (int q = 0; q < n; ++q) rank += m.unsorted[t * K + q] < r;
      m.row[t * K + rank] = r;
      m.gate[t * K + rank] = g;
      if (bands) atomicMax(&sm.task_band, band_of_row(sm, a, r));
    } else {
      m.row[i] = 0;
      m.gate[i] = 0.f;
    }
  }
  __syncthreads();
}

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
constexpr int kColBlocks = kCommTN / 256;   // 256-column blocks of a task, 4 columns per lane
static_assert(kCommTN % 256 == 0, "task columns");

__device__ __forceinline__ void fma4(float (&acc)[4], float g, const u32x2& v) {
  acc[0] = fmaf(g, bf16lo(v[0]), acc[0]);
  acc[1] = fmaf(g, bf16hi(v[0]), acc[1]);
  acc[2] = fmaf(g, bf16lo(v[1]), acc[2]);
  acc[3] = fmaf(g, bf16hi(v[1]), acc[3]);
}

// Rows j0 .. j0+U-1 of two tokens at every column block: all loads first
// (a padding row j >= n re-reads row n-1 and gets weight 0), then the FMAs
// in ascending row order.  n >= 1 for both tokens; every row read is one
// this launch has written, so its values are finite and weight 0 adds 0.
template <int U>
__device__ __forceinline__ void gather_step(const KArgs& a, int j0, const int (&rs)[2],
                                            const int (&gs)[2], const int (&n)[2],
                                            const int (&col)[kColBlocks], int ydelta,
                                            float (&acc)[2][kColBlocks][4]) {
  u32x2 v[2][U][kColBlocks];
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u < n[p] ? j0 + u : n[p] - 1;
      const uint16_t* yr =
          a.Y + (size_t)__builtin_amdgcn_readlane(rs[p], j) * a.ypitch + ydelta;
#pragma unroll
      for (int b = 0; b < kColBlocks; ++b)
        v[p][u][b] = __builtin_nontemporal_load((const u32x2*)(yr + col[b]));
    }
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u;
      const float gj = j < n[p] ? __int_as_float(__builtin_amdgcn_readlane(gs[p], j)) : 0.f;
#pragma unroll
      for (int b = 0; b < kColBlocks; ++b) fma4(acc[p][b], gj, v[p][u][b]);
    }
}

// out[t, col0 : col0+ncols] for the tokens [t0, t0+ntok) whose metadata is in
// m: wave w takes the token pairs w, w+nwaves, ...; lane l owns columns
// 256b + 4l .. 256b + 4l + 3 of every block b, so each output store of a
// wave writes 1 KB of one row contiguously (whole cache lines).
// ydelta: Y column minus output column for the task's columns (its split's
// segment of a Y row starts on a line).
__device__ void consume_task(const KArgs& a, const TaskMeta& m, int t0, int ntok, int col0,
                             int ncols, int ydelta) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  int col[kColBlocks];
  bool cok[kColBlocks];
#pragma unroll
  for (int b = 0; b < kColBlocks; ++b) {
    const int c = 256 * b + 4 * lane;
    cok[b] = c < ncols;
    col[b] = col0 + (cok[b] ? c : 0);   // in-range address; the store is skipped
  }
  for (int pp = 2 * wave; pp < ntok; pp += 2 * nwaves) {
    int rs[2], gs[2], n[2], t[2];
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      t[p] = t0 + pp + p;
      n[p] = 0;
      rs[p] = 0;
      gs[p] = 0;
      if (pp + p < ntok) {
        const int q = pp + p;
        n[p] = m.n[q];
        if (lane < n[p]) {
          rs[p] = m.row[q * a.topk + lane];
          gs[p] = __float_as_int(m.gate[q * a.topk + lane]);
        }
      }
    }
    float acc[2][kColBlocks][4];
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int b = 0; b < kColBlocks; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[p][b][i] = 0.f;
    // A token without rows borrows the other token's row list for its
    // loads, with all weights zero, so both tokens share one load stream.
    const int nl[2] = {n[0] > 0 ? n[0] : n[1], n[1] > 0 ? n[1] : n[0]};
    const int rl[2] = {n[0] > 0 ? rs[0] : rs[1], n[1] > 0 ? rs[1] : rs[0]};
    const int gl[2] = {n[0] > 0 ? gs[0] : 0, n[1] > 0 ? gs[1] : 0};
    const int nmax = nl[0] > nl[1] ? nl[0] : nl[1];
    for (int j0 = 0; j0 < nmax; j0 += 8) {
      const int left = nmax - j0;
      if (left <= 2)
        gather_step<2>(a, j0, rl, gl, nl, col, ydelta, acc);
      else if (left <= 4)
        gather_step<4>(a, j0, rl, gl, nl, col, ydelta, acc);
      else if (left <= 6)
        gather_step<6>(a, j0, rl, gl, nl, col, ydelta, acc);
      else
        gather_step<8>(a, j0, rl, gl, nl, col, ydelta, acc);
    }
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      if (pp + p >= ntok) continue;
      float* o = a.out + (size_t)t[p] * a.H;
#pragma unroll
      for (int b = 0; b < kColBlocks; ++b) {
        if (!cok[b]) continue;
        const f32x4 v = {acc[p][b][0], acc[p][b][1], acc[p][b][2], acc[p][b][3]};
        __builtin_nontemporal_store(v, (f32x4*)(o + col[b]));
      }
    }
  }
}

// ---- consumer role, atomic scatter: one compute tile ---------------------------
// fp32 add at agent scope, as the hardware's no-return atomic instruction
// (the output is ordinary device memory of this process, not fine-grained
// or peer memory, so no compare-and-swap loop is needed).
__device__ __forceinline__ void atomic_add_f32(float* p, float v) {
  (void)__builtin_amdgcn_global_atomic_fadd_f32((__attribute__((address_space(1))) float*)p, v);
}

// out[token_ids[r], n0 + c] += gate_w[r] * Y[r, n0 + c] for every row r and
// column c of tile ti.  Wave w takes rows w*U .. w*U+U-1, then the next
// kWaves*U rows; lane l takes columns l, l+64, l+128, l+192, so every load
// and every atomic instruction of a wave covers one contiguous run of its
// row.  Rows whose token id is out of range are skipped (and flagged).
__device__ void scatter_tile(const KArgs& a, const TileInfo& ti) {
  constexpr int U = 4;
  constexpr int kCols = kBN / 64;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  bool bad = false;
  for (int m0 = wave * U; m0 < ti.rows_valid; m0 += kWaves * U) {
    int tok[U];
    float g[U];
    uint16_t y[U][kCols];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int m = m0 + u < ti.rows_valid ? m0 + u : ti.rows_valid - 1;
      const long long r = (long long)ti.r0 + m;
      tok[u] = a.token_ids[r];
      g[u] = m0 + u < ti.rows_valid ? a.gate_w[r] : 0.f;
      const uint16_t* yr = a.Y + r * a.ypitch + ti.ny0;
#pragma unroll
      for (int i = 0; i < kCols; ++i) {
        const int c = lane + 64 * i;
        y[u][i] = __builtin_nontemporal_load(yr + (c < ti.cols_valid ? c : 0));
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (m0 + u >= ti.rows_valid) continue;
      if (tok[u] < 0 || tok[u] >= a.T) {
        bad = true;
        continue;
      }
      float* o = a.out + (long long)tok[u] * a.H + ti.n0;
#pragma unroll
      for (int i = 0; i < kCols; ++i) {
        const int c = lane + 64 * i;
        if (c < ti.cols_valid) atomic_add_f32(o + c, g[u] * __uint_as_float((uint32_t)y[u][i] << 16));
      }
    }
  }
  if (bad && lane == 0)
    __hip_atomic_fetch_or(a.status, kStBadRouting, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// What a workgroup knows while it serves consumer tasks.
struct Consumer {
  int ready;     // splits [0, ready] were acquired by this workgroup (token bands:
                 // the tiles [0, ready) are known published)
  int split;     // the first split that may still have unclaimed tasks
  int meta_t0;   // first token of the block whose metadata is in LDS (-1: none)
  int meta_n;    // ... and its token count
  bool inv_ok;   // every workgroup's inverse-map share is published
  bool inv_acq;  // ... and acquired by this workgroup
  int tiles;     // atomic scatter: the tiles [0, tiles) of the global sequence are
                 // known published and acquired by this workgroup
};

// Owner-write tasks of split s: their token count and how many there are
// (column splits cut the last split's token blocks finer).
__device__ __forceinline__ int task_tm(const KArgs& a, int s) {
  return a.mode == 0 && s == a.L - 1 ? a.comm_tm_last : a.comm_tm;
}
__device__ __forceinline__ int split_tasks(const KArgs& a, int s) {
  return a.mode == 0 && s == a.L - 1 ? a.tasks_last : a.tasks_per_split;
}

// The owner-write task idx's metadata in LDS (unless it is there already:
// a block's metadata also serves any block that starts at the same token
// and has no more tokens).
__device__ void ensure_task_meta(Smem& sm, const KArgs& a, int tm, int idx, Consumer& cs) {
  const int t0 = (idx / a.cb_per_split) * tm;
  const int ntok = min(tm, a.T - t0);
  if (t0 != cs.meta_t0 || ntok > cs.meta_n) {
    __syncthreads();   // every wave is done with the previous task's metadata
    load_task_meta(sm, task_meta(sm), a, count_epoch(sm), t0, ntok);
    cs.meta_t0 = t0;
    cs.meta_n = ntok;
  }
}

// Task idx of split s (owner-write: token block idx / cb_per_split, column
// block idx % cb_per_split; atomic scatter: compute tile idx of the split).
__device__ void run_task(Smem& sm, const KArgs& a, int W_comp, int tps, int s, int idx,
                         Consumer& cs, u64 t_wait, u64 t_go) {
  if (a.mode == 1) {
    scatter_tile(a, decode_tile(sm, a, W_comp, s * W_comp + idx));
  } else {
    const int tm = task_tm(a, s);
    const int tb = idx / a.cb_per_split;
    const int cb = idx - tb * a.cb_per_split;
    const int t0 = tb * tm;
    const int ntok = min(tm, a.T - t0);
    const int col0 = s * a.nsplit + cb * a.comm_tn;
    const int ncols = min(a.comm_tn, (s + 1) * a.nsplit - col0);
    ensure_task_meta(sm, a, tm, idx, cs);
    consume_task(a, task_meta(sm), t0, ntok, col0, ncols, s * (a.ysplit - a.nsplit));
  }
  if (a.trace) {
    __syncthreads();
    if (threadIdx.x == 0) {
      u64* rec = a.trace + 4 * a.max_tiles + 4 * ((long long)s * tps + idx);
      rec[0] = t_wait;
      rec[1] = t_go;
      rec[2] = now_100mhz();
      rec[3] = blockIdx.x;
    }
  }
}

// Serves consumer tasks until none is left.  Each split has its own task
// counter and its tasks are claimed in order, split 0 first, so whichever
// workgroup is free takes the next one: consumers that finish early, or
// compute workgroups with fewer tiles, absorb more of the earlier splits'
// work.
__device__ void consumer_loop(Smem& sm, const KArgs& a, int W_comp, Consumer& cs) {
  // overlapping expert ranges (bad offsets, flagged) may need more tiles
  // than the flag array holds; the compute workgroups then stop at once
  if ((long long)W_comp * a.L > a.max_tiles) return;
  // An acquire invalidates this XCD's L2 (also under the compute workgroups
  // still running there), so there is one per split: the inverse map's
  // flags are acquired together with the first split's, before any read.
  if (!cs.inv_ok) {
    // (acquired here when the split's own acquire would come too late for
    // the metadata: no tiles, or a single split, whose inverse map is
    // published at the start)
    const bool acq = W_comp == 0 || a.L == 1;
    if (!wait_flags(sm, a.wg_flags, gridDim.x, a, acq)) return;
    cs.inv_ok = true;
    cs.inv_acq = acq;
  }
  // owner-write: tasks of comm_tm tokens x comm_tn columns; atomic scatter:
  // one task per compute tile
  // (trace records: split s's tasks start at s tps, only the last split's
  // count differs)
  const int tps = a.mode == 1 ? (int)W_comp : a.tasks_per_split;
  // owner-write: a split is ready once every compute workgroup has flagged
  // it (P flags, one per workgroup, instead of one per tile)
  const bool by_wg = a.mode == 0;
  for (; cs.split < a.L; ++cs.split) {
    const int s = cs.split;
    uint32_t* sflags = a.split_flags + (long long)s * kMaxGrid;
    const int ntask = a.mode == 1 ? (int)W_comp : split_tasks(a, s);
    while (true) {
      const u64 t_wait = now_100mhz();
      if (threadIdx.x < 64) {
        // the claim, and the first look at the split's flags, in one round trip
        uint32_t claimed = 0;
        if (threadIdx.x == 0)
          claimed = __hip_atomic_fetch_add(&a.task_ctr[s], 1u, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
        const bool look = by_wg && s > cs.ready && a.P <= kPollSpan;
        const int first = look ? first_unpublished(sflags, 0, a.P, flag_epoch(sm), threadIdx.x) : 0;
        if (threadIdx.x == 0) {
          sm.task = (int)min(claimed, (uint32_t)ntask);
          sm.split_seen = look && first == kPollSpan;
        }
      }
      __syncthreads();
      const int idx = sm.task;
      const bool seen = sm.split_seen != 0;
      __syncthreads();   // sm.task is rewritten by the next claim
      if (idx >= ntask) break;
      if (a.mode == 1) {
        // a scatter task needs only its own tile: it waits for the published
        // prefix of the tile sequence up to that tile (tiles are claimed in
        // sequence order, so this is the compute wave that holds it), and
        // takes what is published beyond it as well, one acquire for all
        const long long g = (long long)s * W_comp + idx;
        if (g >= cs.tiles) {
          const long long end = wait_prefix(sm, a.tile_flags, cs.tiles, g + 1,
                                            (long long)W_comp * a.L, a);
          if (end < 0) return;
          cs.tiles = (int)end;
          cs.inv_acq = true;   // that acquire covered the zeroed output as well
        }
      } else if (s > cs.ready) {
        // a task's metadata needs the inverse map only: once that is
        // acquired, it loads while the task's split is still computing
        if (cs.inv_acq && !seen) ensure_task_meta(sm, a, task_tm(a, s), idx, cs);
        if (seen) {
          acquire_workgroup();
        } else if (W_comp > 0) {
          const bool ok = by_wg ? wait_flags(sm, sflags, a.P, a)
                                : wait_flags(sm, a.tile_flags + (long long)s * W_comp, W_comp, a);
          if (!ok) return;
        }
        cs.ready = s;
        cs.inv_acq = true;   // that acquire covered the inverse map as well
      }
      run_task(sm, a, W_comp, tps, s, idx, cs, t_wait, now_100mhz());
    }
  }
}

// Token bands (mode 2): one task counter over all tasks (token block major,
// then column block of the full width).  A task waits until every tile of
// the bands up to the last one holding its rows is published: the flags of
// the band sequence's prefix [0, band_start[b+1]), polled incrementally,
// with one acquire per newly published prefix (and one for the inverse map,
// which a task's band requirement is computed from).
__device__ void consumer_loop_bands(Smem& sm, const KArgs& a, Consumer& cs) {
  const int total = sm.band_start[a.L];
  if (total > a.max_tiles) return;
  if (!cs.inv_ok) {
    if (!wait_flags(sm, a.wg_flags, gridDim.x, a)) return;
    cs.inv_ok = true;
  }
  const int ntasks = a.tasks_per_split;
  while (true) {
    const u64 t_wait = now_100mhz();
    if (threadIdx.x == 0)
      sm.task = (int)min(__hip_atomic_fetch_add(&a.task_ctr[0], 1u, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT),
                         (uint32_t)ntasks);
    __syncthreads();
    const int idx = sm.task;
    __syncthreads();   // sm.task is rewritten by the next claim
    if (idx >= ntasks) break;
    const int tb = idx / a.cb_per_split;
    const int cb = idx - tb * a.cb_per_split;
    const int t0 = tb * a.comm_tm;
    const int ntok = min(a.comm_tm, a.T - t0);
    const int col0 = cb * a.comm_tn;
    const int ncols = min(a.comm_tn, a.H - col0);
    ensure_task_meta(sm, a, a.comm_tm, idx, cs);
    const int need = sm.band_start[min(sm.task_band, a.L - 1) + 1];
    if (need > cs.ready) {   // cs.ready: tiles [0, ready) are published and acquired
      if (!wait_flags(sm, a.tile_flags + cs.ready, need - cs.ready, a)) return;
      cs.ready = need;
    }
    const u64 t_go = now_100mhz();
    consume_task(a, task_meta(sm), t0, ntok, col0, ncols, 0);
    if (a.trace) {
      __syncthreads();
      if (threadIdx.x == 0) {
        u64* rec = a.trace + 4 * a.max_tiles + 4 * (long long)idx;
        rec[0] = t_wait;
        rec[1] = t_go;
        rec[2] = now_100mhz();
        rec[3] = blockIdx.x;
      }
    }
  }
}

// Compute index of workgroup b >= C such that consecutive indices share an
// XCD (workgroups are dispatched to the 8 XCDs round-robin by id), keeping a
// wave's neighbouring tiles, which share x rows and W2 columns, in one L2.
__device__ __forceinline__ int compute_index(int b, int C, int N) {
  auto below = [](int n, int x) { return n > x ? (n - x + 7) >> 3 : 0; };
  const int xcd = b & 7;
  int c = 0;
  for (int x = 0; x < xcd; ++x) c += below(N, x) - below(C, x);
  return c + below(b, xcd) - below(C, xcd);
}

__device__ __forceinline__ void fused_body(Smem& sm, const KArgs& a) {
  if (threadIdx.x == 0) {
    sm.epoch = launch_epoch(a);   // load_experts synchronises
    __hip_atomic_fetch_add(a.start_ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  load_experts(sm, a);
  const bool bands = a.mode == 2;
  if (bands) load_bands(sm, a);
  const long long rows_dev = a.E > 0 ? (long long)sm.start[a.E - 1] + sm.count[a.E - 1] : 0;
  const int m_tiles = sm.tile_prefix[a.E];
  const int W_comp = m_tiles * a.ntps;   // tiles per split (column splits)
  const int b = blockIdx.x;
  const int c = b < a.C ? 0 : compute_index(b, a.C, (int)gridDim.x);
  const int total = bands ? sm.band_start[a.L] : W_comp * a.L;
  const int first_split_end = bands ? sm.band_start[1] : W_comp;
  auto split_of = [&](int g) { return bands ? band_of_tile(sm, a, g) : g / W_comp; };
  // Round k of the sequence is tiles [k P, (k+1) P).  Compute workgroup c
  // takes tile k P + c of every round (XCD-aware: the workgroups of
  // consecutive c share an XCD, and so do their tiles).  The ntps workgroups
  // on the n-tiles of one m-tile share its x rows; with P a multiple of
  // ntps the same workgroups meet again in every round and request the same
  // lines at the same moment.  Launches of at least kRotMinRounds rounds
  // then give workgroup c tile k P + (c + k) mod P, which moves the m-tile
  // boundaries by one workgroup each round, so the partners change.  (On
  // shorter launches the fixed partners measured as fast or faster.)
  const int rounds = (total + a.P - 1) / a.P;
  const bool rot = rounds >= kRotMinRounds && a.P % a.ntps == 0;
  auto tile_of = [&](int k) { return k * a.P + (rot ? (c + k) % a.P : c); };
  const int g_first = b >= a.C && c < total ? c : -1;
  // A compute workgroup with a tile in split 0 publishes its share of the
  // inverse map with that split (consumers read it only after a split).
  // With a single split that publish comes only at the end of the tiles, so
  // the share is published at once instead: the consumers then stage their
  // first task's metadata while the split is still computing.
  const bool defer_inverse =
      a.L > 1 && g_first >= 0 && g_first < first_split_end && total <= a.max_tiles;
  auto decode = [&](int g) {
    return bands ? decode_band_tile(sm, a, g) : decode_tile(sm, a, W_comp, g);
  };
  const int nk = (a.I + kBK - 1) / kBK;
  // A compute workgroup issues its first tile's ring fill before building
  // its share of the inverse map, so those loads fly during its atomics.
  TileInfo cur = {0, 0, 0, 0, 0};
  TileCtx tctx;   // the load addresses of the tile whose ring stages are in flight
  bool filled = false;
  if (total <= a.max_tiles && g_first >= 0) {
    cur = decode(g_first);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    tctx = make_ctx(sm, a, cur, wave);
    issue_prologue(a, tctx, nk, 0, wave);
    filled = true;
  }
  consumer_prologue(sm, a, rows_dev, !defer_inverse);

  if (b >= a.C) {   // compute role
    if (total > a.max_tiles) {  // cannot happen with sanitized offsets; stay in bounds
      if (threadIdx.x == 0)
        __hip_atomic_fetch_or(a.status, kStBadRouting, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return;
    }
    int split_first = 0;   // round of this workgroup's first tile of the current split
    int base = 0;                // ring slot of the current tile's stage 0
    // Column splits: this workgroup's flag of split s (its compute index c)
    // says that it has published all its tiles of s, or has none there; the
    // owner-write consumers wait for a split's P flags.  Thread 0 stores
    // them, in split order: splits before the first tile (none of its tiles
    // there) now, the others with each split's publish.
    int flagged = 0;   // (thread 0) splits [0, flagged) flagged
    auto flag_splits = [&](int upto) {
      for (; flagged < upto; ++flagged)
        __hip_atomic_store(&a.split_flags[(long long)flagged * kMaxGrid + c], flag_epoch(sm),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };
    if (!bands && threadIdx.x == 0) flag_splits(g_first >= 0 ? g_first / W_comp : a.L);
    // the inverse-map stores are done before the tile loop (once), so that
    // the compiler has nothing in flight to wait for inside it
    waitcnt_vm<0>();
    for (int g = g_first, k = 0; g >= 0; ++k) {
      const int g_next = tile_of(k + 1) < total ? tile_of(k + 1) : -1;
      const bool next = g_next >= 0;
      const TileInfo nt = next ? decode(g_next) : cur;
      const u64 t_start = now_100mhz();
      u64 t_mid[2];
      const bool last_of_split = !next || split_of(g_next) != split_of(g);
      // A split's last tile holds the x half of its next tile's stage 1
      // back until the publish, so that the publish's waits cover nothing
      // issued after the Y stores.
      compute_tile(sm, a, cur, filled, next, nt, base, t_mid, tctx, last_of_split);
      base = (base + nk) % kStages;   // the next tile's stages follow this tile's
      // Publish once per split: consumers wait for whole splits, so the tiles
      // of a split are published together after this workgroup's last tile of
      // it (an agent-scope release writes back the whole L2; once per tile it
      // cost ~3.6 us per tile).  Every wave waits until its Y stores are
      // acknowledged by the L2 (vmcnt counts in issue order, so only the next
      // tile's stage 1, issued after them, may stay in flight), the barrier
      // orders those waits before thread 0, whose release fence writes back
      // the L2 before it stores the flags.
      if (last_of_split) {
        // only the next tile's stage 0 and stage-1 W2 half (older) and the
        // Y stores are in flight
        waitcnt_vm<0>();
        if (a.delay_ticks > 0 && threadIdx.x == 0 && c % a.delay_mod == 0) {
          // debug: hold this publish back for a bounded time, so that
          // consumers reach the split's flags long before they are set
          const u64 until = now_100mhz() + (u64)a.delay_ticks;
          while (now_100mhz() < until) __builtin_amdgcn_s_sleep(16);
        }
        __syncthreads();
        if (threadIdx.x == 0) {
          release_agent();
          const uint32_t epoch = flag_epoch(sm);
          for (int kk = split_first; kk <= k; ++kk)
            __hip_atomic_store(&a.tile_flags[tile_of(kk)], epoch, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
          // this workgroup is done with every split before its next tile's
          if (!bands) flag_splits(next ? g_next / W_comp : a.L);
          if (defer_inverse && split_first == 0)   // first publish: also the inverse map
            __hip_atomic_store(&a.wg_flags[blockIdx.x], epoch, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        }
        // nothing the compiler tracks stays in flight past the publish: else
        // it would wait for it (and, in order, for the ring loads issued
        // since) at the next tile's start, on every tile
        waitcnt_vm<0>();
        split_first = k + 1;
        if (next && nk >= 2) issue_stage1_a(a, tctx, base);
      }
      if (a.trace && threadIdx.x == 0) {
        store8(&a.trace[4 * g + 0], t_start);
        store8(&a.trace[4 * g + 1], t_mid[0]);
        store8(&a.trace[4 * g + 2], t_mid[1]);
        store8(&a.trace[4 * g + 3], now_100mhz());
      }
      cur = nt;
      filled = next;
      g = g_next;
    }
    // after its tiles, a compute workgroup serves consumer tasks only with
    // C = 0 (the role switch), and only if every workgroup of the grid has
    // started: the tasks wait on tiles of other workgroups, and waiting on
    // one that has not started yet could hold a CU it needs (another launch
    // may share the GPU).  Workgroups started later serve the tasks instead;
    // the last one to start always sees the whole grid started.
    if (!a.drain) return;
    if (threadIdx.x == 0)
      sm.flag = __hip_atomic_load(a.start_ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >=
                gridDim.x;
    __syncthreads();
    const bool all_started = sm.flag != 0;
    __syncthreads();   // sm.flag is rewritten by the consumers' waits
    if (!all_started) return;
  }
  // consumers, and role-switch workgroups after their tiles (one call site,
  // so that the loop is inlined)
  if (bands) {
    Consumer cs = {0, 0, -1, 0, false, false};
    consumer_loop_bands(sm, a, cs);
  } else {
    Consumer cs = {-1, 0, -1, 0, false, false};
    consumer_loop(sm, a, W_comp, cs);
  }
}

__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
moe_gemm2_fused(KArgs a) {
  __shared__ Smem sm;
  fused_body(sm, a);
  // The last workgroup to finish advances the workspace's launch epoch (and
  // rearms the counter) for the next launch on this workspace.
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t done = __hip_atomic_fetch_add(a.done_ctr, 1u, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT);
    if (done == gridDim.x - 1) {
      u64 e = sm.epoch;
      if ((uint32_t)(e + 1) == 0) ++e;   // the next launch's flags must not be 0
      __hip_atomic_store(a.done_ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.start_ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.epoch_word, e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// ---- the up-projection stage: grouped GEMM1 + SwiGLU -----------------------------
// Every workgroup computes: tiles expert -> m-tile -> n-tile of the packed
// 2I columns, workgroup c (XCD-aware index) taking tiles c, c+P, ...
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
moe_gemm1_swiglu_kernel(G1Args a) {
  __shared__ Smem sm;
  load_experts(sm, a);
  const int m_tiles = sm.tile_prefix[a.E];
  const int total = m_tiles * a.ntps;
  const int P = (int)gridDim.x;
  const int c = compute_index((int)blockIdx.x, 0, P);
  if (c >= total) return;
  const int nk = (a.H + kBK - 1) / kBK;
  bool filled = false;
  TileCtx tctx;
  int base = 0;
  for (int g = c; g < total; g += P) {
    const bool next = g + P < total;
    const TileInfo cur = decode_tile(sm, a, total, g);
    const TileInfo nt = decode_tile(sm, a, total, next ? g + P : g);
    u64 t_mid[2];
    compute_tile(sm, a, cur, filled, next, nt, base, t_mid, tctx);
    base = (base + nk) % kStages;
    filled = next;
  }
}

// W1 from [E, H, 2I] (gate columns 0..I-1, up columns I..2I-1) to the
// packed layout: column 32b + j holds gate column 16b + j and column
// 32b + 16 + j up column 16b + j (j < 16).
__global__ void pack_w1_kernel(const uint16_t* src, uint16_t* dst, long long n, int I) {
  const int N = 2 * I;
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < n;
       idx += (long long)gridDim.x * blockDim.x) {
    const long long row = idx / N;
    const int p = (int)(idx - row * N);
    const int b = p >> 5, j = p & 31;
    const int col = j < 16 ? 16 * b + j : I + 16 * b + (j - 16);
    dst[idx] = src[row * N + col];
  }
}

// Zeroes n words at p, except the 64-bit word at word index epoch_at (when
// epoch_at + 1 < n), which takes `epoch`.
__global__ void fill_zero_kernel(uint32_t* p, size_t n, size_t epoch_at, u64 epoch) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = i == epoch_at ? (uint32_t)epoch : i == epoch_at + 1 ? (uint32_t)(epoch >> 32) : 0u;
}

// ---- host side -----------------------------------------------------------------

struct Layout {
  size_t status, wg_flags, split_flags, flags, tok_cnt, inv, Y, total;
  long long rows, max_tiles;
  int nsplit, ntps, comm_tm, comm_tn, cb_per_split, tasks_per_split, comm_tm_last, tasks_last;
};

inline size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Tokens of the last split's owner-write tasks for tasks of comm_tm tokens.
// The last split's task: a quarter of the others' tokens, at least
// kCommTMMin (and never more than the others').
inline int last_split_tm(int comm_tm) {
  const int q = comm_tm / 4 > kCommTMMin ? comm_tm / 4 : kCommTMMin;
  return q < comm_tm ? q : comm_tm;
}

int check_shape(const moe_workload_t* wl) {
  if (!wl) return MOE_ERR_INVALID_ARG;
  if (wl->T < 0 || wl->H <= 0 || wl->I <= 0 || wl->E <= 0 || wl->topk <= 0 ||
      wl->splits <= 0 || wl->rows < 0)
    return MOE_ERR_INVALID_ARG;
  if (wl->E > kMaxE || wl->topk > kMaxTopk || wl->splits > kMaxSplits) return MOE_ERR_UNSUPPORTED;
  // (column splits also need H % (8 splits) == 0, checked per launch mode)
  if (wl->I % 8 != 0 || wl->H % 8 != 0) return MOE_ERR_UNSUPPORTED;
  // an expert's W2 slice is addressed with 32-bit byte offsets
  if ((long long)wl->I * wl->H * 2 > 0x7fffffffLL) return MOE_ERR_UNSUPPORTED;
  const long long rows = wl->rows > 0 ? wl->rows : (long long)wl->T * wl->topk;
  if (rows > (long long)INT32_MAX || (long long)wl->T * wl->topk > (long long)INT32_MAX)
    return MOE_ERR_UNSUPPORTED;
  // tile indices are 32-bit on the device, also for the most tiles that
  // bad offsets (every expert spanning all rows) could make
  const long long ntps = ((wl->H + wl->splits - 1) / wl->splits + kBN - 1) / kBN;
  if ((long long)wl->E * ((rows + kBM - 1) / kBM + 1) * ntps * wl->splits > (long long)INT32_MAX / 2)
    return MOE_ERR_UNSUPPORTED;
  return MOE_OK;
}

bool make_layout(const moe_workload_t* wl, Layout* L) {
  if (check_shape(wl) != MOE_OK) return false;
  L->rows = wl->rows > 0 ? wl->rows : (long long)wl->T * wl->topk;
  L->nsplit = (wl->H + wl->splits - 1) / wl->splits;   // ceil: sizes also cover token bands
  L->ntps = (L->nsplit + kBN - 1) / kBN;
  L->comm_tn = L->nsplit < kCommTN ? L->nsplit : kCommTN;
  L->cb_per_split = (L->nsplit + L->comm_tn - 1) / L->comm_tn;
  // Owner-write tasks of kCommTM tokens, halved (down to kCommTMMin) while
  // the launch would have fewer than kTaskTarget of them: a small batch's
  // combine then still spreads over every CU, and the last tasks of the
  // launch are short.
  L->comm_tm = kCommTM;
  while (L->comm_tm > kCommTMMin &&
         (long long)wl->splits * ((wl->T + L->comm_tm - 1) / L->comm_tm) * L->cb_per_split <
             kTaskTarget)
    L->comm_tm /= 2;
  L->tasks_per_split = ((wl->T + L->comm_tm - 1) / L->comm_tm) * L->cb_per_split;
  // The last split's tasks take a quarter of the tokens (down to
  // kCommTMMin): they start only after the last tiles, so finer tasks end
  // the launch more evenly over the CUs.
  L->comm_tm_last = last_split_tm(L->comm_tm);
  L->tasks_last = ((wl->T + L->comm_tm_last - 1) / L->comm_tm_last) * L->cb_per_split;
  L->max_tiles = (long long)wl->splits * L->ntps * ((L->rows + kBM - 1) / kBM + wl->E);
  size_t off = 0;
  L->status = off;   // word 0: status bits; bytes 4..255: reserved;
                     // 256..319: per-split consumer task counters;
                     // 320: launch epoch (u64); 328: finished workgroups;
                     // 332: started workgroups
  off += 512;
  L->wg_flags = off;
  off += (size_t)kMaxGrid * 4;
  L->split_flags = off;
  off += (size_t)wl->splits * kMaxGrid * 4;
  L->flags = off;
  off = round_up(off + (size_t)L->max_tiles * 4, 256);
  L->tok_cnt = off;
  off = round_up(off + (size_t)wl->T * 8, 256);
  L->inv = off;
  off = round_up(off + (size_t)wl->T * wl->topk * 8, 256);
  L->Y = off;
  // rows of L line-aligned split segments plus the padding (token bands use
  // one segment of round_up(H) <= L round_up(ceil(H/L)) elements)
  off = round_up(off + (size_t)L->rows * ((size_t)wl->splits * round_up_line(L->nsplit) + kYPad) * 2,
                 256);
  L->total = off;
  return true;
}

struct DevInfo {
  bool ready = false;
  int cus = 0;
  int occ = 0;
};
std::mutex g_mu;
DevInfo g_dev[64];

int device_info(int dev, DevInfo* out) {
  if (dev < 0 || dev >= 64) return MOE_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_dev[dev].ready) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return MOE_ERR_HIP;
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return MOE_ERR_HIP;
    if (cur != dev && hipSetDevice(dev) != hipSuccess) return MOE_ERR_HIP;
    int occ = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
        &occ, reinterpret_cast<const void*>(moe_gemm2_fused), kThreads, 0);
    hipFuncAttributes fa;
    const hipError_t e2 = hipFuncGetAttributes(&fa, reinterpret_cast<const void*>(moe_gemm2_fused));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || e2 != hipSuccess || occ <= 0) return MOE_ERR_HIP;
    // Every workgroup of the persistent grid must be resident at once (the
    // consumers wait on tiles of other workgroups), so the residency used
    // for the grid must never exceed what fits.  The occupancy query has
    // over-reported on this target for kernels that use the unified
    // register file, so it is capped by the LDS bound and by the one
    // workgroup per CU the kernel is compiled for (one wave per SIMD).
    const size_t lds = fa.sharedSizeBytes > 0 ? fa.sharedSizeBytes : sizeof(Smem);
    const int occ_lds = (int)(prop.maxSharedMemoryPerMultiProcessor / lds);
    occ = occ < occ_lds ? occ : occ_lds;
    occ = occ < kResidentPerCu ? occ : kResidentPerCu;
    if (occ <= 0) return MOE_ERR_UNSUPPORTED;
    g_dev[dev].cus = prop.multiProcessorCount;
    g_dev[dev].occ = occ;
    g_dev[dev].ready = true;
  }
  *out = g_dev[dev];
  return MOE_OK;
}

// rho_ref of the fused kernel on MI355X: mean consumer-task time over mean
// compute-tile time (one consumer wave over one compute wave), measured with
// the traced entry point at the reference configuration (T=16384, H=2048,
// I=704, E=32, top-6, L=2, C=32, 64-token tasks; the last split's 16-token
// tasks counted at four times their time): 30.4 us / 19.1 us = 1.59 (three
// runs: 1.576 to 1.598).  MOE_GEMM2_RHO_REF="num/den" overrides it.
constexpr int64_t kRhoRefNum = 159;
constexpr int64_t kRhoRefDen = 100;
// The same ratio for the atomic scatter (one task = one compute tile's
// rows), measured the same way: 26.2 us / 21.5 us = 1.22.
constexpr int64_t kRhoScatterNum = 122;
constexpr int64_t kRhoScatterDen = 100;
// The same for token bands (mode 2), 64-token tasks over 1024 columns:
// 36.7 us / 20.3 us = 1.81.
constexpr int64_t kRhoBandsNum = 181;
constexpr int64_t kRhoBandsDen = 100;
// The split cost of token bands: the compute workgroups' busy time per band
// boundary (the publish, ~5 us, and the slower stages around it) over the
// mean tile time, traced at T = 16384, H = 2048, I = 704, E = 32, top-6,
// uniform routing, C = 0, L = 1, 2, 4: 8.5 us / 19.7 us = 0.43.
constexpr int64_t kSplitCostBandsNum = 43;
constexpr int64_t kSplitCostBandsDen = 100;
constexpr int kDefaultFixedC = 8;
// C_max (eq:c-domain) from the kernel's saturation characterization: with
// T = 16384, H = 2048, I = 704, E = 32, top-6, uniform routing, L = 2, the
// launch takes 454 / 447 / 445 / 454 / 475 us at C = 64 / 72 / 80 / 96 /
// 112 (three runs alike), a plateau from 64 to 96.  The candidate set ends
// where the plateau starts: the model's tile time does not depend on P, so
// inside the plateau its picks fall short of the measured best (with
// C_max = 80 up to 8.9% above it, against 3.3% at most with 64).
constexpr int kCMax = 64;

// Selector parameters of a launch.  comm_tm is the owner-write task's token
// count; rho_ref, calibrated for kCommTM-token tasks, scales with it (a
// task's bytes are proportional to its tokens).
void fill_params(const DevInfo& d, int mode, int topk, int comm_tm, moe_select_params_t* p) {
  p->tile_m = kBM;
  p->tile_n = kBN;
  p->comm_tile_m = comm_tm;
  p->comm_tile_n = kCommTN;
  if (mode == 1) {
    // a scatter task is one compute tile: kBM routed rows, i.e. about
    // kBM / topk tokens' worth of rows, by kBN columns
    p->comm_tile_m = topk > 0 && kBM / topk > 0 ? kBM / topk : 1;
    p->comm_tile_n = kBN;
  }
  p->occ_comp = d.occ;
  p->occ_comm = d.occ;
  p->num_cus = d.cus;
  // C = 0 (every workgroup computes, then every workgroup consumes) is a
  // legal launch of this kernel, so it is part of the candidate set.
  p->c_min = 0;
  p->c_max = kCMax;
  p->groups = 1;
  p->rho_ref_num = mode == 1 ? kRhoScatterNum : mode == 2 ? kRhoBandsNum : kRhoRefNum;
  p->rho_ref_den = mode == 1 ? kRhoScatterDen : mode == 2 ? kRhoBandsDen : kRhoRefDen;
  p->split_axis = mode == 2 ? 1 : 0;
  // token bands: the compute workgroups drain into every band's remaining
  // tasks (the work-conserving drain)
  p->drain = mode == 2 ? 2 : 0;
  // a scatter task needs only its own tile and waits for the published
  // prefix up to it: its work is released a compute wave at a time
  p->readiness = mode == 1 ? 1 : 0;
  const char* env = mode == 1 ? "MOE_GEMM2_RHO_REF_SCATTER"
                    : mode == 2 ? "MOE_GEMM2_RHO_REF_BANDS" : "MOE_GEMM2_RHO_REF";
  if (const char* s = std::getenv(env)) {
    long long n = 0, q = 0;
    if (std::sscanf(s, "%lld/%lld", &n, &q) == 2 && n > 0 && q > 0) {
      p->rho_ref_num = n;
      p->rho_ref_den = q;
    }
  }
  if (mode != 1 && comm_tm != kCommTM) {
    p->rho_ref_num *= comm_tm;
    p->rho_ref_den *= kCommTM;
  }
  // owner-write over column splits: the last split's tasks are cut finer
  p->comm_tile_m_last = mode == 0 ? last_split_tm(comm_tm) : 0;
  p->k_ref = 704;
  p->tile_m_ref = kBM;
  p->tile_n_ref = kBN;
  p->d_ref = 1;
  // the calibration's top-k and task width, for the k/H-aware rho of the
  // owner-write consumers (off unless MOE_GEMM2_RHO_KH=1; a scatter task's
  // bytes do not depend on top-k)
  p->topk_ref = 6;
  p->comm_tile_n_ref = kCommTN;
  p->rho_kh = 0;
  // token bands, where L is chosen as well: what each band's publish costs
  // the compute (the owner-write selection keeps the paper's model)
  p->split_cost_num = mode == 2 ? kSplitCostBandsNum : 0;
  p->split_cost_den = mode == 2 ? kSplitCostBandsDen : 1;
  if (mode != 1)
    if (const char* s = std::getenv("MOE_GEMM2_RHO_KH")) p->rho_kh = std::atoi(s) == 1 ? 1 : 0;
}

inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// A workspace's metadata regions (flags, per-token counters, inverse map)
// sit at offsets that depend on the workload's dimensions.  Their epoch
// tags make stale values harmless only within one layout: after a launch
// with another layout, a region may hold what another region left (a large
// flag word read as a per-token counter would never reopen).  So the
// library remembers the layout each workspace was last launched with, and
// zeroes the metadata (everything before the Y staging, a few hundred KB)
// on the launch's stream when the layout changes.  A workspace that
// moe_gemm2_workspace_init zeroed accepts any layout.
constexpr uint64_t kWsZeroed = 0;
std::mutex g_ws_mu;
std::unordered_map<uintptr_t, uint64_t> g_ws_layout;

uint64_t layout_signature(const moe_workload_t* wl, const Layout& L) {
  uint64_t h = 1469598103934665603ull;   // FNV-1a over the fields that place or index regions
  const long long f[] = {(long long)L.flags, (long long)L.tok_cnt, (long long)L.inv,
                         (long long)L.Y,     wl->T,                  wl->topk,
                         L.rows,             L.max_tiles,            wl->H};
  for (long long v : f)
    for (int i = 0; i < 8; ++i) {
      h ^= (uint64_t)((v >> (8 * i)) & 0xff);
      h *= 1099511628211ull;
    }
  return h | 1;   // never kWsZeroed
}

void note_workspace_zeroed(const void* ws) {
  std::lock_guard<std::mutex> lk(g_ws_mu);
  if (g_ws_layout.size() > 4096) g_ws_layout.clear();
  g_ws_layout[(uintptr_t)ws] = kWsZeroed;
}

// True when the metadata regions must be zeroed before a launch with
// layout `sig` (a workspace not seen before, or last used with another
// layout); records `sig` as the workspace's layout.
bool workspace_needs_clear(const void* ws, uint64_t sig) {
  std::lock_guard<std::mutex> lk(g_ws_mu);
  auto it = g_ws_layout.find((uintptr_t)ws);
  if (it != g_ws_layout.end() && (it->second == sig || it->second == kWsZeroed)) {
    it->second = sig;
    return false;
  }
  if (g_ws_layout.size() > 4096) g_ws_layout.clear();
  g_ws_layout[(uintptr_t)ws] = sig;
  return true;
}

// The workspace of moe_gemm2_combine_noalloc, for callers that cannot
// allocate device memory: one array in the code object's device memory,
// which every GPU the library runs on holds (at its own address) until the
// process ends.  Host code never uses its name as an address: the device
// address is looked up once per device (hipGetSymbolAddress) and kept.
constexpr size_t kScratchBytes = (size_t)MOE_GEMM2_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "scratch size");
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

struct ScratchDev {
  void* ptr = nullptr;   // device address of `scratch` on that device
  uint64_t layout = 0;   // layout of its last launch (0: none yet, so the first clears it)
};
ScratchDev g_scratch[64];   // guarded by g_mu

// The scratch's device address on `dev` (the current device), looked up on
// the first call on that device.
int scratch_on_device(int dev, ScratchDev** out) {
  if (dev < 0 || dev >= 64) return MOE_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch[dev].ptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return MOE_ERR_HIP;
    if (!aligned(p, 256)) return MOE_ERR_HIP;
    g_scratch[dev].ptr = p;
  }
  *out = &g_scratch[dev];
  return MOE_OK;
}

// The launch epoch a freshly zeroed workspace starts from.  Readiness flags
// hold the low 32 bits of a launch's epoch, and a flag left by an earlier
// use of the same memory (another workspace at a reused address, or this
// workspace before a re-initialisation) must never equal a new launch's
// epoch, also where a stale copy of it may still be visible: so every
// initialisation starts 2^20 launches past the previous one, from a
// per-process random origin, and never at the zeroed state.  Epochs stay
// in [2^32, 2^33 + 2^32), far below the 2^40 at which the per-token
// counters' epoch tags would wrap.
std::atomic<uint64_t> g_epoch_inits{0};
uint64_t fresh_epoch_base() {
  static const uint64_t origin = [] {
    std::random_device rd;
    return ((uint64_t)rd() << 16) ^ (uint64_t)std::chrono::steady_clock::now().time_since_epoch().count();
  }();
  const uint64_t k = g_epoch_inits.fetch_add(1, std::memory_order_relaxed);
  return (1ull << 32) | ((origin + (k << 20)) & 0xffffffffull);
}
constexpr size_t kEpochWordIndex = 320 / 4;   // the header's launch-epoch word (bytes 320..327)

// Zeroes `bytes` (a multiple of 4) at workspace p on stream with a fill
// kernel (no memset node, so that a captured graph replays it correctly),
// and gives the workspace a fresh launch epoch.
hipError_t zero_async(void* p, size_t bytes, hipStream_t stream) {
  const size_t words = bytes / 4;
  const unsigned blocks = (unsigned)((words + 255) / 256 < 4096 ? (words + 255) / 256 : 4096);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks ? blocks : 1), dim3(256), 0, stream,
                     static_cast<uint32_t*>(p), words, kEpochWordIndex, fresh_epoch_base());
  return hipGetLastError();
}

// Consumer task geometry of a token-band launch (mode 2): tasks of TM tokens
// x min(1024, H) columns over the full width, TM = kCommTM halved (down to
// kCommTMMin) while there would be fewer than kTaskTarget tasks.  The
// workspace layout (sized for column splits) covers it: it has fewer tasks
// and no more tiles.
struct BandTasks {
  int comm_tm, comm_tn, cb, tasks;
};
BandTasks band_tasks(const moe_workload_t* wl) {
  BandTasks t;
  t.comm_tn = wl->H < kCommTN ? wl->H : kCommTN;
  t.cb = (wl->H + t.comm_tn - 1) / t.comm_tn;
  t.comm_tm = kCommTM;
  while (t.comm_tm > kCommTMMin &&
         (long long)((wl->T + t.comm_tm - 1) / t.comm_tm) * t.cb < kTaskTarget)
    t.comm_tm /= 2;
  t.tasks = ((wl->T + t.comm_tm - 1) / t.comm_tm) * t.cb;
  return t;
}

// Host-side checks of a launch's arguments other than the workspace (no HIP
// call); fills *L.
int validate_args(const void* x_perm, const void* w2, const int32_t* expert_offsets,
                  const int32_t* token_ids, const float* gate_w, const float* out,
                  const moe_workload_t* wl, int32_t num_consumers, int32_t mode, Layout* L) {
  int st = check_shape(wl);
  if (st != MOE_OK) return st;
  if (mode != 0 && mode != 1 && mode != 2) return MOE_ERR_INVALID_ARG;
  if (mode == 2 && (long long)(wl->E + 1) * wl->splits > kMaxBandTab) return MOE_ERR_UNSUPPORTED;
  if (mode != 2 && wl->H % (8 * wl->splits) != 0) return MOE_ERR_UNSUPPORTED;
  if (!make_layout(wl, L)) return MOE_ERR_INVALID_ARG;
  if (!expert_offsets || !out || (L->rows > 0 && (!x_perm || !token_ids || !gate_w)) || !w2)
    return MOE_ERR_INVALID_ARG;
  if (!aligned(x_perm, 16) || !aligned(w2, 16) || !aligned(out, 16) ||
      !aligned(expert_offsets, 4) || !aligned(token_ids, 4) || !aligned(gate_w, 4))
    return MOE_ERR_ALIGNMENT;
  if (wl->host_expert_counts) {
    long long sum = 0;
    for (int e = 0; e < wl->E; ++e) {
      if (wl->host_expert_counts[e] < 0) return MOE_ERR_INVALID_ARG;
      sum += wl->host_expert_counts[e];
    }
    if (sum != L->rows) return MOE_ERR_INVALID_ARG;
  }
  if (num_consumers < -1) return MOE_ERR_INVALID_ARG;
  return MOE_OK;
}

// `layout_slot`: where the workspace's last layout is kept when the
// workspace is the library's own scratch (NULL: the per-address record).
int launch(const void* x_perm, const void* w2, const int32_t* expert_offsets,
           const int32_t* token_ids, const float* gate_w, float* out, const moe_workload_t* wl,
           int32_t num_consumers, int32_t mode, void* workspace, size_t workspace_bytes,
           void* stream, uint64_t* trace, size_t trace_bytes, uint64_t* layout_slot = nullptr) {
  Layout L;
  int st = validate_args(x_perm, w2, expert_offsets, token_ids, gate_w, out, wl, num_consumers,
                         mode, &L);
  if (st != MOE_OK) return st;
  if (!workspace) return MOE_ERR_WORKSPACE;
  if (!aligned(workspace, 256)) return MOE_ERR_ALIGNMENT;
  if (workspace_bytes < L.total) return MOE_ERR_WORKSPACE;
  if (trace) {
    if (!aligned(trace, 8)) return MOE_ERR_ALIGNMENT;
    if (trace_bytes < moe_gemm2_trace_size(wl)) return MOE_ERR_INVALID_ARG;
  }

  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MOE_ERR_HIP;
  DevInfo d;
  st = device_info(dev, &d);
  if (st != MOE_OK) return st;

  int C = num_consumers;
  if (C < 0) {
    const char* sel = std::getenv("MOE_GEMM2_SELECTOR");
    if (sel && sel[0] == '0') {
      C = kDefaultFixedC;
    } else {
      moe_select_params_t p;
      fill_params(d, mode, wl->topk, mode == 2 ? band_tasks(wl).comm_tm : L.comm_tm, &p);
      moe_workload_t w = *wl;
      if (w.ranks <= 0) w.ranks = 1;
      moe_partition_t part;
      const int r = moe_select_partition(&w, &p, &part);
      if (r < 0) return r;
      C = part.C;
    }
  }
  int P, drain = mode == 2 ? 1 : 0;   // token bands: compute workgroups always drain
  if (C == 0) {
    P = d.occ * d.cus;
    drain = 1;
  } else {
    const int R = (C + d.occ - 1) / d.occ;
    P = d.occ * (d.cus - R);
    if (P <= 0) return MOE_ERR_NO_LEGAL_PARTITION;
  }
  if (wl->T == 0) return C;  // nothing to write
  if (C + P > kMaxGrid) return MOE_ERR_UNSUPPORTED;

  char* ws = static_cast<char*>(workspace);
  KArgs a;
  a.x = static_cast<const uint16_t*>(x_perm);
  a.w2 = static_cast<const uint16_t*>(w2);
  a.offsets = expert_offsets;
  a.token_ids = token_ids;
  a.gate_w = gate_w;
  a.out = out;
  a.Y = reinterpret_cast<uint16_t*>(ws + L.Y);
  a.tile_flags = reinterpret_cast<uint32_t*>(ws + L.flags);
  a.wg_flags = reinterpret_cast<uint32_t*>(ws + L.wg_flags);
  a.tok_cnt = reinterpret_cast<u64*>(ws + L.tok_cnt);
  a.inv = reinterpret_cast<int32_t*>(ws + L.inv);
  a.status = reinterpret_cast<uint32_t*>(ws + L.status);
  a.task_ctr = reinterpret_cast<uint32_t*>(ws + L.status + 256);
  a.split_flags = reinterpret_cast<uint32_t*>(ws + L.split_flags);
  a.trace = reinterpret_cast<u64*>(trace);
  a.rows = L.rows;
  a.max_tiles = L.max_tiles;
  a.spin_limit = 4000000;
  if (const char* s = std::getenv("MOE_GEMM2_SPIN_LIMIT")) {
    long long v = std::atoll(s);
    if (v > 0) a.spin_limit = v;
  }
  a.T = wl->T;
  a.H = wl->H;
  a.ysplit = round_up_line(L.nsplit);
  a.ypitch = wl->splits * a.ysplit + kYPad;
  a.I = wl->I;
  a.E = wl->E;
  a.topk = wl->topk;
  a.L = wl->splits;
  a.nsplit = L.nsplit;
  a.ntps = L.ntps;
  a.C = C;
  a.P = P;
  a.drain = drain;
  a.comm_tm = L.comm_tm;
  a.comm_tn = L.comm_tn;
  a.cb_per_split = L.cb_per_split;
  a.tasks_per_split = L.tasks_per_split;
  a.comm_tm_last = L.comm_tm_last;
  a.tasks_last = L.tasks_last;
  a.mode = mode;
  if (mode == 2) {   // token bands: every band spans the full width
    const BandTasks bt = band_tasks(wl);
    a.nsplit = wl->H;
    a.ntps = (wl->H + kBN - 1) / kBN;
    a.ysplit = round_up_line(wl->H);   // one segment; fits the column-split layout
    a.ypitch = a.ysplit + kYPad;
    a.comm_tm = bt.comm_tm;
    a.comm_tn = bt.comm_tn;
    a.cb_per_split = bt.cb;
    a.tasks_per_split = bt.tasks;
  }
  a.epoch_word = reinterpret_cast<u64*>(ws + L.status + 320);
  a.done_ctr = reinterpret_cast<uint32_t*>(ws + L.status + 328);
  a.start_ctr = reinterpret_cast<uint32_t*>(ws + L.status + 332);
  a.delay_mod = 1;
  a.delay_ticks = 0;
  if (const char* s = std::getenv("MOE_GEMM2_DEBUG_PUBLISH_DELAY")) {
    // "mod:ticks": compute workgroups c with c % mod == 0 hold every split
    // publish back by ticks of the 100 MHz clock (at most 10^6 = 10 ms)
    long long m = 0, t = 0;
    if (std::sscanf(s, "%lld:%lld", &m, &t) == 2 && m >= 1 && t > 0) {
      a.delay_mod = (int)(m < 4096 ? m : 4096);
      a.delay_ticks = t < 1000000 ? t : 1000000;
    }
  }

  hipStream_t s = static_cast<hipStream_t>(stream);
  const uint64_t sig = layout_signature(wl, L);
  bool clear;
  if (layout_slot) {
    std::lock_guard<std::mutex> lk(g_ws_mu);
    clear = *layout_slot != sig;
    *layout_slot = sig;
  } else {
    clear = workspace_needs_clear(workspace, sig);
  }
  if (clear && zero_async(workspace, L.Y, s) != hipSuccess) return MOE_ERR_HIP;
  hipLaunchKernelGGL(moe_gemm2_fused, dim3(C + P), dim3(kThreads), 0, s, a);
  if (hipGetLastError() != hipSuccess) return MOE_ERR_HIP;
  return C;
}

}  // namespace

extern "C" size_t moe_gemm2_workspace_size(const moe_workload_t* wl) {
  Layout L;
  return make_layout(wl, &L) ? L.total : 0;
}

extern "C" size_t moe_gemm2_trace_size(const moe_workload_t* wl) {
  Layout L;
  if (!make_layout(wl, &L)) return 0;
  // compute tiles, then consumer tasks (owner-write tasks or, for the
  // atomic scatter, one per compute tile)
  // consumer-task records: the most of the column-split tasks, the token-band
  // tasks and (atomic scatter) the compute tiles
  long long tasks = (long long)(wl->splits - 1) * L.tasks_per_split + L.tasks_last;
  const long long band = band_tasks(wl).tasks;
  if (band > tasks) tasks = band;
  return (size_t)(4 * L.max_tiles + 4 * (tasks > L.max_tiles ? tasks : L.max_tiles)) * 8;
}

extern "C" int moe_gemm2_workspace_init(void* workspace, size_t workspace_bytes, void* stream) {
  if (!workspace || workspace_bytes == 0) return MOE_ERR_INVALID_ARG;
  if (!aligned(workspace, 256)) return MOE_ERR_ALIGNMENT;
  if (zero_async(workspace, workspace_bytes, static_cast<hipStream_t>(stream)) != hipSuccess)
    return MOE_ERR_HIP;
  note_workspace_zeroed(workspace);
  return MOE_OK;
}

extern "C" int moe_gemm2_default_params(int device, moe_select_params_t* out) {
  if (!out) return MOE_ERR_INVALID_ARG;
  DevInfo d;
  const int st = device_info(device, &d);
  if (st != MOE_OK) return st;
  fill_params(d, 0, 0, kCommTM, out);
  return MOE_OK;
}

extern "C" int moe_gemm2_default_params_ex(int device, int32_t mode, int32_t topk,
                                           moe_select_params_t* out) {
  if (!out || (mode != 0 && mode != 1 && mode != 2) || topk <= 0) return MOE_ERR_INVALID_ARG;
  DevInfo d;
  const int st = device_info(device, &d);
  if (st != MOE_OK) return st;
  fill_params(d, mode, topk, kCommTM, out);
  return MOE_OK;
}

extern "C" int moe_gemm2_launch_params(int device, int32_t mode, const moe_workload_t* wl,
                                       moe_select_params_t* out) {
  if (!out || (mode != 0 && mode != 1 && mode != 2)) return MOE_ERR_INVALID_ARG;
  Layout L;
  if (!make_layout(wl, &L)) return check_shape(wl) == MOE_ERR_UNSUPPORTED ? MOE_ERR_UNSUPPORTED
                                                                          : MOE_ERR_INVALID_ARG;
  if (mode != 2 && wl->H % (8 * wl->splits) != 0) return MOE_ERR_UNSUPPORTED;
  if (mode == 2 && (long long)(wl->E + 1) * wl->splits > kMaxBandTab) return MOE_ERR_UNSUPPORTED;
  DevInfo d;
  const int st = device_info(device, &d);
  if (st != MOE_OK) return st;
  fill_params(d, mode, wl->topk, mode == 2 ? band_tasks(wl).comm_tm : L.comm_tm, out);
  return MOE_OK;
}

extern "C" int moe_gemm2_combine(const void* x_perm, const void* w2,
                                 const int32_t* expert_offsets, const int32_t* token_ids,
                                 const float* gate_w, float* out, const moe_workload_t* wl,
                                 int32_t num_consumers, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  return launch(x_perm, w2, expert_offsets, token_ids, gate_w, out, wl, num_consumers, 0,
                workspace, workspace_bytes, stream, nullptr, 0);
}

extern "C" int moe_gemm2_combine_traced(const void* x_perm, const void* w2,
                                        const int32_t* expert_offsets, const int32_t* token_ids,
                                        const float* gate_w, float* out,
                                        const moe_workload_t* wl, int32_t num_consumers,
                                        void* workspace, size_t workspace_bytes, void* stream,
                                        uint64_t* trace, size_t trace_bytes) {
  if (!trace) return MOE_ERR_INVALID_ARG;
  return launch(x_perm, w2, expert_offsets, token_ids, gate_w, out, wl, num_consumers, 0,
                workspace, workspace_bytes, stream, trace, trace_bytes);
}

extern "C" int moe_gemm2_combine_ex(const void* x_perm, const void* w2,
                                    const int32_t* expert_offsets, const int32_t* token_ids,
                                    const float* gate_w, float* out, const moe_workload_t* wl,
                                    int32_t num_consumers, int32_t mode, void* workspace,
                                    size_t workspace_bytes, void* stream, uint64_t* trace,
                                    size_t trace_bytes) {
  return launch(x_perm, w2, expert_offsets, token_ids, gate_w, out, wl, num_consumers, mode,
                workspace, workspace_bytes, stream, trace, trace_bytes);
}

extern "C" int moe_gemm2_combine_noalloc(const void* x_perm, const void* w2,
                                         const int32_t* expert_offsets, const int32_t* token_ids,
                                         const float* gate_w, float* out,
                                         const moe_workload_t* wl, int32_t num_consumers,
                                         int32_t mode, void* stream) {
  Layout L;
  const int st = validate_args(x_perm, w2, expert_offsets, token_ids, gate_w, out, wl,
                               num_consumers, mode, &L);
  if (st != MOE_OK) return st;
  if (L.total > kScratchBytes) return MOE_ERR_WORKSPACE;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MOE_ERR_HIP;
  ScratchDev* sd = nullptr;
  const int r = scratch_on_device(dev, &sd);
  if (r != MOE_OK) return r;
  return launch(x_perm, w2, expert_offsets, token_ids, gate_w, out, wl, num_consumers, mode,
                sd->ptr, kScratchBytes, stream, nullptr, 0, &sd->layout);
}

extern "C" int moe_gemm2_status(void* workspace, void* stream, int clear) {
  if (!workspace) return MOE_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (hipStreamSynchronize(s) != hipSuccess) return MOE_ERR_HIP;
  uint32_t v = 0;
  if (hipMemcpy(&v, workspace, 4, hipMemcpyDeviceToHost) != hipSuccess) return MOE_ERR_HIP;
  if (clear) {
    const uint32_t z = 0;
    if (hipMemcpy(workspace, &z, 4, hipMemcpyHostToDevice) != hipSuccess) return MOE_ERR_HIP;
  }
  if (v & kStTimeout) return MOE_ERR_TIMEOUT;
  if (v & kStBadRouting) return MOE_ERR_BAD_ROUTING;
  return MOE_OK;
}

// ---- the up-projection stage and the whole post-router layer ----------------------
namespace {

int check_gemm1_shape(const moe_workload_t* wl) {
  if (!wl) return MOE_ERR_INVALID_ARG;
  if (wl->T < 0 || wl->H <= 0 || wl->I <= 0 || wl->E <= 0 || wl->topk <= 0 || wl->rows < 0)
    return MOE_ERR_INVALID_ARG;
  if (wl->E > kMaxE || wl->topk > kMaxTopk) return MOE_ERR_UNSUPPORTED;
  if (wl->H % 8 != 0 || wl->I % 16 != 0) return MOE_ERR_UNSUPPORTED;
  const long long rows = wl->rows > 0 ? wl->rows : (long long)wl->T * wl->topk;
  if (rows > (long long)INT32_MAX) return MOE_ERR_UNSUPPORTED;
  // hidden and an expert's W1 slice are addressed with 32-bit byte offsets
  if ((long long)wl->T * wl->H * 2 > 0x7fffffffLL || (long long)wl->H * wl->I * 4 > 0x7fffffffLL)
    return MOE_ERR_UNSUPPORTED;
  const long long ntps = (2LL * wl->I + kBN - 1) / kBN;
  if ((long long)wl->E * ((rows + kBM - 1) / kBM + 1) * ntps > (long long)INT32_MAX / 2)
    return MOE_ERR_UNSUPPORTED;
  return MOE_OK;
}

int launch_gemm1(const void* hidden, const void* w1, const int32_t* expert_offsets,
                 const int32_t* token_ids, void* x_perm, const moe_workload_t* wl, void* workspace,
                 size_t workspace_bytes, void* stream) {
  const int st = check_gemm1_shape(wl);
  if (st != MOE_OK) return st;
  const long long rows = wl->rows > 0 ? wl->rows : (long long)wl->T * wl->topk;
  if (!hidden || !w1 || !expert_offsets || (rows > 0 && (!token_ids || !x_perm)))
    return MOE_ERR_INVALID_ARG;
  if (!aligned(hidden, 16) || !aligned(w1, 16) || !aligned(x_perm, 16) ||
      !aligned(expert_offsets, 4) || !aligned(token_ids, 4))
    return MOE_ERR_ALIGNMENT;
  if (!workspace) return MOE_ERR_WORKSPACE;
  if (!aligned(workspace, 256)) return MOE_ERR_ALIGNMENT;
  if (workspace_bytes < 512) return MOE_ERR_WORKSPACE;
  if (wl->host_expert_counts) {
    long long sum = 0;
    for (int e = 0; e < wl->E; ++e) {
      if (wl->host_expert_counts[e] < 0) return MOE_ERR_INVALID_ARG;
      sum += wl->host_expert_counts[e];
    }
    if (sum != rows) return MOE_ERR_INVALID_ARG;
  }
  if (rows == 0 || wl->T == 0) return MOE_OK;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MOE_ERR_HIP;
  DevInfo d;
  const int r = device_info(dev, &d);
  if (r != MOE_OK) return r;
  char* ws = static_cast<char*>(workspace);
  G1Args a;
  a.hidden = static_cast<const uint16_t*>(hidden);
  a.w1 = static_cast<const uint16_t*>(w1);
  a.offsets = expert_offsets;
  a.token_ids = token_ids;
  a.xout = static_cast<uint16_t*>(x_perm);
  a.status = reinterpret_cast<uint32_t*>(ws);
  a.rows = rows;
  a.T = wl->T;
  a.H = wl->H;
  a.I = wl->I;
  a.E = wl->E;
  a.ntps = (2 * wl->I + kBN - 1) / kBN;
  a.nsplit = 2 * wl->I;
  const int grid = d.occ * d.cus;
  hipLaunchKernelGGL(moe_gemm1_swiglu_kernel, dim3(grid), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), a);
  return hipGetLastError() == hipSuccess ? MOE_OK : MOE_ERR_HIP;
}

}  // namespace

extern "C" int moe_gemm1_swiglu(const void* hidden, const void* w1, const int32_t* expert_offsets,
                                const int32_t* token_ids, void* x_perm, const moe_workload_t* wl,
                                void* workspace, size_t workspace_bytes, void* stream) {
  return launch_gemm1(hidden, w1, expert_offsets, token_ids, x_perm, wl, workspace,
                      workspace_bytes, stream);
}

extern "C" int moe_gemm1_pack_weights(const void* w_gate_up, void* w1_packed, int32_t E,
                                      int32_t H, int32_t I, void* stream) {
  if (!w_gate_up || !w1_packed || w_gate_up == w1_packed || E <= 0 || H <= 0 || I <= 0)
    return MOE_ERR_INVALID_ARG;
  if (I % 16 != 0) return MOE_ERR_UNSUPPORTED;
  if (!aligned(w_gate_up, 2) || !aligned(w1_packed, 2)) return MOE_ERR_ALIGNMENT;
  const long long n = (long long)E * H * 2 * I;
  const long long blocks = (n + 255) / 256;
  hipLaunchKernelGGL(pack_w1_kernel, dim3((unsigned)(blocks < 8192 ? blocks : 8192)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), static_cast<const uint16_t*>(w_gate_up),
                     static_cast<uint16_t*>(w1_packed), n, (int)I);
  return hipGetLastError() == hipSuccess ? MOE_OK : MOE_ERR_HIP;
}

extern "C" size_t moe_layer_workspace_size(const moe_workload_t* wl) {
  Layout L;
  if (check_gemm1_shape(wl) != MOE_OK || !make_layout(wl, &L)) return 0;
  return round_up(L.total, 256) + round_up((size_t)L.rows * wl->I * 2, 256);
}

extern "C" int moe_layer_forward(const void* hidden, const void* w1, const void* w2,
                                 const int32_t* expert_offsets, const int32_t* token_ids,
                                 const float* gate_w, float* out, const moe_workload_t* wl,
                                 int32_t num_consumers, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  int st = check_gemm1_shape(wl);
  if (st != MOE_OK) return st;
  st = check_shape(wl);
  if (st != MOE_OK) return st;
  Layout L;
  if (!make_layout(wl, &L)) return MOE_ERR_INVALID_ARG;
  if (!workspace) return MOE_ERR_WORKSPACE;
  if (!aligned(workspace, 256)) return MOE_ERR_ALIGNMENT;
  const size_t gemm2_bytes = round_up(L.total, 256);
  if (workspace_bytes < moe_layer_workspace_size(wl)) return MOE_ERR_WORKSPACE;
  void* x_perm = static_cast<char*>(workspace) + gemm2_bytes;
  st = launch_gemm1(hidden, w1, expert_offsets, token_ids, x_perm, wl, workspace, gemm2_bytes,
                    stream);
  if (st != MOE_OK) return st;
  return launch(x_perm, w2, expert_offsets, token_ids, gate_w, out, wl, num_consumers, 0,
                workspace, gemm2_bytes, stream, nullptr, 0);
}
