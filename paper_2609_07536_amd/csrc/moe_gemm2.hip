// Fused MoE GEMM2 + combine for gfx950 (MI355X), and its C ABI.
//
// One persistent kernel, two workgroup roles (paper: Background,
// "Fine-Grained Overlap and GPU Residency"; Method, "Split-level
// dependency"):
//
//  * compute workgroups walk the global tile sequence (split-major, then
//    expert, then m-tile, then n-tile; compute workgroup b takes tiles b,
//    b+P, b+2P, ...), run one 256x256 tile of Y = x_perm @ W2[e] on bf16
//    MFMA with LDS double buffering, store it to the bf16 staging buffer and
//    publish it (per-tile flag and per-split counter, agent-scope release);
//  * consumer workgroups wait until every tile of a split is published
//    (agent-scope acquire), then, per task of 128 tokens x 1024 columns,
//    gather each token's rows, weight them by the gates and write the
//    token's output once, summing the rows in ascending row order so the
//    result does not depend on the partition.
//
// Every workgroup first adds its share of rows to the token->rows inverse
// map.  Flags and counters carry the launch's epoch, so nothing has to be
// cleared between launches and a stale value can never satisfy a wait.
// Compute workgroups never wait, so the grid drains even if consumers are
// not all resident; every consumer wait is bounded.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>

#include "moe_gemm2.h"

namespace {

constexpr int kThreads = 256;           // 4 waves of 64
constexpr int kBM = 256;                // compute tile rows (routed rows)
constexpr int kBN = 256;                // compute tile columns (hidden)
constexpr int kBK = 64;                 // reduction step staged in LDS
constexpr int kCommTM = 128;            // consumer task: tokens
constexpr int kCommTN = 1024;           // consumer task: columns (at most)
constexpr int kMaxE = 1024;
constexpr int kMaxSplits = 16;
constexpr int kMaxTopk = 64;
constexpr int kMaxGrid = 4096;

constexpr uint32_t kStBadRouting = 1u;
constexpr uint32_t kStTimeout = 2u;

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned long long u64;

struct KArgs {
  const uint16_t* x;          // [rows, I] bf16
  const uint16_t* w2;         // [E, I, H] bf16
  const int32_t* offsets;     // [E+1]
  const int32_t* token_ids;   // [rows]
  const float* gate_w;        // [rows]
  float* out;                 // [T, H]
  uint16_t* Y;                // [rows, H] bf16 staging
  uint32_t* tile_flags;       // [max_tiles]: epoch once tile g is published
  uint32_t* wg_flags;         // [kMaxGrid]: epoch once workgroup b added its inverse-map rows
  u64* tok_cnt;               // [T]: epoch-tagged count of each token's rows
  int32_t* inv;               // [T, topk]
  uint32_t* status;           // [1]
  u64* trace;                 // optional
  long long rows;             // capacity of x / Y / token_ids / gate_w
  long long max_tiles;        // capacity of tile_flags
  long long spin_limit;
  int T, H, I, E, topk, L;
  int nsplit;                 // columns per split (H / L)
  int ntps;                   // compute n-tiles per split
  int C, P;                   // consumer and compute workgroups
  int drain;                  // compute workgroups also take consumer tasks
  int comm_tn;                // consumer task width (<= kCommTN)
  int cb_per_split;           // consumer column blocks per split
  int tasks_per_split;
  uint32_t epoch;
};

struct Smem {
  uint16_t a[2][kBM * kBK];   // x tile: row m, 8 chunks of 8 k (swizzled)
  uint16_t b[2][kBN * kBK];   // W2^T tile: row n, 8 chunks of 8 k (swizzled)
  int start[kMaxE];           // sanitized first row of each expert
  int count[kMaxE];           // sanitized row count of each expert
  int tile_prefix[kMaxE + 1]; // exclusive prefix of ceil(count/kBM)
  int scan[kThreads];
  int flag;
};

// ---- LDS swizzles ----------------------------------------------------------
// A row holds 64 bf16 = 8 chunks of 16 bytes; the chunk index is XORed with
// a row function so that 8 consecutive lanes of every access pattern hit 8
// distinct chunks.  x tile: MFMA reads walk 8 consecutive rows.  W2^T tile:
// MFMA reads walk rows {8q + i + 4h}, staging writes walk rows {8l + c}.
__device__ __forceinline__ int swz_a(int m) { return (m ^ (m >> 3)) & 7; }
__device__ __forceinline__ int swz_b(int n) {
  return ((n ^ (n >> 3)) & 3) | ((((n >> 3) ^ (n >> 5)) & 1) << 2);
}

// ---- memory-model helpers ----------------------------------------------------
__device__ __forceinline__ u64 ld_relaxed(u64* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Increment an epoch-tagged counter (high 32 bits: epoch, low: count); a
// counter from an older epoch counts as zero.  Returns the count before.
__device__ uint32_t epoch_inc(u64* p, uint32_t epoch) {
  u64 old = ld_relaxed(p);
  while (true) {
    const bool cur = (uint32_t)(old >> 32) == epoch;
    const u64 nw = cur ? old + 1ull : (((u64)epoch << 32) | 1ull);
    if (__hip_atomic_compare_exchange_strong(p, &old, nw, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT))
      return cur ? (uint32_t)old : 0u;
  }
}

__device__ __forceinline__ uint32_t epoch_count(u64 v, uint32_t epoch) {
  return (uint32_t)(v >> 32) == epoch ? (uint32_t)v : 0u;
}

__device__ __forceinline__ u64 now_100mhz() { return __builtin_amdgcn_s_memrealtime(); }

// Wave 0 polls flags[0..n) until every flag equals the epoch (bounded),
// advancing past the leading run of set flags; then the whole workgroup
// acquires.  Returns false (and records a timeout) if the bound expired.
__device__ bool wait_flags(Smem& sm, uint32_t* flags, long long n, const KArgs& a) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    long long i = 0, spins = 0;
    int ok = 1;
    while (i < n) {
      const long long idx = i + lane;
      const uint32_t v = idx < n ? __hip_atomic_load(&flags[idx], __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT)
                                 : a.epoch;
      const u64 ready = __ballot(v == a.epoch);
      if (ready == ~0ull) {
        i += 64;
        continue;
      }
      i += __builtin_ctzll(~ready);   // leading set flags stay set
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
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  __syncthreads();  // sm.flag may be rewritten by the next wait
  return ok;
}

// ---- prologue: expert ranges and the routed-tile prefix ----------------------
// Offsets are clamped into [0, rows] and made non-decreasing so every row
// range stays inside the buffers even for bad input (which is flagged).
__device__ void load_experts(Smem& sm, const KArgs& a) {
  const int tid = threadIdx.x;
  bool bad = false;
  for (int e = tid; e < a.E; e += kThreads) {
    long long s = a.offsets[e], en = a.offsets[e + 1];
    if (e == 0 && s != 0) bad = true;
    if (en < s || en > a.rows) bad = true;
    s = s < 0 ? 0 : (s > a.rows ? a.rows : s);
    en = en < s ? s : (en > a.rows ? a.rows : en);
    sm.start[e] = (int)s;
    sm.count[e] = (int)(en - s);
  }
  if (bad && a.status)
    __hip_atomic_fetch_or(a.status, kStBadRouting, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  // exclusive scan of ceil(count/kBM): each thread scans a contiguous chunk
  const int chunk = (a.E + kThreads - 1) / kThreads;
  const int lo = tid * chunk, hi = min(a.E, lo + chunk);
  int local = 0;
  for (int e = lo; e < hi; ++e) local += (sm.count[e] + kBM - 1) / kBM;
  sm.scan[tid] = local;
  __syncthreads();
  for (int d = 1; d < kThreads; d <<= 1) {
    const int v = tid >= d ? sm.scan[tid - d] : 0;
    __syncthreads();
    sm.scan[tid] += v;
    __syncthreads();
  }
  int run = sm.scan[tid] - local;
  for (int e = lo; e < hi; ++e) {
    sm.tile_prefix[e] = run;
    run += (sm.count[e] + kBM - 1) / kBM;
  }
  if (tid == kThreads - 1) sm.tile_prefix[a.E] = sm.scan[kThreads - 1];
  __syncthreads();
}

// Rows of each token, for the owner-write combine.
__device__ void build_inverse(const KArgs& a, long long rows_dev) {
  const long long stride = (long long)gridDim.x * kThreads;
  for (long long r = (long long)blockIdx.x * kThreads + threadIdx.x; r < rows_dev; r += stride) {
    const int t = a.token_ids[r];
    if (t < 0 || t >= a.T) {
      __hip_atomic_fetch_or(a.status, kStBadRouting, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      continue;
    }
    const uint32_t slot = epoch_inc(&a.tok_cnt[t], a.epoch);
    if (slot >= (uint32_t)a.topk) {
      __hip_atomic_fetch_or(a.status, kStBadRouting, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      continue;
    }
    a.inv[(long long)t * a.topk + slot] = (int32_t)r;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __syncthreads();
  if (threadIdx.x == 0) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __hip_atomic_store(&a.wg_flags[blockIdx.x], a.epoch, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  }
}

// ---- compute role: one 256x256 tile ------------------------------------------
// The MFMA computes D = Y^T for the tile: its A operand is W2^T (rows n) and
// its B operand is x (columns m), both holding 8 consecutive k per lane.  A
// wave owns 128 n x 128 m as 8 x 8 blocks of v_mfma_f32_16x16x32_bf16.
// Inside a pair of n-blocks (2c, 2c+1) the MFMA row rho of block 2c+h maps
// to n = 32c + 8(rho/4) + 4h + rho%4, so a lane's 4+4 accumulators of the
// pair are 8 consecutive columns of one row of Y: one 16-byte store.
__device__ __forceinline__ void stage_load(const KArgs& a, const uint16_t* xg, const uint16_t* wg,
                                           int rows_valid, int cols_valid, int kt, u32x4 (&ra)[8],
                                           u32x4 (&rb)[8]) {
  const int tid = threadIdx.x;
  const int k0 = kt * kBK;
  const int kx = k0 + 8 * (tid & 7);
  const bool kx_ok = kx < a.I;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int m = (tid >> 3) + 32 * j;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (kx_ok && m < rows_valid) v = *(const u32x4*)(xg + (size_t)m * a.I + kx);
    ra[j] = v;
  }
  const int kb = k0 + 8 * (tid >> 5);
  const int nn = 8 * (tid & 31);
  const bool n_ok = nn < cols_valid;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    u32x4 v = {0u, 0u, 0u, 0u};
    if (n_ok && kb + j < a.I) v = *(const u32x4*)(wg + (size_t)(kb + j) * a.H + nn);
    rb[j] = v;
  }
}

__device__ __forceinline__ void stage_store(Smem& sm, int buf, const u32x4 (&ra)[8],
                                            const u32x4 (&rb)[8]) {
  const int tid = threadIdx.x;
  uint16_t* As = sm.a[buf];
  uint16_t* Bs = sm.b[buf];
  const int kc = tid & 7;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int m = (tid >> 3) + 32 * j;
    *(u32x4*)(As + m * kBK + ((kc ^ swz_a(m)) << 3)) = ra[j];
  }
  // rb[j] = W2[k = kb + j][n = nn .. nn+7]; write row n = nn + c of W2^T
  // holding k = kb .. kb+7: an 8x8 transpose of 16-bit values.
  const int kcb = tid >> 5;
  const int nn = 8 * (tid & 31);
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int d = c >> 1;
    const uint32_t sel = (c & 1) ? 0x07060302u : 0x05040100u;
    u32x4 v;
    v[0] = __builtin_amdgcn_perm(rb[1][d], rb[0][d], sel);
    v[1] = __builtin_amdgcn_perm(rb[3][d], rb[2][d], sel);
    v[2] = __builtin_amdgcn_perm(rb[5][d], rb[4][d], sel);
    v[3] = __builtin_amdgcn_perm(rb[7][d], rb[6][d], sel);
    const int n = nn + c;
    *(u32x4*)(Bs + n * kBK + ((kcb ^ swz_b(n)) << 3)) = v;
  }
}

__device__ __forceinline__ void mma_step(const Smem& sm, int buf, f32x4 (&acc)[8][8]) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wn0 = (wave & 1) * 128;
  const int wm0 = (wave >> 1) * 128;
  const int lr = lane & 15, lq = lane >> 4;
  const uint16_t* As = sm.a[buf];
  const uint16_t* Bs = sm.b[buf];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const int kc = ks * 4 + lq;
    bf16x8 af[8], bm[8];
#pragma unroll
    for (int nb = 0; nb < 8; ++nb) {
      const int n = wn0 + 32 * (nb >> 1) + 8 * (lr >> 2) + 4 * (nb & 1) + (lr & 3);
      af[nb] = *(const bf16x8*)(Bs + n * kBK + ((kc ^ swz_b(n)) << 3));
    }
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      const int m = wm0 + 16 * mb + lr;
      bm[mb] = *(const bf16x8*)(As + m * kBK + ((kc ^ swz_a(m)) << 3));
    }
#pragma unroll
    for (int nb = 0; nb < 8; ++nb)
#pragma unroll
      for (int mb = 0; mb < 8; ++mb)
        acc[nb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[nb], bm[mb], acc[nb][mb], 0, 0, 0);
  }
}

__device__ void compute_tile(Smem& sm, const KArgs& a, int e, int r0, int rows_valid, int n0,
                             int cols_valid, u64* t_mid) {
  const uint16_t* xg = a.x + (size_t)r0 * a.I;
  const uint16_t* wg = a.w2 + (size_t)e * a.I * a.H + n0;
  const int nk = (a.I + kBK - 1) / kBK;

  f32x4 acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 ra[8], rb[8];
  stage_load(a, xg, wg, rows_valid, cols_valid, 0, ra, rb);
  stage_store(sm, 0, ra, rb);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) stage_load(a, xg, wg, rows_valid, cols_valid, kt + 1, ra, rb);
    mma_step(sm, cur, acc);
    if (more) stage_store(sm, cur ^ 1, ra, rb);
    __syncthreads();
  }
  t_mid[0] = now_100mhz();

  // epilogue: bf16 rows of Y, 16 bytes per lane per n-block pair
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wn0 = (wave & 1) * 128;
  const int wm0 = (wave >> 1) * 128;
  const int lr = lane & 15, lq = lane >> 4;
#pragma unroll
  for (int mb = 0; mb < 8; ++mb) {
    const int m = wm0 + 16 * mb + lr;
    if (m >= rows_valid) continue;
    uint16_t* yrow = a.Y + (size_t)(r0 + m) * a.H + n0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int n = wn0 + 32 * c + 8 * lq;
      if (n >= cols_valid) continue;
      bf16x8 v;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[i] = (__bf16)acc[2 * c][mb][i];
        v[4 + i] = (__bf16)acc[2 * c + 1][mb][i];
      }
      __builtin_nontemporal_store(v, (bf16x8*)(yrow + n));
    }
  }
  t_mid[1] = now_100mhz();
}

// ---- consumer role: one task --------------------------------------------------
__device__ __forceinline__ float bf16lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

// The rows of token t sorted ascending, spread over the wave: lane j < n
// holds the j-th row (rs) and its gate bits (gs).  Rows of a token are
// distinct, so a lane's rank among the n rows is its sorted position.
__device__ __forceinline__ int token_rows(const KArgs& a, int t, int* rs, int* gs) {
  const int lane = threadIdx.x & 63;
  const uint32_t have = epoch_count(ld_relaxed(&a.tok_cnt[t]), a.epoch);
  const int n = (int)(have < (uint32_t)a.topk ? have : (uint32_t)a.topk);
  int r = 0;
  float g = 0.f;
  if (lane < n) {
    r = a.inv[(long long)t * a.topk + lane];
    g = a.gate_w[r];
  }
  int rank = lane;
  if (lane < n) {
    rank = 0;
    for (int i = 0; i < n; ++i) rank += __builtin_amdgcn_readlane(r, i) < r ? 1 : 0;
  }
  *rs = __builtin_amdgcn_ds_permute(rank << 2, r);
  *gs = __builtin_amdgcn_ds_permute(rank << 2, __float_as_int(g));
  return n;
}

__device__ __forceinline__ void fma8(float (&acc)[8], float g, const u32x4& v) {
  acc[0] = fmaf(g, bf16lo(v[0]), acc[0]);
  acc[1] = fmaf(g, bf16hi(v[0]), acc[1]);
  acc[2] = fmaf(g, bf16lo(v[1]), acc[2]);
  acc[3] = fmaf(g, bf16hi(v[1]), acc[3]);
  acc[4] = fmaf(g, bf16lo(v[2]), acc[4]);
  acc[5] = fmaf(g, bf16hi(v[2]), acc[5]);
  acc[6] = fmaf(g, bf16lo(v[3]), acc[6]);
  acc[7] = fmaf(g, bf16hi(v[3]), acc[7]);
}

// Rows j0 .. j0+U-1 of two tokens at two column chunks: all loads first
// (a padding row j >= n re-reads row n-1 and gets weight 0), then the FMAs
// in ascending row order.  n >= 1 for both tokens; every row read is one
// this launch has written, so its values are finite and weight 0 adds 0.
template <int U>
__device__ __forceinline__ void gather_step(const KArgs& a, int j0, const int (&rs)[2],
                                            const int (&gs)[2], const int (&n)[2],
                                            const int (&col)[2], float (&acc)[2][2][8]) {
  u32x4 v[2][U][2];
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u < n[p] ? j0 + u : n[p] - 1;
      const uint16_t* yr = a.Y + (size_t)__builtin_amdgcn_readlane(rs[p], j) * a.H;
#pragma unroll
      for (int h = 0; h < 2; ++h) v[p][u][h] = __builtin_nontemporal_load((const u32x4*)(yr + col[h]));
    }
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u;
      const float gj = j < n[p] ? __int_as_float(__builtin_amdgcn_readlane(gs[p], j)) : 0.f;
#pragma unroll
      for (int h = 0; h < 2; ++h) fma8(acc[p][h], gj, v[p][u][h]);
    }
}

// out[t, col0 : col0+ncols] for the tokens [t0, t0+ntok): wave w takes the
// token pairs w, w+4, ...; lane l owns columns 8l..8l+7 and 512+8l..512+8l+7.
__device__ void consume_task(const KArgs& a, int t0, int ntok, int col0, int ncols) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  int col[2];
  bool cok[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int c = 512 * h + 8 * lane;
    cok[h] = c < ncols;
    col[h] = col0 + (cok[h] ? c : 0);   // in-range address; the store is skipped
  }
  for (int pp = 2 * wave; pp < ntok; pp += 2 * nwaves) {
    int rs[2], gs[2], n[2], t[2];
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      t[p] = t0 + pp + p;
      n[p] = 0;
      rs[p] = 0;
      gs[p] = 0;
      if (pp + p < ntok) n[p] = token_rows(a, t[p], &rs[p], &gs[p]);
    }
    float acc[2][2][8];
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[p][h][i] = 0.f;
    // A token without rows borrows the other token's row list for its
    // loads, with all weights zero, so both tokens share one load stream.
    const int nl[2] = {n[0] > 0 ? n[0] : n[1], n[1] > 0 ? n[1] : n[0]};
    const int rl[2] = {n[0] > 0 ? rs[0] : rs[1], n[1] > 0 ? rs[1] : rs[0]};
    const int gl[2] = {n[0] > 0 ? gs[0] : 0, n[1] > 0 ? gs[1] : 0};
    const int nmax = nl[0] > nl[1] ? nl[0] : nl[1];
    for (int j0 = 0; j0 < nmax; j0 += 8) {
      const int left = nmax - j0;
      if (left <= 2)
        gather_step<2>(a, j0, rl, gl, nl, col, acc);
      else if (left <= 4)
        gather_step<4>(a, j0, rl, gl, nl, col, acc);
      else if (left <= 6)
        gather_step<6>(a, j0, rl, gl, nl, col, acc);
      else
        gather_step<8>(a, j0, rl, gl, nl, col, acc);
    }
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      if (pp + p >= ntok) continue;
      float* o = a.out + (size_t)t[p] * a.H;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        if (!cok[h]) continue;
        const f32x4 lo = {acc[p][h][0], acc[p][h][1], acc[p][h][2], acc[p][h][3]};
        const f32x4 hi = {acc[p][h][4], acc[p][h][5], acc[p][h][6], acc[p][h][7]};
        __builtin_nontemporal_store(lo, (f32x4*)(o + col[h]));
        __builtin_nontemporal_store(hi, (f32x4*)(o + col[h] + 4));
      }
    }
  }
}

__device__ void consumer_loop(Smem& sm, const KArgs& a, int cid, int ncons, long long W_comp) {
  if (!wait_flags(sm, a.wg_flags, gridDim.x, a)) return;
  const int total = a.L * a.tasks_per_split;
  u64* trace_tasks = a.trace ? a.trace + 4 * a.max_tiles : nullptr;
  int ready = -1;  // splits [0, ready] are known to be published
  for (int task = cid; task < total; task += ncons) {
    const int s = task / a.tasks_per_split;
    const int rem = task - s * a.tasks_per_split;
    const int tb = rem / a.cb_per_split;
    const int cb = rem - tb * a.cb_per_split;
    const u64 t_wait = now_100mhz();
    if (s > ready) {
      if (W_comp > 0 && !wait_flags(sm, a.tile_flags + (long long)s * W_comp, W_comp, a)) return;
      ready = s;
    }
    const u64 t_go = now_100mhz();
    const int t0 = tb * kCommTM;
    const int ntok = min(kCommTM, a.T - t0);
    const int col0 = s * a.nsplit + cb * a.comm_tn;
    const int ncols = min(a.comm_tn, (s + 1) * a.nsplit - col0);
    consume_task(a, t0, ntok, col0, ncols);
    if (trace_tasks) {
      __syncthreads();
      if (threadIdx.x == 0) {
        trace_tasks[4 * (long long)task + 0] = t_wait;
        trace_tasks[4 * (long long)task + 1] = t_go;
        trace_tasks[4 * (long long)task + 2] = now_100mhz();
        trace_tasks[4 * (long long)task + 3] = blockIdx.x;
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

__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
moe_gemm2_fused(KArgs a) {
  __shared__ Smem sm;
  load_experts(sm, a);
  const long long rows_dev = a.E > 0 ? (long long)sm.start[a.E - 1] + sm.count[a.E - 1] : 0;
  build_inverse(a, rows_dev);
  const long long m_tiles = sm.tile_prefix[a.E];
  const long long W_comp = m_tiles * a.ntps;

  const int b = blockIdx.x;
  if (b < a.C) {
    consumer_loop(sm, a, b, a.C, W_comp);
    return;
  }
  const int c = compute_index(b, a.C, (int)gridDim.x);
  const long long total = W_comp * a.L;
  if (total > a.max_tiles) {  // cannot happen with sanitized offsets; stay in bounds
    if (threadIdx.x == 0)
      __hip_atomic_fetch_or(a.status, kStBadRouting, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return;
  }
  for (long long g = c; g < total; g += a.P) {
    const int s = (int)(g / W_comp);
    const long long idx = g - (long long)s * W_comp;
    const int mt = (int)(idx / a.ntps);
    const int nt = (int)(idx - (long long)mt * a.ntps);
    // expert owning m-tile mt: last e with tile_prefix[e] <= mt
    int lo = 0, hi = a.E - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (sm.tile_prefix[mid] <= mt) lo = mid; else hi = mid - 1;
    }
    const int e = lo;
    const int r0 = sm.start[e] + (mt - sm.tile_prefix[e]) * kBM;
    const int rows_valid = min(kBM, sm.start[e] + sm.count[e] - r0);
    const int n0 = s * a.nsplit + nt * kBN;
    const int cols_valid = min(kBN, (s + 1) * a.nsplit - n0);
    const u64 t_start = now_100mhz();
    u64 t_mid[2];
    compute_tile(sm, a, e, r0, rows_valid, n0, cols_valid, t_mid);
    // publish: every wave's Y stores reach agent scope before the flag
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __syncthreads();
    if (threadIdx.x == 0) {
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      __hip_atomic_store(&a.tile_flags[g], a.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (a.trace) {
        a.trace[4 * g + 0] = t_start;
        a.trace[4 * g + 1] = t_mid[0];
        a.trace[4 * g + 2] = t_mid[1];
        a.trace[4 * g + 3] = now_100mhz();
      }
    }
  }
  if (a.drain) consumer_loop(sm, a, c, a.P, W_comp);
}

__global__ void fill_zero_kernel(uint32_t* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// ---- host side -----------------------------------------------------------------

struct Layout {
  size_t status, wg_flags, flags, tok_cnt, inv, Y, total;
  long long rows, max_tiles;
  int nsplit, ntps, comm_tn, cb_per_split, tasks_per_split;
};

inline size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

int check_shape(const moe_workload_t* wl) {
  if (!wl) return MOE_ERR_INVALID_ARG;
  if (wl->T < 0 || wl->H <= 0 || wl->I <= 0 || wl->E <= 0 || wl->topk <= 0 ||
      wl->splits <= 0 || wl->rows < 0)
    return MOE_ERR_INVALID_ARG;
  if (wl->E > kMaxE || wl->topk > kMaxTopk || wl->splits > kMaxSplits) return MOE_ERR_UNSUPPORTED;
  if (wl->I % 8 != 0 || wl->H % (8 * wl->splits) != 0) return MOE_ERR_UNSUPPORTED;
  const long long rows = wl->rows > 0 ? wl->rows : (long long)wl->T * wl->topk;
  if (rows > (long long)INT32_MAX || (long long)wl->T * wl->topk > (long long)INT32_MAX)
    return MOE_ERR_UNSUPPORTED;
  return MOE_OK;
}

bool make_layout(const moe_workload_t* wl, Layout* L) {
  if (check_shape(wl) != MOE_OK) return false;
  L->rows = wl->rows > 0 ? wl->rows : (long long)wl->T * wl->topk;
  L->nsplit = wl->H / wl->splits;
  L->ntps = (L->nsplit + kBN - 1) / kBN;
  L->comm_tn = L->nsplit < kCommTN ? L->nsplit : kCommTN;
  L->cb_per_split = (L->nsplit + L->comm_tn - 1) / L->comm_tn;
  L->tasks_per_split = ((wl->T + kCommTM - 1) / kCommTM) * L->cb_per_split;
  L->max_tiles = (long long)wl->splits * L->ntps * ((L->rows + kBM - 1) / kBM + wl->E);
  size_t off = 0;
  L->status = off;
  off += 256;
  L->wg_flags = off;
  off += (size_t)kMaxGrid * 4;
  L->flags = off;
  off = round_up(off + (size_t)L->max_tiles * 4, 256);
  L->tok_cnt = off;
  off = round_up(off + (size_t)wl->T * 8, 256);
  L->inv = off;
  off = round_up(off + (size_t)wl->T * wl->topk * 4, 256);
  L->Y = off;
  off = round_up(off + (size_t)L->rows * wl->H * 2, 256);
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
std::atomic<uint32_t> g_epoch{0};

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
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || occ <= 0) return MOE_ERR_HIP;
    g_dev[dev].cus = prop.multiProcessorCount;
    g_dev[dev].occ = occ;
    g_dev[dev].ready = true;
  }
  *out = g_dev[dev];
  return MOE_OK;
}

// rho_ref of the fused kernel on MI355X: mean consumer-task time over mean
// compute-tile time, measured with the traced entry point at the
// reference configuration below (T=16384, H=2048, I=704, E=32, top-6, L=2,
// C=32).  MOE_GEMM2_RHO_REF="num/den" overrides it.
constexpr int64_t kRhoRefNum = 4;
constexpr int64_t kRhoRefDen = 3;
constexpr int kDefaultFixedC = 8;

void fill_params(const DevInfo& d, moe_select_params_t* p) {
  p->tile_m = kBM;
  p->tile_n = kBN;
  p->comm_tile_m = kCommTM;
  p->comm_tile_n = kCommTN;
  p->occ_comp = d.occ;
  p->occ_comm = d.occ;
  p->num_cus = d.cus;
  p->c_min = 1;
  p->c_max = 64;
  p->groups = 1;
  p->rho_ref_num = kRhoRefNum;
  p->rho_ref_den = kRhoRefDen;
  if (const char* s = std::getenv("MOE_GEMM2_RHO_REF")) {
    long long n = 0, q = 0;
    if (std::sscanf(s, "%lld/%lld", &n, &q) == 2 && n > 0 && q > 0) {
      p->rho_ref_num = n;
      p->rho_ref_den = q;
    }
  }
  p->k_ref = 704;
  p->tile_m_ref = kBM;
  p->tile_n_ref = kBN;
  p->d_ref = 1;
}

inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

int launch(const void* x_perm, const void* w2, const int32_t* expert_offsets,
           const int32_t* token_ids, const float* gate_w, float* out, const moe_workload_t* wl,
           int32_t num_consumers, void* workspace, size_t workspace_bytes, void* stream,
           uint64_t* trace, size_t trace_bytes) {
  int st = check_shape(wl);
  if (st != MOE_OK) return st;
  Layout L;
  if (!make_layout(wl, &L)) return MOE_ERR_INVALID_ARG;
  if (!expert_offsets || !out || (L.rows > 0 && (!x_perm || !token_ids || !gate_w)) || !w2)
    return MOE_ERR_INVALID_ARG;
  if (!aligned(x_perm, 16) || !aligned(w2, 16) || !aligned(out, 16) ||
      !aligned(expert_offsets, 4) || !aligned(token_ids, 4) || !aligned(gate_w, 4))
    return MOE_ERR_ALIGNMENT;
  if (!workspace) return MOE_ERR_WORKSPACE;
  if (!aligned(workspace, 256)) return MOE_ERR_ALIGNMENT;
  if (workspace_bytes < L.total) return MOE_ERR_WORKSPACE;
  if (trace) {
    if (!aligned(trace, 8)) return MOE_ERR_ALIGNMENT;
    if (trace_bytes < moe_gemm2_trace_size(wl)) return MOE_ERR_INVALID_ARG;
  }
  if (wl->host_expert_counts) {
    long long sum = 0;
    for (int e = 0; e < wl->E; ++e) {
      if (wl->host_expert_counts[e] < 0) return MOE_ERR_INVALID_ARG;
      sum += wl->host_expert_counts[e];
    }
    if (sum != L.rows) return MOE_ERR_INVALID_ARG;
  }
  if (num_consumers < -1) return MOE_ERR_INVALID_ARG;

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
      fill_params(d, &p);
      moe_workload_t w = *wl;
      if (w.ranks <= 0) w.ranks = 1;
      moe_partition_t part;
      const int r = moe_select_partition(&w, &p, &part);
      if (r < 0) return r;
      C = part.C;
    }
  }
  int P, drain = 0;
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
  a.I = wl->I;
  a.E = wl->E;
  a.topk = wl->topk;
  a.L = wl->splits;
  a.nsplit = L.nsplit;
  a.ntps = L.ntps;
  a.C = C;
  a.P = P;
  a.drain = drain;
  a.comm_tn = L.comm_tn;
  a.cb_per_split = L.cb_per_split;
  a.tasks_per_split = L.tasks_per_split;
  uint32_t ep = g_epoch.fetch_add(1) + 1;
  if (ep == 0) ep = g_epoch.fetch_add(1) + 1;  // 0 is the cleared state
  a.epoch = ep;

  hipStream_t s = static_cast<hipStream_t>(stream);
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
  return (size_t)(4 * L.max_tiles + 4LL * wl->splits * L.tasks_per_split) * 8;
}

extern "C" int moe_gemm2_workspace_init(void* workspace, size_t workspace_bytes, void* stream) {
  if (!workspace || workspace_bytes == 0) return MOE_ERR_INVALID_ARG;
  if (!aligned(workspace, 256)) return MOE_ERR_ALIGNMENT;
  const size_t words = workspace_bytes / 4;
  const unsigned blocks = (unsigned)((words + 255) / 256 < 4096 ? (words + 255) / 256 : 4096);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks ? blocks : 1), dim3(256), 0,
                     static_cast<hipStream_t>(stream), static_cast<uint32_t*>(workspace), words);
  return hipGetLastError() == hipSuccess ? MOE_OK : MOE_ERR_HIP;
}

extern "C" int moe_gemm2_default_params(int device, moe_select_params_t* out) {
  if (!out) return MOE_ERR_INVALID_ARG;
  DevInfo d;
  const int st = device_info(device, &d);
  if (st != MOE_OK) return st;
  fill_params(d, out);
  return MOE_OK;
}

extern "C" int moe_gemm2_combine(const void* x_perm, const void* w2,
                                 const int32_t* expert_offsets, const int32_t* token_ids,
                                 const float* gate_w, float* out, const moe_workload_t* wl,
                                 int32_t num_consumers, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  return launch(x_perm, w2, expert_offsets, token_ids, gate_w, out, wl, num_consumers, workspace,
                workspace_bytes, stream, nullptr, 0);
}

extern "C" int moe_gemm2_combine_traced(const void* x_perm, const void* w2,
                                        const int32_t* expert_offsets, const int32_t* token_ids,
                                        const float* gate_w, float* out,
                                        const moe_workload_t* wl, int32_t num_consumers,
                                        void* workspace, size_t workspace_bytes, void* stream,
                                        uint64_t* trace, size_t trace_bytes) {
  if (!trace) return MOE_ERR_INVALID_ARG;
  return launch(x_perm, w2, expert_offsets, token_ids, gate_w, out, wl, num_consumers, workspace,
                workspace_bytes, stream, trace, trace_bytes);
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
