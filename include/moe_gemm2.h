/*
 * moe_gemm2.h - C ABI of the MI355X MoE down-projection + combine stage and
 * its launch-time partition selector.
 *
 * The operation (paper: Background, "Distributed MoE Execution", third step;
 * Method, "System Integration and Correctness"):
 *
 *   Y[r, :]   = x_perm[r, :] @ W2[e(r)]      e(r): expert_offsets[e] <= r < expert_offsets[e+1]
 *   out[t, :] = sum over rows r with token_ids[r] == t of gate_w[r] * Y[r, :]
 *
 * computed by one persistent kernel whose workgroups take one of two roles:
 * compute workgroups run the grouped GEMM tile by tile and publish their
 * tiles with per-tile readiness flags (one release per workgroup and split,
 * after its last tile of the split); consumer workgroups (or, with C = 0,
 * every workgroup once its tiles are done) claim tasks in order, wait until
 * the task's split is published and then gather each token's
 * rows, weight them by the gates and write the token's output once.  The
 * number of consumer workgroups C is the paper's decision variable; the
 * selector below evaluates its wave-quantized makespan model (Method,
 * "Wave-Quantized Pipeline Model" and Algorithm 1) to choose it.
 *
 * Conventions for every function:
 *   - all functions are extern "C"; none throws, aborts or prints;
 *   - a negative return value is a moe_status_t error; 0 or a documented
 *     non-negative value is success;
 *   - device pointers are plain HIP device addresses; the caller allocates
 *     and owns every buffer, including the workspace; the library allocates
 *     no device memory;
 *   - "stream" is a hipStream_t passed as void* (NULL = the null stream);
 *     calls that take one only enqueue work on it and return without
 *     synchronising, except moe_gemm2_status;
 *   - tensors are dense and row-major.
 */
#ifndef MOE_GEMM2_H
#define MOE_GEMM2_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MOE_OK = 0,
  MOE_ERR_INVALID_ARG = -1,        /* null pointer, bad dimension or bad parameter */
  MOE_ERR_ALIGNMENT = -2,          /* a pointer is not aligned as documented */
  MOE_ERR_WORKSPACE = -3,          /* workspace missing or smaller than moe_gemm2_workspace_size */
  MOE_ERR_NO_LEGAL_PARTITION = -4, /* no C in [c_min, c_max] leaves P(C) > 0 */
  MOE_ERR_HIP = -5,                /* a HIP runtime call failed (no device, launch error, ...) */
  MOE_ERR_TIMEOUT = -6,            /* a consumer's bounded wait expired (reported by moe_gemm2_status) */
  MOE_ERR_UNSUPPORTED = -7,        /* shape outside what the kernel handles (see moe_gemm2_combine) */
  MOE_ERR_BAD_ROUTING = -8         /* device saw a token id outside [0,T), a token with more than
                                      topk rows, or offsets that are not a non-decreasing prefix
                                      of [0, rows] (reported by moe_gemm2_status) */
} moe_status_t;

/* One invocation's workload (paper: Table "Workload and tile notation").
 *   T      tokens before top-k expansion (M; one GPU, so D = 1 and M/D = T)
 *   H      hidden size = GEMM2 output width (N)
 *   I      local expert intermediate size = GEMM2 reduction length (K)
 *   E      local experts
 *   topk   maximum routed rows per token (k)
 *   splits pipeline splits along H (L), >= 1
 *   ranks  participating ranks (D) for the service-rate scaling; 1 on one GPU
 *   rows   permuted rows = expert_offsets[E]; 0 means T * topk
 *   host_expert_counts  optional host array [E] of routed rows per expert
 *          (M_e); NULL makes the selector use the even-load estimate. */
typedef struct {
  int32_t T, H, I, E, topk, splits, ranks;
  int64_t rows;
  const int32_t* host_expert_counts;
} moe_workload_t;

/* Kernel and GPU residency facts the selector needs (paper: Table "Resource
 * notation"; Method, "Launch-Time Analytical Selection"), plus the
 * service-time ratio rho_ref measured once at a reference configuration
 * (eq:rho-reference) and that configuration (eq:rho-config). */
typedef struct {
  int32_t tile_m, tile_n;            /* compute tile T_M^comp x T_N^comp */
  int32_t comm_tile_m, comm_tile_n;  /* consumer task tile T_M^comm x T_N^comm */
  int32_t occ_comp, occ_comm;        /* resident workgroups per CU of each role */
  int32_t num_cus;                   /* G */
  int32_t c_min, c_max;              /* legal candidates, eq:c-domain; c_min = 0 adds the
                                        role-switch candidate (see moe_select_partition) */
  int32_t groups;                    /* g, input groups (1) */
  int64_t rho_ref_num, rho_ref_den;  /* rho_ref as a positive rational */
  int32_t k_ref, tile_m_ref, tile_n_ref, d_ref;
  int32_t split_axis;                /* 0: the L splits cut the output columns N (the paper);
                                        1: they cut the routed rows (token bands, see
                                        moe_gemm2_combine_ex mode 2) */
  int32_t drain;                     /* 0: the paper's recurrence; 1: compute slots join the
                                        consumers after their tiles (the last split is served
                                        by all C + P slots); 2: they serve whatever remains of
                                        every split (the work-conserving drain) */
  int32_t rho_kh;                    /* 0: eq:rho-scaling as printed; 1: also scale rho by the
                                        consumer task's bytes relative to the calibration:
                                        (2 topk + 4) / (2 topk_ref + 4) for the Y rows read
                                        (bf16) and the output written (fp32) per token, and
                                        the task width over comm_tile_n_ref */
  int32_t topk_ref, comm_tile_n_ref; /* top-k and task width at the calibration (used with
                                        rho_kh = 1) */
  int32_t readiness;                 /* 0: consumer work becomes ready a split at a time (the
                                        paper); 1: a compute wave at a time (consumer tasks
                                        that each need one compute tile, the atomic scatter) */
  int32_t comm_tile_m_last;          /* tokens of the last split's consumer tasks (T_M^last);
                                        0 or comm_tile_m: as the other splits' (the paper).
                                        Column splits with readiness = 0 only */
  int64_t split_cost_num, split_cost_den; /* pi_ref >= 0: compute waves (at the reference K and
                                        tile, scaled as rho's first two factors) by which each
                                        split's publish delays the compute of the splits
                                        after it; split_cost_num = 0: none (the paper).
                                        readiness = 0 only */
} moe_select_params_t;

/* The chosen partition.  T(C) = T_num / T_den in compute-wave units; W_comp
 * and W_comm are the per-split work counts (eq:compute-work,
 * eq:communication-work); delta_comp is eq:tie-breaker. */
typedef struct {
  int32_t C, R, P, delta_comp;
  int64_t T_num, T_den;
  int64_t W_comp, W_comm;
} moe_partition_t;

/* Algorithm 1: for C = c_min..c_max compute R(C) = ceil(C/o_comm)
 * (eq:reservation), P(C) = o_comp (G - R(C)) (eq:compute-capacity), the split
 * readiness times A_s (eq:split-arrival), V_comm (eq:communication-waves),
 * q = rho V_comm (eq:comm-service) with rho from eq:rho-scaling, and the
 * completion recurrence F_s (eq:split-finish); return the C with the least
 * T(C) = F_{L-1} (eq:makespan), ties to the least Delta_comp
 * (eq:tie-breaker), then to the least C.  Candidates with P(C) <= 0 are
 * illegal.  Arithmetic is exact (rational rho, integer time).
 * Extension beyond the paper's legal set {1..C_max}: with c_min = 0 the
 * candidate C = 0 is also evaluated, the role switch where all
 * P0 = o_comp G slots run every compute tile and then all serve the consumer
 * tasks: T(0) = ceil(L W_comp / P0) + rho ceil(L W_comm / P0), R = 0, P = P0,
 * Delta = ceil(W_comp/P0) P0 - W_comp.
 * Extensions selected by the parameters (both 0 gives the paper's model):
 *   split_axis = 1 (token bands): per-split work
 *     W_comp = ceil(g sum_e ceil(M_e/T_M) / L) ceil(N/T_N),
 *     W_comm = ceil(ceil(ceil(M/D)/T_M^comm) / L) ceil(N/T_N^comm);
 *   drain = 1: the last split's service uses every slot,
 *     F_{L-1} = max(A_{L-1}, F_{L-2}) + rho ceil(W_comm / (C + P));
 *   drain = 2 (readiness = 0, comm_tile_m_last = comm_tile_m or 0): every
 *     slot serves what remains of every split once the compute ends at
 *     E = A_{L-1}.  Until then the C consumers take the splits in order,
 *     split s from start = max(A_s, the end of split s-1), in rounds of C
 *     tasks of rho each; the rounds begun before E claim
 *     min(W_comm, C ceil((E - start)/rho)) tasks of it, stopping at the first
 *     split they do not wholly claim.  The Idle = V P - L W_comp compute
 *     slots without a tile in the last compute wave (V = ceil(L W_comp / P))
 *     are free from E - 1: in their ceil(1/rho) rounds begun before E they
 *     claim up to Idle ceil(1/rho) of the unclaimed tasks of the splits
 *     with A_s <= E - 1 (s < L - 1), ending at E - 1 + rho ceil(taken/Idle).
 *     With R the tasks left of all L W_comm and e the end of the last
 *     claimed round, T(C) = max(E + rho ceil(R / (C + P)), e); C = 0 is the
 *     same with no consumers and P = P0.  F_s is the end of split s where
 *     the consumers finished it before E, else T(C);
 *   split_cost = pi_ref > 0 (readiness = 0): pi = pi_ref (K_ref/K)
 *     (T_M,ref T_N,ref)/(T_M T_N) compute waves per split boundary, so
 *     A_s = ceil((s+1) W_comp / P) + s pi (and for C = 0 the end of the
 *     compute is ceil(L W_comp / P0) + (L-1) pi); T_den is then the least
 *     common multiple of rho's denominator and pi's;
 *   readiness = 1 (column splits only): the consumer work is released
 *     a compute wave at a time instead of a split at a time.  The L W_comp
 *     tiles complete in V = ceil(L W_comp / P) waves, wave v (1-based) the
 *     tiles [(v-1) P, min(v P, L W_comp)); it releases
 *     w_v = ceil(t_v L W_comm / (L W_comp)) - ceil(t_{v-1} L W_comm / (L W_comp))
 *     tasks, t_v = min(v P, L W_comp), and
 *     F_v = max(v, F_{v-1}) + rho ceil(w_v / C), T(C) = F_V (with drain = 1
 *     the last wave's tasks are served by C + P slots); C = 0 is unchanged;
 *     a candidate with V > 2^20 is an error (MOE_ERR_INVALID_ARG);
 *   rho_kh = 1: rho of eq:rho-scaling times
 *     (2 topk + 4) / (2 topk_ref + 4) * w / comm_tile_n_ref, with the task
 *     width w = min(comm_tile_n, ceil(N/L)) (column splits) or
 *     min(comm_tile_n, N) (token bands); topk_ref, comm_tile_n_ref > 0;
 *   comm_tile_m_last = T_M^last > 0 (column splits, readiness = 0): the last
 *     split's tasks hold T_M^last tokens:
 *     W_last = ceil(ceil(M/D)/T_M^last) ceil(ceil(N/L)/T_N^comm) tasks of
 *     rho_last = rho T_M^last / T_M^comm, the last split served as
 *     F_{L-1} = max(A_{L-1}, F_{L-2}) + rho_last ceil(W_last / C) (drain:
 *     C + P slots), and with a : b = T_M^comm : T_M^last in lowest terms
 *     T(0) = ceil(L W_comp / P0) + (rho/a) ceil((a (L-1) W_comm + b W_last) / P0);
 *     T_den is then rho's denominator times a / gcd(rho's numerator, a).
 * Pure host code: no HIP call, no allocation, thread-safe.
 * Since P(C) does not grow with C, the candidates past the first illegal
 * C >= 1 are not evaluated (any c_max up to INT32_MAX costs no more than the
 * legal range).
 * Returns C* >= c_min and fills *out when out != NULL; MOE_ERR_INVALID_ARG for a
 * null wl/p, non-positive dimensions or parameters, o_comp G > INT32_MAX,
 * more than 2^20 splits, a negative host count or arithmetic overflow;
 * MOE_ERR_NO_LEGAL_PARTITION when no candidate is legal. */
int moe_select_partition(const moe_workload_t* wl, const moe_select_params_t* p,
                         moe_partition_t* out);

/* L as a second decision variable (Method, eq:split-arrival and
 * eq:split-finish take L as given; here it is chosen as well): for every
 * L = l_min..l_max, moe_select_partition on the workload with splits = L;
 * returns the C of the (L, C) pair with the least T(C), ties to the least L
 * (fewer publishes), and writes that L to *splits_out and its partition to
 * *out (each when non-NULL).  wl->splits is ignored.  The caller keeps L
 * within what the launch accepts (column splits: H % (8 L) == 0; token
 * bands: (E + 1) L <= 2048).  Returns C >= 0, MOE_ERR_INVALID_ARG
 * (l_min < 1, l_max < l_min, l_max > 1024, or as moe_select_partition) or
 * MOE_ERR_NO_LEGAL_PARTITION. */
int moe_select_partition_splits(const moe_workload_t* wl, const moe_select_params_t* p,
                                int32_t l_min, int32_t l_max, moe_partition_t* out,
                                int32_t* splits_out);

/* The model's internals for one candidate C, for checking the model against
 * measured traces: rho = *rho_num / *rho_den after eq:rho-scaling (and the
 * extensions the parameters select), and the split arrival and finish
 * times A_s and F_s (eq:split-arrival, eq:split-finish) in units of
 * 1 / *rho_den compute waves, written to A_out[s] and F_out[s] for s < L;
 * for C = 0 (the role switch) one entry each, the end of all tiles and the
 * end of all tasks; with readiness = 1 one entry per compute wave (V of
 * them, as in moe_select_partition).  rho_num, rho_den, A_out and F_out may each be NULL;
 * n is the capacity of A_out and F_out (at least the number of entries
 * when either is given).  Pure host code.  Returns the number of entries
 * (L; 1 for C = 0; V with readiness = 1), MOE_ERR_INVALID_ARG (as
 * moe_select_partition, C < 0, or n too small) or
 * MOE_ERR_NO_LEGAL_PARTITION when P(C) <= 0. */
int moe_select_candidate(const moe_workload_t* wl, const moe_select_params_t* p, int32_t C,
                         int64_t* rho_num, int64_t* rho_den, int64_t* A_out, int64_t* F_out,
                         int32_t n);

/* The whole T(C) table of the same model: T_num_out[i] is the numerator of
 * T(c_min + i) over the common denominator *T_den_out, or -1 where P <= 0.
 * n must be >= c_max - c_min + 1.  Returns the number of entries written, or
 * a negative status as moe_select_partition does. */
int moe_select_evaluate(const moe_workload_t* wl, const moe_select_params_t* p,
                        int64_t* T_num_out, int32_t n, int64_t* T_den_out);

/* Parameters for the fused kernel on a HIP device: its tile shapes (the
 * owner-write consumer task at its full size of 64 tokens x 1024 columns,
 * the last split's at 16 tokens: comm_tile_m_last = 16),
 * its occupancy from hipOccupancyMaxActiveBlocksPerMultiprocessor (capped
 * by its LDS and register budget), the device's CU count, the candidate set
 * C = 0..64 (C = 0 is the role switch, a legal launch of this kernel; 64
 * is where the kernel's launch time reaches its plateau in C, eq:c-domain) and
 * the MI355X calibration of rho_ref.  Device facts are cached
 * on first use (Method, "System Integration and Correctness").  Returns 0 or
 * MOE_ERR_HIP / MOE_ERR_INVALID_ARG. */
int moe_gemm2_default_params(int device, moe_select_params_t* out);

/* The same for a consumer mode (see moe_gemm2_combine_ex): mode 0 gives
 * what moe_gemm2_default_params gives; mode 1 (atomic scatter, one consumer
 * task per compute tile) sets the consumer tile to
 * max(1, tile_m / topk) tokens x tile_n columns, so that W_comm counts
 * about one task per compute tile, and rho_ref to that mode's calibration
 * (MOE_GEMM2_RHO_REF_SCATTER="num/den" overrides it) and readiness = 1 (a
 * scatter task waits only for the published prefix of the tile sequence up
 * to its own tile); mode 2 (token bands)
 * sets split_axis = 1, drain = 2, rho_ref to that mode's calibration
 * (MOE_GEMM2_RHO_REF_BANDS overrides it) and the split cost pi_ref = 43/100
 * (split_cost_num / split_cost_den).  Modes 0 and 1 leave split_axis, drain
 * and the split cost 0.  Every mode sets topk_ref = 6 and comm_tile_n_ref = 1024 (the
 * calibration's) and rho_kh = 0; modes 0 and 2 set rho_kh = 1 when the
 * environment sets MOE_GEMM2_RHO_KH=1.  Returns 0 or MOE_ERR_HIP / MOE_ERR_INVALID_ARG (also for a
 * mode other than 0, 1 or 2 or topk <= 0). */
int moe_gemm2_default_params_ex(int device, int32_t mode, int32_t topk, moe_select_params_t* out);

/* The parameters a launch of this workload hands to the selector (what
 * num_consumers = -1 uses).  Mode 0: an owner-write task is TM tokens x
 * min(1024, H/splits) columns, where TM = 64, halved down to 16 while the
 * launch would have fewer than 512 tasks (splits * ceil(T/TM) *
 * ceil(H/splits/1024)), so that a small batch's combine still spreads over
 * every CU; comm_tile_m = TM and rho_ref, calibrated for 64-token tasks, is
 * scaled by TM/64 (a task's bytes are proportional to its tokens); the last
 * split's tasks take TM_last = max(16, TM/4) tokens (at most TM), so that
 * the launch ends evenly over the CUs: comm_tile_m_last = TM_last.  Mode 1:
 * as moe_gemm2_default_params_ex(device, 1, wl->topk).  Mode 2: tasks of
 * TM tokens x min(1024, H) columns of the full width, TM = 64 halved down
 * to 16 while there would be fewer than 512 (ceil(T/TM) ceil(H/1024)),
 * rho_ref scaled by TM/64, split_axis = 1, drain = 2, and the split cost
 * pi_ref = 43/100 (split_cost_num / split_cost_den; 0 in modes 0 and 1).
 * Returns 0,
 * MOE_ERR_INVALID_ARG (null pointer, mode other than 0, 1 or 2, invalid
 * workload), MOE_ERR_UNSUPPORTED (shape outside moe_gemm2_combine_ex's
 * range for that mode) or MOE_ERR_HIP. */
int moe_gemm2_launch_params(int device, int32_t mode, const moe_workload_t* wl,
                            moe_select_params_t* out);

/* Bytes of workspace moe_gemm2_combine needs for this workload (flags,
 * counters, the token->rows inverse map and the bf16 staging of Y).
 * Returns 0 for an invalid workload. */
size_t moe_gemm2_workspace_size(const moe_workload_t* wl);

/* Prepare a workspace (required once after allocating it, before its first
 * use): zero it and give it a launch epoch no earlier initialisation in
 * this process used, so that readiness flags left in that memory by an
 * earlier user can never read as published.  Enqueued on stream.  Returns
 * 0 or MOE_ERR_HIP / MOE_ERR_INVALID_ARG. */
int moe_gemm2_workspace_init(void* workspace, size_t workspace_bytes, void* stream);

/* The stage.
 *   x_perm          device bf16 [rows, I], rows grouped by expert (16-byte aligned)
 *   w2              device bf16 [E, I, H], H contiguous (16-byte aligned)
 *   expert_offsets  device int32 [E+1]: 0 = offsets[0] <= ... <= offsets[E] = rows
 *   token_ids       device int32 [rows]: token of each permuted row, in [0, T);
 *                   a token may own at most topk rows (fewer is allowed: dropped slots)
 *   gate_w          device fp32 [rows]: gate weight of each permuted row
 *   out             device fp32 [T, H] (16-byte aligned): fully overwritten
 *                   (tokens without rows get zeros); never read
 *   wl              dimensions (+ optional host counts for the selector)
 *   num_consumers   >= 1: that many consumer workgroups (an explicit choice
 *                   wins, Method "System Integration and Correctness");
 *                   0: no dedicated consumers, every workgroup computes its
 *                   tiles and then takes consumer tasks;
 *                   -1: chosen by moe_select_partition with
 *                   moe_gemm2_launch_params(device, 0, wl), unless the
 *                   environment sets
 *                   MOE_GEMM2_SELECTOR=0, which restores a fixed C = 8
 *   workspace       device memory of at least moe_gemm2_workspace_size(wl)
 *                   bytes, 256-byte aligned, zeroed once by
 *                   moe_gemm2_workspace_init; calls that may overlap in
 *                   time need distinct workspaces.  The workspace keeps a
 *                   launch epoch that each launch advances on the device,
 *                   so a call captured in a HIP graph may be replayed
 *                   (with wl->host_expert_counts NULL the call reads
 *                   nothing from the device on the host).  A workspace may
 *                   serve workloads of different dimensions in turn: the
 *                   library remembers the layout each workspace address was
 *                   last launched with and, when it changes, zeroes the
 *                   workspace's metadata (the bytes before the Y staging)
 *                   with a small kernel on stream before the launch (also
 *                   inside a captured graph, where it then runs on every
 *                   replay)
 *   stream          hipStream_t the kernel is enqueued on
 * Supported shapes: H % (8 * splits) == 0, I % 8 == 0, 1 <= E <= 1024,
 * 1 <= topk <= 64, splits <= 16, 2 I H < 2^31 (one expert's W2 slice
 * within 2 GiB) (else MOE_ERR_UNSUPPORTED).
 * Values inside device arrays are checked by the kernel, which skips bad
 * entries and records MOE_ERR_BAD_ROUTING for moe_gemm2_status.
 * Launches on other streams may share the GPU: compute workgroups never
 * wait while they hold tiles, with C = 0 a workgroup waits on other
 * workgroups' tiles only once its whole grid has started, and dedicated
 * consumers (C >= 1) wait only on compute workgroups, which never wait; so
 * concurrent launches drain as long as their dedicated consumers together
 * leave a CU free.  Every wait is bounded (MOE_GEMM2_SPIN_LIMIT polls, then
 * MOE_ERR_TIMEOUT).  Debugging aid: MOE_GEMM2_DEBUG_PUBLISH_DELAY="m:t"
 * makes the compute workgroups whose index is a multiple of m hold each
 * split publish back by t ticks of the 100 MHz clock (t <= 10^6).
 * Returns the number of consumer workgroups launched (>= 0) or a negative
 * status (host-side validation and launch errors only). */
int moe_gemm2_combine(const void* x_perm, const void* w2, const int32_t* expert_offsets,
                      const int32_t* token_ids, const float* gate_w, float* out,
                      const moe_workload_t* wl, int32_t num_consumers,
                      void* workspace, size_t workspace_bytes, void* stream);

/* Same as moe_gemm2_combine, and also records timestamps (the device's
 * constant 100 MHz clock) into trace (device, 8-byte aligned, at least
 * moe_gemm2_trace_size(wl) bytes).  Layout, uint64 words: for each compute
 * tile g of the global sequence, words 4g..4g+3 = start, end of the
 * reduction loop, end of the Y stores, end of the tile (after the split's
 * publish for a workgroup's last tile of a split); then, from word
 * 4 * max_tiles (max_tiles = splits * ceil(ceil(H/splits)/256) *
 * (ceil(rows/256) + E)), for each consumer task j, words 4j..4j+3 = wait
 * start, wait end, finish, workgroup id (task j: split
 * s = min(j / tasks_per_split, splits - 1), task i = j - s tasks_per_split of
 * that split, token block and column block from i, with tasks_per_split =
 * ceil(T/TM) * ceil(H/splits/1024); the last split has
 * ceil(T/TM_last) * ceil(H/splits/1024) tasks; TM and TM_last are the
 * comm_tile_m and comm_tile_m_last that moe_gemm2_launch_params gives).  The
 * arithmetic and the result are identical to the untraced call. */
int moe_gemm2_combine_traced(const void* x_perm, const void* w2, const int32_t* expert_offsets,
                             const int32_t* token_ids, const float* gate_w, float* out,
                             const moe_workload_t* wl, int32_t num_consumers,
                             void* workspace, size_t workspace_bytes, void* stream,
                             uint64_t* trace, size_t trace_bytes);

/* The stage with a choice of consumer (Method, "System Integration and
 * Correctness": the paper's consumers write each token's output once; a
 * scatter of fp32 atomic additions is the other way to combine):
 *   mode 0  owner-write, exactly as moe_gemm2_combine (deterministic: the
 *           result does not depend on C or on timing);
 *   mode 1  atomic scatter: the kernel first zeroes out (each workgroup its
 *           share, published like the inverse map of mode 0), then a
 *           consumer task is one published compute tile (it waits for the
 *           published prefix of the tile sequence up to that tile, i.e. for
 *           the compute wave that holds it, not for the whole split), whose
 *           rows r it adds, weighted by gate_w[r], into out[token_ids[r], :] with
 *           fp32 atomic additions at device scope.  The order of the
 *           additions varies from run to run, so the result does too, by
 *           rounding only.  Rows with an out-of-range token id are skipped
 *           and flagged; the topk bound per token is not checked (every
 *           in-range row is added);
 *   mode 2  owner-write over token bands: the wl->splits = L pipeline
 *           splits cut the routed rows instead of the columns.  Expert
 *           e's n_e = ceil(M_e/256) m-tiles are cut into L runs, band b
 *           holding m-tiles [b n_e / L, (b+1) n_e / L) over the full width
 *           H; tiles run band -> expert -> m-tile -> n-tile.  A consumer
 *           task (TM tokens x min(1024, H) columns, one counter over all
 *           tasks) waits until every tile of the bands up to the last band
 *           holding one of its rows is published (an agent-scope acquire
 *           for the inverse map and one per newly published band prefix),
 *           and compute workgroups always join the consumers after their
 *           tiles.  The
 *           result is bitwise that of mode 0 (same per-token order).  Any
 *           L >= 1 with (E + 1) L <= 2048 (else MOE_ERR_UNSUPPORTED); H % 8
 *           == 0 suffices (modes 0 and 1 need H % (8 L) == 0).
 * trace: NULL, or a buffer as for moe_gemm2_combine_traced (in mode 1 the
 * consumer-task words hold one record per compute tile of the global
 * sequence; in mode 2 record j is task j of the single task sequence).
 * With num_consumers = -1 the selector runs with
 * moe_gemm2_launch_params(device, mode, wl).  Everything else is as
 * for moe_gemm2_combine; MOE_ERR_INVALID_ARG for a mode other than 0, 1
 * or 2. */
int moe_gemm2_combine_ex(const void* x_perm, const void* w2, const int32_t* expert_offsets,
                         const int32_t* token_ids, const float* gate_w, float* out,
                         const moe_workload_t* wl, int32_t num_consumers, int32_t mode,
                         void* workspace, size_t workspace_bytes, void* stream,
                         uint64_t* trace, size_t trace_bytes);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the stage
 * exactly as moe_gemm2_combine_ex with no trace, but its workspace is the
 * library's own scratch, a static device array of
 * MOE_GEMM2_NOALLOC_SCRATCH_BYTES that every GPU the library runs on holds
 * until the process ends (each GPU its own copy, looked up on the first call
 * on that device).  The call allocates nothing: no hipMalloc, hipFree or
 * allocating library routine, on the host or the device.  The caller still
 * passes inputs and outputs (same meaning, layout and alignment as for
 * moe_gemm2_combine_ex).
 *   - Workloads whose moe_gemm2_workspace_size exceeds
 *     MOE_GEMM2_NOALLOC_SCRATCH_BYTES are rejected with MOE_ERR_WORKSPACE
 *     before anything is enqueued.
 *   - Every call on a GPU shares that GPU's scratch, which keeps the last
 *     call's contents: the first call on a device, and any call whose
 *     workload has another layout than the previous call's, first zeroes
 *     the scratch's metadata with a small kernel on stream.  Calls that may
 *     overlap in time on one GPU (other streams, other threads) race on it
 *     and must not be issued.
 *   - The device status word (MOE_ERR_TIMEOUT, MOE_ERR_BAD_ROUTING) lives
 *     in the scratch and is not reported; bad routing entries are skipped
 *     and waits are bounded as for moe_gemm2_combine.
 * Returns the number of consumer workgroups launched (>= 0) or a negative
 * status as moe_gemm2_combine_ex does. */
#define MOE_GEMM2_NOALLOC_SCRATCH_BYTES (96u << 20)
int moe_gemm2_combine_noalloc(const void* x_perm, const void* w2, const int32_t* expert_offsets,
                              const int32_t* token_ids, const float* gate_w, float* out,
                              const moe_workload_t* wl, int32_t num_consumers, int32_t mode,
                              void* stream);

/* Bytes the trace buffer needs for this workload (0 for an invalid one):
 * 4 * max_tiles words for the compute tiles, then 4 words for each of
 * max((splits - 1) * tasks_per_split + last split's tasks, band tasks,
 * max_tiles) consumer tasks
 * (tasks_per_split as for moe_gemm2_combine_traced, band tasks as for
 * moe_gemm2_combine_ex mode 2); max_tiles = splits * ceil(ceil(H/splits)/256)
 * * (ceil(rows/256) + E). */
size_t moe_gemm2_trace_size(const moe_workload_t* wl);

/* ---- The rest of the post-router layer on one GPU: the up-projection.
 * Paper: Background, "Distributed MoE Execution" (the grouped GEMM1 with
 * the gate and up projections and the gated activation that feed GEMM2).
 * It is not what the paper's method changes; it is here so that the whole
 * layer after the router runs on the device and the down-projection stage's
 * share of it can be measured.
 *
 *   h_r          = hidden[token_ids[r], :]                  (the dispatch gather)
 *   x_perm[r, c] = silu(h_r . Wg[e(r)][:, c]) * (h_r . Wu[e(r)][:, c]),
 *   silu(z)      = z / (1 + exp(-z)),   c < I,
 *
 * products in bf16 with fp32 accumulation, the activation in fp32, x_perm
 * rounded once to bf16 (round to nearest even). */

/* Repacks the up-projection weights for moe_gemm1_swiglu:
 *   w_gate_up   device bf16 [E, H, 2I]: columns 0..I-1 the gate projection
 *               Wg[e], columns I..2I-1 the up projection Wu[e] (each row k
 *               of length 2I is the k-th input feature's weights)
 *   w1_packed   device bf16 [E, H, 2I], a different buffer: column 32b + j
 *               holds gate column 16b + j and column 32b + 16 + j up column
 *               16b + j (j < 16), so each 32-column block carries the gate
 *               and up weights of 16 outputs
 * Enqueued on stream.  I % 16 == 0 (else MOE_ERR_UNSUPPORTED); E, H, I > 0
 * and distinct non-null buffers (else MOE_ERR_INVALID_ARG); 2-byte aligned
 * (else MOE_ERR_ALIGNMENT).  Returns 0 or MOE_ERR_HIP. */
int moe_gemm1_pack_weights(const void* w_gate_up, void* w1_packed, int32_t E, int32_t H,
                           int32_t I, void* stream);

/* The up-projection: x_perm from hidden, as above, for the rows grouped by
 * expert exactly as for moe_gemm2_combine.
 *   hidden          device bf16 [T, H] (16-byte aligned)
 *   w1              device bf16 [E, H, 2I], packed by moe_gemm1_pack_weights
 *                   (16-byte aligned)
 *   expert_offsets  device int32 [E+1], as for moe_gemm2_combine
 *   token_ids       device int32 [rows]: the token of each permuted row; an id
 *                   outside [0, T) is replaced by 0 and flagged
 *                   (MOE_ERR_BAD_ROUTING from moe_gemm2_status)
 *   x_perm          device bf16 [rows, I] (16-byte aligned), fully written for
 *                   every row inside the expert ranges
 *   wl              T, H, I, E, topk, rows as for moe_gemm2_combine (splits,
 *                   ranks and host counts are not used, except that host
 *                   counts, when given, must sum to rows)
 *   workspace       a moe_gemm2 workspace (at least 512 bytes, 256-byte
 *                   aligned, zeroed once by moe_gemm2_workspace_init): only
 *                   its status word is used
 * One persistent launch, every workgroup computing 256 x 256 tiles of the
 * packed columns.  Supported: H % 8 == 0, I % 16 == 0, 1 <= E <= 1024,
 * 1 <= topk <= 64, 2 T H < 2^31 and 4 H I < 2^31 (hidden and one expert's
 * W1 slice within 2 GiB) (else MOE_ERR_UNSUPPORTED).  Returns 0 or a negative
 * status (host-side validation and launch errors). */
int moe_gemm1_swiglu(const void* hidden, const void* w1, const int32_t* expert_offsets,
                     const int32_t* token_ids, void* x_perm, const moe_workload_t* wl,
                     void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of workspace moe_layer_forward needs: a moe_gemm2 workspace followed
 * by x_perm.  0 for an invalid or unsupported workload. */
size_t moe_layer_workspace_size(const moe_workload_t* wl);

/* The post-router layer: moe_gemm1_swiglu into the workspace's x_perm, then
 * moe_gemm2_combine on it (same stream, two launches).  Arguments as for
 * those two functions; workspace of at least moe_layer_workspace_size(wl)
 * bytes, 256-byte aligned, zeroed once by moe_gemm2_workspace_init.  Shapes
 * must satisfy both functions' limits.  Returns the number of consumer
 * workgroups of the second launch (>= 0) or a negative status. */
int moe_layer_forward(const void* hidden, const void* w1, const void* w2,
                      const int32_t* expert_offsets, const int32_t* token_ids,
                      const float* gate_w, float* out, const moe_workload_t* wl,
                      int32_t num_consumers, void* workspace, size_t workspace_bytes,
                      void* stream);

/* Synchronises stream, then reports the device-side status of the last
 * launches that used this workspace: 0, MOE_ERR_TIMEOUT or
 * MOE_ERR_BAD_ROUTING (or MOE_ERR_HIP).  clear != 0 resets it. */
int moe_gemm2_status(void* workspace, void* stream, int clear);

/* Static description of an error code. */
const char* moe_strerror(int status);

/* ABI version of this header (major * 100 + minor): 108. */
int moe_gemm2_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* MOE_GEMM2_H */
