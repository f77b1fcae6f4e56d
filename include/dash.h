/*
 * dash.h -- C ABI of libdash: deterministic FlashAttention backward for
 * AMD Instinct MI355X (gfx950), with the dQ reduction order scheduled as in
 * "DASH: Deterministic Attention Scheduling for High-throughput Reproducible
 * LLM Training" (arXiv 2601.21824).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All tensor pointers are DEVICE pointers owned by the caller.  The library
 *    keeps no pointer after a call returns.
 *  - q, k, v, o, dO, dq, dk, dv: bf16 values (stored as uint16_t), layout
 *    [B][H][N][d], row-major and contiguous (one head = an N x d matrix).
 *  - lse: fp32 [B][H][N], the natural-log logsumexp of the scaled scores of
 *    each query row (the "logsumexp vector L" that Algorithm 1 takes as input).
 *  - Self-attention only: N queries attend to N keys.  With causal != 0,
 *    query i sees key j iff j <= i.
 *  - d must be 64, 128 or 256.  N >= 0 is arbitrary (ragged last tiles are masked);
 *    B, H >= 0, B*H*N < 2^30.  A problem with B*H*N == 0 is a successful no-op.
 *  - scale is the softmax scale s in S = s * Q K^T (the _ex and _noalloc
 *    forms take it, 0 selecting 1/sqrt(d); the others use 1/sqrt(d)).  dQ and
 *    dK include the factor s, dV does not.
 *  - Calls are asynchronous on the given HIP stream (hipStream_t passed as
 *    void*; NULL = the default stream) unless stated otherwise.
 *  - No C++ exception crosses this interface.  Every int-returning function
 *    returns a dash_status_t; on a non-OK return dash_last_error() gives a
 *    message (thread-local, valid until the next call from that thread).
 */
#ifndef DASH_H
#define DASH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Order in which the dQ partials of the KV tiles are summed (the schedule). */
typedef enum {
  /* fp32 hardware atomic adds, order = completion order: NOT deterministic.
     The conventional backward the paper starts from (Background section). */
  DASH_SCHED_ATOMIC = 0,
  /* every KV tile visits its Q tiles in ascending order; each dQ tile is summed
     in ascending KV order (the deterministic baseline, Section 3.2). */
  DASH_SCHED_NAIVE = 1,
  /* Descending Q-Tile Iteration (Section 3.3): Q tiles visited last to first,
     same ascending-KV summation order as NAIVE (so dQ is bitwise equal). */
  DASH_SCHED_DESCENDING = 2,
  /* Shift Scheduling (Section 3.4): the workgroup of KV tile j starts at a
     cyclically shifted Q tile; dQ summed in visiting order.  Full mask.  With
     a causal mask it selects Symmetric Shift. */
  DASH_SCHED_SHIFT = 3,
  /* Symmetric Shift (Section 3.4, causal masks): KV tiles j and T-1-j share a
     workgroup; two-phase fold.  Causal mask only. */
  DASH_SCHED_SYMSHIFT = 4,
  /* The deterministic schedule the DAG model of Section 3.1, calibrated on
     MI355X, predicts to be fastest for the call's (B, H, N, d, mask) on the
     current device: SHIFT, NAIVE or DESCENDING for a full mask, DESCENDING,
     NAIVE or SYMSHIFT for a causal mask (see dash_auto_schedule). */
  DASH_SCHED_AUTO = 5,
  /* Comparison point (related work, "Deterministic Implementations"): every
     KV tile stores its dQ partial in its own fp32 buffer, no ordering waits;
     a second kernel sums the partials of each dQ tile in ascending KV order.
     dQ is bitwise equal to NAIVE's; the workspace holds all T_c partials
     (dash_bwd_workspace_size grows by a factor T_c).  d = 64 and 128. */
  DASH_SCHED_PARTIALS = 6,
  /* Comparison point (the same related-work paragraph): two passes, no
     cross-workgroup reduction -- dK, dV with NAIVE's chains and no dQ work,
     then a Q-block-parallel dQ kernel that recomputes S and dP and reads K, V
     again.  d = 64 and 128. */
  DASH_SCHED_SPLIT = 7
} dash_schedule_t;

typedef enum {
  DASH_OK = 0,
  DASH_ERR_INVALID_ARG = -1, /* null pointer, negative size, d not 64/128/256, bad enum */
  DASH_ERR_UNSUPPORTED = -2, /* valid request the library cannot run (e.g. SYMSHIFT
                                with a full mask, too many KV tiles per head) */
  DASH_ERR_HIP = -3,         /* a HIP runtime call or kernel launch failed */
  DASH_ERR_TIMEOUT = -4,     /* an ordering wait exceeded its spin limit; outputs
                                of that call are undefined */
  DASH_ERR_NO_DEVICE = -5    /* no usable GPU */
} dash_status_t;

/* Debug / failure-injection flags of dash_bwd_options_t.flags */
#define DASH_FLAG_POISON_COUNTERS 1 /* start every ordering counter at a value no
                                       rank ever waits for: each wait times out
                                       (exercises the watchdog; kernels still exit) */

/* Optional knobs of dash_attn_bwd_ex.  Pass NULL for defaults. */
typedef struct {
  /* Polls an ordering wait makes before it gives up and flags a timeout
     (0 = default, about 2^24 polls).  The kernel always exits. */
  int spin_limit;
  /* DASH_FLAG_* bits */
  int flags;
  /* If non-NULL: int32 [B*H][ceil(N/64)][T_c], T_c = ceil(N/bc) KV tiles of
     bc rows (geometry[4] of dash_schedule_table for the call's B*H heads).  The workgroup that adds its partial to 64-row dQ
     block p with order position r writes its KV-tile index at [bh][p][r]
     (ordering witness). */
  int32_t* witness;
  /* If non-NULL: fp32 [B*H][T_c][N][d], T_c as above.  Each KV tile's
     unscaled dQ partial (its dS K for every query row) is written at [bh][j]. */
  float* partials;
  /* If non-NULL: fp32 [B*H][N][d].  Receives the final unscaled fp32 dQ sum
     (deterministic schedules only). */
  float* dq_accum;
  /* If both non-NULL: hipEvent_t handles (passed as void*) recorded on the
     call's stream immediately before and after the main backward kernel, so
     a caller can time that kernel alone. */
  void* event_main_begin;
  void* event_main_end;
  /* If > 0: at most this many persistent workgroups for the main kernel (0 =
     as many as the GPU keeps resident).  Shift needs at least the chains of
     one group (geometry[5] of dash_schedule_table), Symmetric Shift the
     chains of one head -- under XCD placement that many per XCD, i.e. times
     the number of XCDs -- else DASH_ERR_INVALID_ARG; naive, Descending and
     atomic run with any count (XCD placement: at least one per XCD).  The
     summation order -- hence every output bit -- does not depend on it. */
  int max_workgroups;
  /* Order in which the persistent workgroups take (head, chain) work items:
     DASH_TICKETS_AUTO (0, the measured faster order for the schedule and d),
     DASH_TICKETS_HEAD_MAJOR (1: all chains of a head in a row) or
     DASH_TICKETS_CHAIN_MAJOR (2: chain w of every head before chain w+1, i.e.
     the longest chains first under a causal mask; naive, Descending, atomic
     and the comparison variants only -- Shift and Symmetric Shift need the
     chains of a head together: DASH_ERR_INVALID_ARG).  The summation order --
     hence every output bit -- does not depend on it. */
  int ticket_order;
  /* Where the chains of a head run (see DASH_PLACEMENT_*).  0 = AUTO.  The
     placement can change Shift's summation order (its group size, geometry[5]
     of dash_schedule_table) when a head has more than 32 KV tiles; no other
     schedule's. */
  int placement;
  /* If non-NULL: device memory, 3 uint64 counters that the call adds to
     (zero them first).  Ordering-wait statistics of the main kernel:
     [0] wave-steps whose turn was not yet visible when the wave first looked
         (one step ahead) and that waited for it at the end of the step;
     [1] real-time clock ticks those waits took, counted from the moment the
         wave's own outstanding loads have landed (polls and sleeps only);
     [2] ticks of every wave's run, from its start to its exit.
     [1] / [2] is the share of wave time spent in the ordering wait.  The
     atomic and comparison variants leave the counters unchanged.  A wave
     keeps its counts in registers and adds them with three atomics when it
     exits (an instrumented kernel, otherwise instruction for instruction the
     production one); the results are the same bits. */
  unsigned long long* wait_stats;
} dash_bwd_options_t;

#define DASH_TICKETS_AUTO 0
#define DASH_TICKETS_HEAD_MAJOR 1
#define DASH_TICKETS_CHAIN_MAJOR 2

/* Placement of the work of a head.
   XCD: every chain of head bh runs on XCD (die) bh % n_xcd; each XCD takes
   work from its own ticket queue.  A Shift group is then at most 32 chains
   (what one XCD keeps resident), and a head's groups run one after another.
   The dQ accumulator is read and written device-coherently as under GLOBAL.
   Ordered schedules (naive, Descending, Shift, Symmetric Shift), when the
   chains that must run at once fit one XCD (Symmetric Shift: T_c <= 64);
   else DASH_ERR_UNSUPPORTED.
   GLOBAL: one ticket queue for the whole GPU (any schedule, any d).
   AUTO: GLOBAL (dash_bwd_placement reports it). */
#define DASH_PLACEMENT_AUTO 0
#define DASH_PLACEMENT_GLOBAL 1
#define DASH_PLACEMENT_XCD 2

/*
 * Forward attention producing O and L (Algorithm 1's inputs): O = softmax(s QK^T
 * + mask) V in bf16, lse = logsumexp per query row in fp32.  Deterministic.
 * Synchronous with respect to the host on the default stream is NOT implied:
 * the plain form runs on the default stream asynchronously.
 */
int dash_attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse,
                  int B, int H, int N, int d, int causal);
int dash_attn_fwd_ex(const void* q, const void* k, const void* v, void* o, float* lse,
                     int B, int H, int N, int d, int causal, float scale, void* stream);

/*
 * Attention backward (Algorithm 1): from Q, K, V, O, dO and L computes
 * D = rowsum(dO o O), then dQ, dK, dV.  Each KV tile's workgroup keeps dK_j,
 * dV_j on chip; the dQ partials are summed into an fp32 buffer in the order
 * fixed by `schedule`, serialized by per-Q-block counters (no atomics on the
 * data), except for DASH_SCHED_ATOMIC.
 *
 * The plain form uses a library-owned workspace on the current device (one
 * per device, grown on demand, freed by dash_release_workspace), runs on the
 * default stream and SYNCHRONIZES before returning so that it can report
 * DASH_ERR_TIMEOUT.  Calls from several host threads take turns on it.
 */
int dash_attn_bwd(const void* q, const void* k, const void* v, const void* o, const void* dO,
                  const float* lse, void* dq, void* dk, void* dv, int B, int H, int N, int d,
                  int causal, int schedule);

/* Bytes of device workspace dash_attn_bwd_ex needs for this problem and
   schedule, under either mask (0 if the arguments are invalid).  The same for
   every schedule except DASH_SCHED_PARTIALS, which needs room for all T_c dQ
   partials: a workspace of this size for any other schedule serves every
   schedule but PARTIALS, with a full or a causal mask. */
size_t dash_bwd_workspace_size(int B, int H, int N, int d, int schedule);

/*
 * Asynchronous backward on `stream` with a caller-provided device workspace of
 * ws_bytes >= dash_bwd_workspace_size(B,H,N,d,schedule) bytes (256-byte aligned).  The
 * workspace must not be used by another call until this one has finished.
 * A wait timeout is recorded in the workspace; read it with dash_bwd_check.
 * A call with no rows (B, H or N zero) computes nothing and may pass null
 * tensors and workspace; given a workspace, it only resets its error flag
 * (one lane of one workgroup on `stream`).
 * Shift and Symmetric Shift chains wait on each other in a cycle (Section
 * 3.1 assumes one KV tile per SM, all running at once): their main kernel is
 * launched cooperatively, so a grid the device cannot keep resident at once
 * (e.g. while other work occupies its CUs) is refused at launch with
 * DASH_ERR_UNSUPPORTED instead of spinning into the wait watchdog.  While one
 * process that has made cooperative launches is alive, the runtime refuses
 * another process's cooperative launch on the same GPU ("the operation cannot
 * be performed in the present state"): its Shift / Symmetric Shift calls fail
 * with DASH_ERR_HIP.  The other schedules wait only on chains that started
 * earlier and launch normally.
 */
int dash_attn_bwd_ex(const void* q, const void* k, const void* v, const void* o, const void* dO,
                     const float* lse, void* dq, void* dk, void* dv, int B, int H, int N, int d,
                     int causal, int schedule, float scale, void* workspace, size_t ws_bytes,
                     const dash_bwd_options_t* opts, void* stream);

/*
 * For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): the backward of
 * dash_attn_bwd_ex with default options, on a fixed workspace that the
 * library holds on every device it runs on -- a 256 MiB array in device
 * memory, present from the library's load until the process ends.  The call
 * allocates nothing (its first call on a device looks the array's address up
 * once).  Problems whose dash_bwd_workspace_size exceeds 256 MiB (e.g. more
 * than B*H*N*d = 64 Mi elements) are rejected with DASH_ERR_UNSUPPORTED.
 * Asynchronous on `stream`; every call on a device uses that device's one
 * array, so calls that overlap in time on one device (other streams, other
 * threads) race and must be serialized by the caller.  The kernels reset what
 * must start at zero themselves (no memset is recorded).  status: optional
 * caller-owned device int; the call sets it to 0, or to 1 if an ordering wait
 * timed out (outputs then undefined) -- read it once the stream has finished
 * the call; a call with no rows only sets it to 0.  Argument errors as
 * dash_attn_bwd_ex.
 */
int dash_attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* o, const void* dO,
                          const float* lse, void* dq, void* dk, void* dv, int B, int H, int N, int d, int causal,
                          int schedule, float scale, int* status, void* stream);

/* Synchronizes `stream`, then returns DASH_ERR_TIMEOUT if the last backward
   that used `workspace` hit a wait timeout, DASH_OK otherwise. */
int dash_bwd_check(void* workspace, void* stream);

/* The concrete schedule SHIFT resolves to for the mask (SYMSHIFT when
   causal); for DASH_SCHED_AUTO, which depends on B, H and N as well, the
   mask's default when no shape is known (SHIFT for a full mask, DESCENDING for
   a causal one; a backward call picks with dash_auto_schedule instead).
   Other schedules are returned unchanged. */
int dash_resolve_schedule(int schedule, int d, int causal);

/* DASH_SCHED_AUTO's choice for a backward of B x H heads of length N at head
   dim d (Section 3.1's DAG model).  Every candidate deterministic schedule is
   simulated as the kernels run it -- its chains of 64-row block steps in
   step-table order, tickets in the library's order, a free workgroup taking
   the next ticket, each block's reductions in its summation order -- with
   the block-step time measured for that schedule on MI355X at this (d, mask)
   and interpolated in N; the shortest predicted makespan wins (ties: SHIFT /
   DESCENDING).  Candidates whose co-running chains exceed the workgroups are
   left out.  `workers` is the number of resident workgroups (0: the current
   device's, which needs the device).  *schedule receives the choice and
   *predicted_ms (if not NULL) the predicted makespan in milliseconds (-1 when
   nothing was calibrated for this d and mask, or the problem is empty).  The
   first call for a shape simulates (enough heads to fill the workgroups three
   and six times, extrapolated, when the call has more; 0.1-1 s of host time
   at large N), later ones read a
   per-process cache of up to 4096 shapes (a full cache starts over; the
   choice is a pure function of the shape and the workgroup count). */
int dash_auto_schedule(int B, int H, int N, int d, int causal, int workers, int* schedule, double* predicted_ms);

/* Section 3.1's DAG model of a backward call with explicit costs: every block
   step (64 query rows against one KV tile, as the kernels step) computes for
   c and then reduces for r; a reduction starts once the block's previous
   contributor in the summation order has reduced.  `schedule` is NAIVE,
   DESCENDING, SHIFT or SYMSHIFT (SHIFT with causal != 0 is SYMSHIFT);
   ticket_order as in dash_bwd_options_t (AUTO: the library's order for
   `workers` resident workgroups).  max_heads = 0 simulates all B*H heads
   (host time grows with B*H*N^2); with max_heads > 0 and B*H > 2 * max_heads
   it simulates max_heads and 2 * max_heads heads and extrapolates linearly
   in the number of heads (dash_auto_schedule uses max_heads =
   ceil(3 * workers / chains per head)).  *makespan receives the critical
   path in the units of c and r.  DASH_ERR_UNSUPPORTED when chains that must
   run together exceed `workers` (no chain can finish); no device needed. */
int dash_model_makespan(int schedule, int B, int H, int N, int d, int causal, int workers, int ticket_order,
                        int max_heads, double c, double r, double* makespan);

/* The placement (DASH_PLACEMENT_GLOBAL or DASH_PLACEMENT_XCD) that
   dash_attn_bwd_ex picks with placement AUTO for this problem on the current
   device, or a negative dash_status_t.  Needs the device (queries it once). */
int dash_bwd_placement(int B, int H, int N, int d, int causal, int schedule);

/* Measured bf16 dense MFMA throughput of the current device, the measured
   counterpart of the published 2.5 PFLOP/s in the main kernel's roofline.
   Two workgroups of 4 waves per CU each run `iters` rounds of 8 independent
   v_mfma_f32_32x32x16_bf16 chains on register operands (iters = 0: 20000,
   about 4 ms); *tflops receives the best of 3 event-timed launches in
   TFLOP/s.  Synchronous; allocates and frees a small device buffer and its
   own stream.  DASH_ERR_INVALID_ARG for a NULL tflops or iters < 0. */
int dash_mfma_peak(int iters, double* tflops);

/*
 * Host-side view of the schedule the kernels follow (no GPU needed).  For one
 * head of length N at head dim d, in a call of `heads` = B*H heads: T_r
 * scheduling Q tiles of br rows and T_c KV tiles of bc rows (bc = 128 at
 * d = 128 and 64 at d = 256; at d = 64, 256 when the call has at least 256 KV
 * tiles of 256 rows over all heads (causal: 512 and N >= 1024), else 128 --
 * so the summation order depends on the call's number of heads at d = 64),
 * under `placement` (DASH_PLACEMENT_GLOBAL or DASH_PLACEMENT_XCD; only
 * Shift's groups depend on it).  Writes, when the pointer is non-NULL:
 *   geometry[6]            = {T_r, T_c, br, number of workgroup chains per
 *                             head, bc, chains per Shift group (the chains
 *                             that must run at the same time; = chains for
 *                             the other schedules)}
 *   chain_len[w]           = tasks of workgroup w
 *   task_kv[w*cap + t], task_q[w*cap + t] = the t-th task of workgroup w,
 *                            cap = max chain length = geometry-dependent
 *                            (use T_r + 1)
 *   rank[i*T_c + j]        = position of KV tile j in Q tile i's summation
 *                            order (-1 when they do not interact)
 * Returns a dash_status_t.
 */
int dash_schedule_table(int schedule, int heads, int N, int d, int causal, int placement, int* geometry, int* chain_len,
                        int* task_kv, int* task_q, int* rank);

const char* dash_last_error(void);
/* Frees the library-owned workspaces of dash_attn_bwd on every device (the
   next call reallocates on its device). */
void dash_release_workspace(void);

#ifdef __cplusplus
}
#endif
#endif /* DASH_H */
