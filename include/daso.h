/*
 * daso.h - C ABI of the DASO parameter-synchronisation step on MI355X (gfx950).
 *
 * DASO (Distributed Asynchronous and Selective Optimization, arXiv 2104.05588)
 * synchronises data-parallel training in two levels.  Per GPU and per batch it
 * averages the gradients of the g GPUs of its node (Section 3, Figure 2), takes a
 * node-local optimizer step (Section 3.1; SGD with momentum in Section 4), and,
 * when the exchange with the other nodes lands S batches late, merges the P
 * received model states into the local one with the staleness-weighted average
 * of Eq. (1):
 *
 *        x  <-  ( 2S * x_local + sum_{i=1..P} x_i ) / ( 2S + P )
 *
 * Parameters travel as bfloat16 by default: they are cast while the send buffer
 * is packed and cast back on receipt (Section 3; Section 4 names bfloat16).
 * DASO_EXCHANGE_F32 and daso_global_merge_f32 cover an uncast fp32 exchange.
 *
 * This library runs that per-element arithmetic for one GPU's parameters, held
 * as flat buffers (all tensors of a model laid end to end) split into buckets,
 * contiguous element ranges that each carry their own staleness S.
 *
 * Arithmetic contract.  Every floating-point operation is one IEEE-754 binary32
 * operation rounded to nearest even, with no fused multiply-add, subnormals kept,
 * correctly rounded division, in this order per element j:
 *     s = G_0[j]; s = s + G_r[j] (r = 1..g-1);  gbar = s / g
 *     d = gbar                 (weight_decay == 0)
 *     d = gbar + weight_decay * x[j]     (otherwise)
 *     m' = mu * m[j] + d ;  xl = x[j] - lr * m'
 *     P == 0:  x' = xl
 *     P >  0, S > 0:  a = (2S) * xl ; a = a + widen(stale_i[j]) (i = 1..P) ; x' = a / (2S+P)
 *     P >  0, S = 0:  a = widen(stale_1[j]) ; a = a + widen(stale_i[j]) (i = 2..P) ; x' = a / P
 *              (the blocking average of the copies: the local state is left out,
 *              so a non-finite xl does not reach x')
 *     wire[j] = bf16_rne(x')   (or bf16_rne(xl) with DASO_PACK_PRE_MERGE)
 * widen(h) places the bf16 pattern h in the top half of a binary32 (exact); with
 * the fp32 exchange widen is the identity and the wire holds x' (or xl) itself.
 * bf16_rne rounds to nearest with ties to even; +-inf stay infinite, finite
 * values past the largest bfloat16 round to infinity, NaN becomes 0x7FC0.
 * Results are deterministic: the same inputs give the same bits on every call.
 *
 * Conventions for every entry point.
 *  - Buffers are device memory owned by the caller (the library allocates none of
 *    them).  fp32 buffers hold n floats, bf16 buffers hold n uint16 bit patterns.
 *  - Every device base pointer must be 16-byte aligned (DASO_EALIGN otherwise);
 *    128-byte alignment (what hipMalloc returns) lets every wavefront access
 *    whole cache lines and is the fast case.
 *  - Host pointer arrays (grads, stale) and bucket tables are read during the call
 *    only; the caller may free or reuse them as soon as the call returns.
 *  - Work is enqueued on `stream` (0 = the null stream) and runs asynchronously;
 *    no call synchronises the device or the stream.  The stream and every buffer
 *    must belong to the calling thread's current device (hipSetDevice); a stream
 *    of another device is rejected with DASO_EINVAL.
 *  - n == 0 is a valid no-op: once the counts and flags are checked the call
 *    returns DASO_OK without looking at any pointer or buffer (statistics
 *    included), so empty buffers may be NULL.
 *  - On an argument error (DASO_EINVAL, DASO_EALIGN, DASO_EALIAS) nothing is
 *    launched and the buffers are untouched; daso_status_string names the
 *    status.  A call may queue more than one kernel: one per 64 buckets of its
 *    table, and a statistics pass after each fused launch with statistics
 *    (except an eager launch of at most 64 tiles of daso_fused_sync_step,
 *    whose last workgroup sums its statistics itself; a call being captured
 *    into a graph keeps the pass, as daso_fused_sync_step_noalloc always
 *    does), and one zeroing kernel on the first eager call that uses a new
 *    statistics workspace.  If
 *    queueing one of them fails (DASO_EHIP), the kernels queued before it still
 *    run: the outputs (params, momentum, wire, grad_avg, stats) of the buckets
 *    they cover may then already be updated, the others are untouched.
 *  - Launch shape: the fused step hands each XCD runs of consecutive tiles
 *    (about 64 blocks of 8 runs per launch from 9 streams) and, from 10
 *    streams, lets at most 2 workgroups share a CU; both were measured best on
 *    MI355X (daso_fused_launch_config reports them).  For each shape of a
 *    single launch (up to 64 buckets), the 6 calls of daso_fused_sync_step
 *    after its first alternate between those runs and plain tile order,
 *    timed with events on the call's stream that later calls poll (never wait
 *    on); once all of them have completed (samples may be taken on different
 *    streams), plain order is kept for the shape if it was at least 1% faster,
 *    the runs otherwise.
 *    Captured calls take no samples, and polling is skipped while a HIP error
 *    is pending on the calling thread, so that error stays for the caller.
 *    The environment variables DASO_FUSED_RUN_ELEMS (elements per run, 0 =
 *    plain order; no sampling), DASO_FUSED_WG_PER_CU (0 = no cap) and
 *    DASO_FUSED_TUNE (0 = no sampling), read once per process, replace them to
 *    reproduce the measurements.  None of this ever changes a result.
 *  - Calls may be made from several host threads.  Fused steps with statistics
 *    share one small per-(device, stream) workspace (24 bytes per tile of 1024
 *    or 2048 parameters, plus a 260-byte table of bucket ranges) that the
 *    library allocates on first use (at least 1 MiB), replaces by a larger one
 *    when a larger call needs it, and never frees before the process ends;
 *    calls on one stream are ordered by that stream, and threads may share a
 *    stream (each call queues its kernels together).  A call that allocates
 *    cannot be captured into a HIP graph: make one call of the largest size on
 *    the capturing stream before capturing; captured calls then launch kernels
 *    only, and stay valid when later calls enlarge the workspace.  A captured
 *    call keeps the capturing stream's workspace: its replays must not overlap
 *    other calls on that stream, or each other.
 */
#ifndef DASO_H
#define DASO_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define DASO_OK 0
#define DASO_EINVAL (-1)  /* null required pointer, bad count (n outside [0, DASO_MAX_N], g or P out of range),
                             S outside [0, DASO_MAX_S], buckets not a tiling of [0,n),
                             a stream of another device */
#define DASO_EALIGN (-2)  /* a device base pointer is not 16-byte aligned */
#define DASO_EALIAS (-3)  /* an output overlaps an input other than in the allowed in-place pairs */
#define DASO_EHIP (-4)    /* a HIP call (launch, allocation of the stats workspace) failed */
#define DASO_ENOSPACE (-5) /* daso_fused_sync_step_noalloc: the statistics need more than
                              DASO_NOALLOC_SCRATCH_BYTES of scratch */

#define DASO_MAX_G 64     /* most replica gradients per call */
#define DASO_MAX_P 64     /* most exchanged copies per call */
#define DASO_MAX_S (1 << 20) /* largest staleness: 2S and 2S + P stay exact in binary32 */
#define DASO_MAX_N ((int64_t)1 << 56) /* most elements per call (far beyond any memory; keeps byte spans in 64 bits) */

/* flags of daso_sync_args */
#define DASO_PACK_PRE_MERGE 1u /* pack xl (after the optimizer step, before Eq. (1)) instead of x' */
#define DASO_EXCHANGE_F32 2u   /* fp32 exchange: copies arrive in stale_f32 and the wire is
                                  wire_f32, both binary32 (no cast; the non-blocking case of
                                  Section 3); stale and wire must then be NULL */

/* A bucket: elements [start, start + numel) merged with staleness S
 * (0 <= S <= DASO_MAX_S).
 * S is the number of batches the exchanged copies are late (Eq. (1)); S = 0
 * gives the plain average of the copies, as in blocking synchronisation. */
typedef struct daso_bucket {
  int64_t start;
  int64_t numel;
  int32_t S;
  int32_t reserved; /* must be 0 */
} daso_bucket;

/* Per-bucket side outputs of a fused step (not part of the paper's method):
 * grad_sq = sum of gbar^2, delta_sq = sum of (x' - xl)^2, both accumulated in
 * binary64 from the binary32 values; nonfinite = number of elements whose x' is
 * NaN or infinite.  The summation order is fixed, so the values are deterministic
 * but may differ from another order in the last bits. */
typedef struct daso_bucket_stats {
  double grad_sq;
  double delta_sq;
  uint64_t nonfinite;
} daso_bucket_stats;

/* Arguments of daso_fused_sync_step. */
typedef struct daso_sync_args {
  int64_t n;                       /* parameters on this GPU */
  int32_t g;                       /* replica gradients, 1..DASO_MAX_G */
  int32_t P;                       /* exchanged copies, 0..DASO_MAX_P */
  const float* const* grads;       /* host array of g device pointers, each n fp32; read only */
  const uint16_t* const* stale;    /* host array of P device pointers, each n bf16; read only
                                      (may be NULL when P == 0) */
  float* params;                   /* n fp32, read and overwritten with x' */
  float* momentum;                 /* n fp32, read and overwritten with m' */
  uint16_t* wire;                  /* n bf16 written, or NULL for no packing */
  float* grad_avg;                 /* n fp32 written with gbar, or NULL; may be exactly
                                      one of the grads buffers (Figure 2: every replica's
                                      gradients become the average) */
  const daso_bucket* buckets;      /* host array; the buckets must tile [0, n) */
  int32_t nbuckets;                /* >= 1 when n > 0 */
  float lr;                        /* learning rate */
  float mu;                        /* momentum factor */
  float weight_decay;              /* coupled L2 term; 0 skips it */
  uint32_t flags;                  /* DASO_PACK_PRE_MERGE | DASO_EXCHANGE_F32, or 0 */
  daso_bucket_stats* stats;        /* device array of nbuckets entries written, or NULL */
  const float* const* stale_f32;   /* with DASO_EXCHANGE_F32: host array of P device pointers,
                                      each n fp32; otherwise NULL */
  float* wire_f32;                 /* with DASO_EXCHANGE_F32: n fp32 written with x' (or xl), or
                                      NULL; otherwise NULL */
} daso_sync_args;

/* Local synchronisation (Section 3, Figure 2): out[j] = (sum_r grads[r][j]) / g,
 * summed in replica order.  grads: host array of g (1..DASO_MAX_G) device pointers
 * to n fp32 each.  out: n fp32; it may be exactly one of the grads buffers but
 * must not otherwise overlap them.  Reads 4g bytes and writes 4 bytes per element. */
int daso_local_avg(const float* const* grads, int32_t g, float* out, int64_t n,
                   hipStream_t stream);

/* Buffer packaging for the global exchange (Section 3; bfloat16 per Section 4):
 * wire[j] = bf16_rne(src[j]).  src: n fp32; wire: n uint16, must not overlap src. */
int daso_pack_bf16(const float* src, uint16_t* wire, int64_t n, hipStream_t stream);

/* Eq. (1), in place, bucket by bucket: params[j] <- (2S*params[j] + sum_i
 * widen(stale[i][j])) / (2S + P) with the S of the bucket holding j; P == 0
 * leaves params unchanged.  stale: host array of P (0..DASO_MAX_P) device
 * pointers to n bf16 each, none overlapping params.  buckets: host array of
 * nbuckets entries tiling [0, n).  wire: NULL, or n uint16 receiving
 * bf16_rne of the merged parameters (must not overlap any other buffer). */
int daso_global_merge(float* params, const uint16_t* const* stale, int32_t P,
                      const daso_bucket* buckets, int32_t nbuckets, uint16_t* wire,
                      int64_t n, hipStream_t stream);

/* Eq. (1) for the fp32 exchange (Section 3: a non-blocking exchange sends the
 * parameters uncast): as daso_global_merge, with P fp32 copies, and wire
 * (NULL, or n fp32) receiving the merged parameters. */
int daso_global_merge_f32(float* params, const float* const* stale, int32_t P,
                          const daso_bucket* buckets, int32_t nbuckets, float* wire,
                          int64_t n, hipStream_t stream);

/* One DASO synchronisation step for one GPU's parameters, in a single pass over
 * memory: local gradient average, SGD-momentum step, Eq. (1) merge per bucket,
 * bf16 pack and (optionally) the per-bucket statistics.  Aliasing rules: params
 * and momentum are updated in place and must not overlap each other or any other
 * buffer; wire, stats and grad_avg (apart from the allowed grads alias) must not
 * overlap anything else; inputs may overlap each other. */
int daso_fused_sync_step(const daso_sync_args* args, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): daso_fused_sync_step
 * with the same arguments, results and rules, except that the statistics
 * scratch (a 256-byte counter, 24 bytes per tile of 1024 or 2048 parameters and
 * a 260-byte table, per launch of up to 64 buckets) lives in a fixed array of
 * DASO_NOALLOC_SCRATCH_BYTES in device memory instead of an allocated
 * workspace.  The call never allocates or frees memory.  Every GPU the library
 * runs on holds its own copy of that array until the process ends; the first
 * call on a device looks up its address there (that device must be current, as
 * for every call).  All calls of this entry point on one GPU share the array and
 * each leaves its contents behind: calls queued on one stream are ordered by it
 * (host threads may share the stream), but calls on different streams of the
 * same GPU that may run at the same time race on the array and can give wrong
 * statistics; the other outputs are never affected.  A call whose statistics
 * need more than the array holds (more than 699,029 tiles in one launch: at
 * least about 715 million parameters) returns DASO_ENOSPACE and launches
 * nothing.  Without statistics (stats == NULL) no scratch is used. */
#define DASO_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
int daso_fused_sync_step_noalloc(const daso_sync_args* args, hipStream_t stream);

/* Launch shape of a fused step (host only, no device work), for tools that
 * time the same memory access pattern: daso_fused_sync_step and
 * daso_fused_sync_step_noalloc with these arguments run tiles of tile_elems
 * parameters, one 256-thread workgroup per tile, hand each XCD runs of
 * xcd_run_tiles consecutive tiles (1: plain order), and give each workgroup
 * lds_bytes of LDS (unused by the kernel; it caps how many workgroups share a
 * CU; 0: no cap).  ntiles counts the tiles of the first launch (the first 64
 * buckets).  Once the tile order of the shape has been chosen from its first
 * calls on the current device, xcd_run_tiles reports that choice.  The
 * arguments are checked as the step checks them and the same status is
 * returned; *out is written only on DASO_OK. */
typedef struct daso_launch_config {
  int64_t tile_elems;
  int64_t ntiles;
  int32_t xcd_run_tiles;
  int32_t lds_bytes;
} daso_launch_config;
int daso_fused_launch_config(const daso_sync_args* args, daso_launch_config* out);

/* Bucket plan for a flat parameter buffer (host only, no device work).  The
 * tensors of a model lie end to end in forward order with element counts
 * numels[0..ntensors).  Buckets are filled walking the tensors from the last to
 * the first, as gradients become ready in backpropagation, and a bucket closes
 * as soon as it holds at least cap_elems elements; what is left forms the last
 * bucket (tensor fusion / bucketing, Sections 2 and 4).  Bucket b of that walk
 * gets S = S_cycle[b % n_cycle].  Writes min(count, out_cap) buckets to out (out
 * may be NULL when out_cap == 0) and returns the bucket count, or DASO_EINVAL
 * for a negative element count, cap_elems < 1, n_cycle < 1, a negative S or a
 * null array that is needed.  Buckets never split a tensor. */
int32_t daso_plan_buckets(const int64_t* numels, int32_t ntensors, int64_t cap_elems,
                          const int32_t* S_cycle, int32_t n_cycle, daso_bucket* out, int32_t out_cap);

/* ------------------------------------------------------------------------
 * Phase and schedule controller (host only; Section 3).  Training runs for a
 * fixed number of epochs in three phases: warm-up and cool-down epochs use
 * blocking global synchronisation after every batch; the cycling phase in
 * between uses non-blocking synchronisation: a global exchange starts every B
 * batches and its copies are merged W batches later with S = W in Eq. (1).  B is
 * set by hand; W starts at a quarter of B.  Whenever the loss stops improving, B
 * and W are halved, never below 1; a further plateau with both at 1 restores
 * their starting values.  The groups (the GPUs with the same local rank on every
 * node) take turns at the exchange: exchange k is done by group k mod
 * group_count, whose member then hands the merged state to the other GPUs of its
 * node.
 *
 * Readings where the paper is silent: a plateau is `patience` consecutive
 * cycling epochs whose loss does not fall below best - plateau_rel_tol * |best|
 * (best: the last loss that did); after a change of B and W the count restarts;
 * the new values apply from the next epoch; in cycling, an exchange is started
 * only if its copies land no later than the last cycling batch and not in a
 * batch where another exchange's copies land; blocking exchanges also rotate
 * between groups; the first exchange of the cycling phase starts after its
 * B-th batch.
 */
#define DASO_PHASE_WARMUP 0
#define DASO_PHASE_CYCLING 1
#define DASO_PHASE_COOLDOWN 2

#define DASO_ACT_SEND 1u       /* after this batch's step, start a non-blocking exchange */
#define DASO_ACT_MERGE 2u      /* copies sent S batches ago arrived: merge them with S */
#define DASO_ACT_BLOCKING 4u   /* blocking exchange and plain average (S = 0) after this batch */
#define DASO_ACT_RECV_BCAST 8u /* take the merged state broadcast by this node's group member */

typedef struct daso_schedule_config {
  int32_t total_epochs;      /* >= 1 */
  int32_t warmup_epochs;     /* >= 0 */
  int32_t cooldown_epochs;   /* >= 0; warmup_epochs + cooldown_epochs <= total_epochs */
  int32_t batches_per_epoch; /* >= 1 */
  int32_t B_init;            /* >= 1: batches between exchanges when cycling starts */
  int32_t W_init;            /* 1..B_init, or 0 for max(1, B_init / 4) */
  int32_t group_count;       /* >= 1: GPUs per node */
  int32_t local_rank;        /* 0..group_count-1: this GPU's group */
  int32_t patience;          /* >= 1 */
  double plateau_rel_tol;    /* finite, >= 0 */
} daso_schedule_config;

/* What this GPU does around one batch. */
typedef struct daso_batch_plan {
  int64_t step;        /* batch index since the start of training */
  int32_t epoch;
  int32_t batch;       /* index within the epoch */
  int32_t phase;       /* DASO_PHASE_* */
  int32_t B;           /* current exchange period (cycling) */
  int32_t W;           /* current wait (cycling) */
  uint32_t actions;    /* DASO_ACT_* bits for this GPU; 0: local synchronisation and step only */
  int32_t S;           /* staleness for DASO_ACT_MERGE (or 0 with DASO_ACT_BLOCKING), else -1 */
  int32_t sync_group;  /* group whose exchange starts (or blocks) after this batch, or -1 */
  int32_t merge_group; /* group that merges arrived copies after this batch, or -1 */
} daso_batch_plan;

typedef struct daso_schedule daso_schedule; /* opaque, owned by the caller through create/destroy */

/* Create a controller; DASO_EINVAL for an invalid configuration.  A controller
 * keeps one GPU's state: calls on it from several threads need the caller's own
 * locking.  daso_schedule_destroy(NULL) does nothing. */
int daso_schedule_create(const daso_schedule_config* cfg, daso_schedule** out);
/* Plan of the next batch: returns 1 and fills *plan, 0 once training is over,
 * DASO_EINVAL if the previous epoch's loss has not been reported yet. */
int daso_schedule_next(daso_schedule* s, daso_batch_plan* plan);
/* Report the training loss of the epoch whose last batch was just planned
 * (DASO_EINVAL otherwise, or for a NaN loss). */
int daso_schedule_end_epoch(daso_schedule* s, double loss);
void daso_schedule_destroy(daso_schedule* s);

/* Static, NUL-terminated description of a status code. */
const char* daso_status_string(int status);

/* ABI version of this header (major * 100 + minor). */
int daso_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DASO_H */
