/*
 * fgd.h -- C ABI of the fused Factored Gossip DiLoCo outer-step engine for
 * AMD MI355X (gfx950).
 *
 * The engine runs the outer synchronization step of Factored Gossip DiLoCo
 * over M simulated worker replicas that live in one GPU's memory
 * (Sec. 4.1, factored outer step; Appendix A, Algorithm 1, outer-step part):
 *
 *   g0_m    = theta_prev_m - theta_local_m        outer gradient; the paper's
 *                                                 Delta = y_H - y_0 enters the
 *                                                 outer optimizer negated
 *   ghat    = Mix2(g0)                            K2 gossip rounds (blocking mix)
 *   x       = Mix1(theta_prev)                    K1 rounds or the global mean
 *                                                 (non-blocking mix)
 *   v'_m    = mu v_m + ghat_m                     Nesterov, two-line form
 *   theta'_m = x_m - lr (ghat_m + mu v'_m)        (Appendix B)
 *
 * Variants set at creation or by a call: plain momentum (theta'_m = x_m -
 * lr v'_m), Mix1 applied to the momentum before its update (Appendix B,
 * GlobalM1S: the outer optimizer state is averaged as part of Mix1), and
 * Mix2 restricted to a subset of the parameters (Sec. 4.1 and Appendix C,
 * the Mix2-subset configuration: identity outside the subset).
 *
 * A Mix round maps row m to sum_n w_{m,n} u_n (Sec. 3, gossip mixing
 * operator), with W given as CSR: row m lists the workers it pulls from.
 * The step optionally reports, per worker, S_m(u) = sum_p (u_m,p - mean_n
 * u_n,p)^2 for every intermediate u (Sec. 4.4 L2 consensus distance; the
 * mean of sqrt(S_m) is the Sec. 4.4 form and the mean of S_m the
 * Appendix D.1 form).
 *
 * Conventions for every call:
 *  - Every call returns an fgd_status.  Nothing throws or aborts across the
 *    ABI.  fgd_last_error() (per thread) then holds a readable reason.  An
 *    argument, state or support error is found before any kernel is
 *    launched (a topology upload may already be enqueued; it writes no
 *    caller buffer).  FGD_ERR_HIP can come from a runtime call after part of
 *    the work was enqueued (the outputs are then unspecified).
 *  - Device arrays are worker-major [M][ld] with ld >= P elements; element p
 *    of worker m is at index m * ld + p.  Each row must start on a 16-byte
 *    boundary (base pointer 16-byte aligned and ld * element size a multiple
 *    of 16).
 *  - The caller owns every device buffer; the engine only borrows them for
 *    the work it enqueues, so they must stay alive until `stream` has passed
 *    that work.  Host arrays handed to the engine are copied before return.
 *  - `stream` is a hipStream_t (NULL = the device's null stream).  Compute
 *    calls are asynchronous with respect to the host.
 *  - An engine is not thread-safe; use one engine per host thread.
 *  - One engine's work on different streams: fgd_outer_step,
 *    fgd_outer_step_blocking and fgd_consensus_distance share the engine's
 *    consensus scratch, so no two of them may run at the same time; two
 *    fgd_mix1 launches share the Mix1 half's own counter and scratch, so they
 *    may not either; one fgd_mix1 may overlap one of the others.  Calls on
 *    one stream are ordered by the stream.
 *  - The engine's compute calls are not meant to be recorded by HIP stream
 *    capture: a topology upload copies from a pinned host staging slot that
 *    later uploads reuse, after waiting on the slot's event from the host.
 *    fgd_js_distance, fgd_stream_js_pattern and fgd_stream_copy enqueue
 *    kernels only.
 *  - Engine calls run on the engine's device (fgd_config.device): they make
 *    it current for their duration and restore the caller's current device
 *    before returning.  The engine-free calls (fgd_js_distance,
 *    fgd_stream_js_pattern, fgd_stream_copy) run on the caller's current
 *    device.
 */
#ifndef FGD_H
#define FGD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct fgd_engine fgd_engine; /* opaque */

typedef enum {
    FGD_OK = 0,
    FGD_ERR_INVALID_ARG = 1,   /* bad pointer, size, alignment, enum or alias */
    FGD_ERR_TOPOLOGY = 2,      /* malformed CSR or masks, or W not doubly stochastic */
    FGD_ERR_UNSUPPORTED = 3,   /* valid request the library does not implement */
    FGD_ERR_OUT_OF_MEMORY = 4, /* host or device allocation failed */
    FGD_ERR_HIP = 5,           /* a HIP runtime call or launch failed */
    FGD_ERR_STATE = 6          /* call not allowed in the engine's current state */
} fgd_status;

typedef enum { FGD_F32 = 0, FGD_BF16 = 1 } fgd_dtype;

/* Which Mix slot a topology call sets. */
typedef enum { FGD_MIX1 = 1, FGD_MIX2 = 2 } fgd_mix;

/* How a Mix slot mixes. */
typedef enum {
    FGD_W_IDENTITY = 0,    /* no mixing */
    FGD_W_GLOBAL_MEAN = 1, /* exact mean over all workers, W = 11^T / M (Sec. 3) */
    FGD_W_CSR = 2          /* num_rounds rounds of a sparse W given in CSR */
} fgd_wkind;

/* How the weights of a CSR round are obtained from the structure, the given
 * weights and that round's edge mask.  A dropped link mixes less rather than
 * aborting the round (Sec. 1 and Sec. 5.2 describe this behaviour of gossip
 * under transient failures; the reweighting rules are this engine's). */
typedef enum {
    FGD_REWEIGHT_NONE = 0,       /* given weights; masks must be NULL or all ones */
    FGD_REWEIGHT_METROPOLIS = 1, /* live graph of the round: d_i = live neighbours of i,
                                    w_ij = 1/(1+max(d_i,d_j)), w_ii = 1 - sum_j w_ij
                                    (ascending j), computed in double, rounded to
                                    float; given weights are ignored (may be NULL) */
    FGD_REWEIGHT_SELF = 2        /* given weights; a dropped entry's weight is added to
                                    its row's diagonal (double, ascending j, rounded) */
} fgd_reweight;

#define FGD_MAX_WORKERS 64          /* largest M the library runs */
#define FGD_MAX_ROUNDS 8            /* largest number of rounds per Mix slot */
#define FGD_MAX_SUBSET_SEGMENTS 4096 /* largest number of Mix2 subset segments */

typedef struct {
    uint32_t struct_size; /* sizeof(fgd_config), checked for equality */
    int32_t num_workers;  /* M, 1..FGD_MAX_WORKERS */
    int64_t num_params;   /* P >= 0 parameters per worker */
    int64_t ld;           /* row stride in elements, >= P, ld * elem size % 16 == 0 */
    int32_t param_dtype;  /* fgd_dtype of theta_prev and theta_local (arithmetic is
                             float32) */
    int32_t state_dtype;  /* fgd_dtype of the momentum: FGD_F32 only (else
                             FGD_ERR_UNSUPPORTED) */
    float outer_lr;       /* lr (gamma), e.g. 0.7 (Sec. 5, Appendix A) */
    float momentum;       /* mu, e.g. 0.9 */
    int32_t nesterov;     /* 1: Nesterov (Appendix B two-line form), 0: plain momentum,
                             theta' = x - lr v' */
    int32_t device;       /* HIP device ordinal; -1 creates a host-only engine that
                             validates topologies but cannot run compute calls */
    int32_t mix1_state;   /* 1: Mix1 is also applied to the momentum before the momentum
                             update (Appendix B, GlobalM1S); 0: momentum stays per worker */
    int32_t reserved;     /* must be 0 */
} fgd_config;

/* Creates an engine.  Allocates the device-side topology slots and the
 * consensus-distance scratch on cfg->device (never later, inside a step).
 * Both Mix slots start unset. */
fgd_status fgd_create(const fgd_config *cfg, fgd_engine **out);

/* Frees the engine and its device memory after synchronizing its device.
 * NULL is accepted. */
fgd_status fgd_destroy(fgd_engine *e);

/* Sets the topology of one Mix slot.
 *   kind        fgd_wkind.  IDENTITY and GLOBAL_MEAN ignore every array
 *               argument and num_rounds.
 *   row_ptr     host int32[M+1]: row_ptr[0] = 0, non-decreasing, row_ptr[M] = nnz
 *   col_idx     host int32[nnz]: strictly ascending within each row, in [0, M),
 *               with the diagonal entry present in every row
 *   weights     host float[nnz] >= 0, finite; NULL only with METROPOLIS
 *   num_rounds  K in [0, FGD_MAX_ROUNDS]; 0 makes the slot the identity
 *   edge_masks  host uint8[K][nnz] with values 0/1, NULL = every entry live.
 *               Diagonal entries must be live.  On a structurally symmetric
 *               graph, entry (i,j) and entry (j,i) must carry the same mask.
 *   reweight    fgd_reweight
 * Per round the engine forms the effective weights, checks that every row
 * and every column of the effective W sums to 1 within 1e-6 (else
 * FGD_ERR_TOPOLOGY; METROPOLIS also needs a structurally symmetric graph),
 * and keeps them.  They are uploaded, stream-ordered, by the next
 * fgd_outer_step.  Host arrays are copied before return. */
fgd_status fgd_set_topology(fgd_engine *e, int32_t which, int32_t kind, const int32_t *row_ptr,
                            const int32_t *col_idx, const float *weights, int32_t num_rounds,
                            const uint8_t *edge_masks, int32_t reweight);

/* Restricts Mix2 to a subset of the parameters (the Mix2-subset
 * configuration of Sec. 4.1 and Appendix C, where the subset is a set of
 * parameter blocks): Mix2 acts on every index inside one of the segments
 * and is the identity elsewhere, in every round.
 *   segments      host int64[num_segments][2] of half-open ranges [begin, end):
 *                 0 <= begin < end <= P, ascending and disjoint (touching is
 *                 allowed)
 *   num_segments  0 .. FGD_MAX_SUBSET_SEGMENTS; 0 removes the restriction
 *                 (Mix2 acts everywhere); segments may then be NULL
 * Takes effect, stream-ordered, at the next fgd_outer_step.  A step with a
 * subset needs a CSR Mix2 (else FGD_ERR_UNSUPPORTED).  The consensus rows of
 * the Mix2 rounds cover every parameter: inside the subset the mixed values,
 * outside it g^0.  Host arrays are copied before return. */
fgd_status fgd_set_mix2_subset(fgd_engine *e, const int64_t *segments, int32_t num_segments);

/* Number of consensus-distance rows fgd_outer_step writes:
 * (K2 + 1) + (K1 + 1) + 1, where a GLOBAL_MEAN slot counts as one round and
 * IDENTITY as zero.  Needs both slots set. */
fgd_status fgd_num_cd_rows(const fgd_engine *e, int32_t *n_rows);

/* One fused outer step, enqueued on `stream`.
 *   theta_prev   device [M][ld] param_dtype, read and overwritten with theta'
 *   theta_local  device [M][ld] param_dtype, read only; must not overlap
 *                theta_prev or momentum
 *   momentum     device [M][ld] float32, read and overwritten with v'
 *   cd_out       device double[n_rows][M] or NULL (no consensus distances).
 *                Rows in order: g^0..g^K2 (Mix2 input and round outputs),
 *                x^0..x^K1 (Mix1 input and round outputs), then the stored
 *                theta'.  Entry [r][m] is S_m of that intermediate.
 * Arithmetic is float32 (bf16 storage is widened exactly; theta' is rounded
 * to bf16 to nearest even); consensus sums accumulate in double.  Both Mix
 * slots must be set (else FGD_ERR_STATE).  Elements of a row at indices
 * [P, ld) may be read but are never written. */
fgd_status fgd_outer_step(fgd_engine *e, void *theta_prev, const void *theta_local, float *momentum,
                          double *cd_out, void *stream);

/* Split execution of a round (Appendix A, Algorithm 1): the non-blocking
 * Mix1 is launched at the start of the round, typically on its own stream so
 * that it overlaps the inner steps, and the blocking Mix2 and the outer
 * optimizer run at the end of the round from the Mix1 output it stored.
 * Compared with fgd_outer_step this moves M * P * 3 * elem_size more bytes
 * (x written and read back, theta_prev read twice); the two halves give the
 * same result as the fused step up to the rounding of x to the storage type.
 * The caller orders the halves: the blocking half must not start before the
 * Mix1 half of the same round is complete, and the next Mix1 half must not
 * start before the blocking half that produced its theta_prev. */

/* Mix1 half: x_out = Mix1(theta_prev), rounded to the storage type.
 *   theta_prev  device [M][ld] param_dtype, read
 *   x_out       device [M][ld] param_dtype, written; must not overlap theta_prev
 *   momentum    device [M][ld] float32: with mix1_state it is replaced by
 *               Mix1(momentum) (the state is mixed here, not in the blocking
 *               half); otherwise ignored and may be NULL
 *   cd_out      device double[K1 + 1][M] or NULL: rows x^0..x^K1 (consensus
 *               of the unrounded Mix1 intermediates)
 *   num_blocks  0: one block per compute unit; n > 0: at most n blocks, so
 *               that a Mix1 overlapping other kernels occupies fewer CUs.
 *               Blocks take chunks of the parameter range from a counter, so
 *               an uneven placement next to other kernels balances itself;
 *               the result does not depend on num_blocks.
 * Enqueued on `stream`.  Two Mix1 launches of one engine must not overlap
 * (they share the engine's counter and consensus scratch). */
fgd_status fgd_mix1(fgd_engine *e, const void *theta_prev, void *x_out, float *momentum, double *cd_out,
                    int32_t num_blocks, void *stream);

/* Blocking half: g0 = theta_prev - theta_local, ghat = Mix2(g0) (on the
 * subset if one is set), v' = mu v + ghat, theta' = x - lr (ghat + mu v')
 * (plain momentum: x - lr v'), with x read from the array fgd_mix1 stored.
 *   x            device [M][ld] param_dtype, read
 *   theta_prev   device [M][ld] param_dtype, read and overwritten with theta'
 *   theta_local  device [M][ld] param_dtype, read; with write_local = 1 it
 *                also receives theta' as stored (the next round's inner
 *                starting point, y_0 = z)
 *   momentum     device [M][ld] float32, read and overwritten with v'
 *   cd_out       device double[K2 + 2][M] or NULL: rows g^0..g^K2 and the
 *                stored theta'
 * No two arrays may overlap.  Enqueued on `stream`. */
fgd_status fgd_outer_step_blocking(fgd_engine *e, const void *x, void *theta_prev, void *theta_local, float *momentum,
                                   double *cd_out, int32_t write_local, void *stream);

/* Which kernel fgd_outer_step launches for the engine's current topology.
 *   FGD_STEP_LANE_PER_PARAM  a lane holds V consecutive parameters of every
 *                            worker (any M, every Mix kind and variant)
 *   FGD_STEP_WORKER_GROUPS   64 workers: a lane holds 16 workers x 4
 *                            parameters; chosen for a CSR Mix2 of at most 4
 *                            rounds with a CSR (at most 2 rounds) or global
 *                            Mix1, rows of at most 15 live entries, tables
 *                            that fit in 80 KiB of LDS with the rows, no
 *                            subset and no state mixing
 * Both compute the same step to the same bars.  Needs both slots set. */
#define FGD_STEP_LANE_PER_PARAM 0
#define FGD_STEP_WORKER_GROUPS 1
fgd_status fgd_step_variant(const fgd_engine *e, int32_t *variant);

/* Consensus rows of the two halves: K1 + 1 and K2 + 2 (GLOBAL_MEAN counts as
 * one round, IDENTITY as zero).  Needs both slots set. */
fgd_status fgd_num_cd_rows_split(const fgd_engine *e, int32_t *mix1_rows, int32_t *blocking_rows);

/* Algorithmic minimum HBM traffic of the two halves:
 *   Mix1 half      M * P * (2 * elem_size + (mix1_state ? 8 : 0))
 *   blocking half  M * P * (4 * elem_size + 8 + (write_local ? elem_size : 0)) */
fgd_status fgd_min_bytes_split(const fgd_engine *e, int32_t write_local, int64_t *mix1_bytes,
                               int64_t *blocking_bytes);

/* S_m = sum_p (x_m,p - mean_n x_n,p)^2 of a device [M][ld] array of the
 * given dtype, written to device double out[M], enqueued on `stream`
 * (Sec. 4.4; Appendix D.1). */
fgd_status fgd_consensus_distance(fgd_engine *e, const void *x, int32_t dtype, double *out, void *stream);

/* For callers that cannot allocate device memory (code under HIP stream
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * S_m as fgd_consensus_distance, with no engine and no allocation.  Its
 * block partials live in a static device array of the library, 2048 blocks
 * x FGD_MAX_WORKERS doubles (1 MiB), held on every device it runs on until
 * the process ends; the first call on a device resolves that array's
 * address (hipGetSymbolAddress) and no call allocates or frees anything.
 *   num_workers  M in [1, FGD_MAX_WORKERS]; larger M is rejected
 *                (FGD_ERR_INVALID_ARG): the array holds 64 workers per block
 *   num_params   P >= 0; ld >= P, ld * elem_size a multiple of 16
 *   x            device [M][ld] dtype, 16-byte aligned, read
 *   out          device double[M], 8-byte aligned: S_m
 * Runs on the caller's current device, enqueued on `stream`.  The grid and
 * summation order are those of fgd_consensus_distance on the same device,
 * so the two give the same bits.  Every call on one device shares the one
 * array: calls that may overlap on that device (different streams, or
 * threads) race and must be ordered by the caller.  Each call writes every
 * partial it reads, so nothing needs clearing between calls. */
fgd_status fgd_consensus_distance_noalloc(int32_t num_workers, int64_t num_params, int64_t ld, int32_t dtype,
                                          const void *x, double *out, void *stream);

/* Effective float weights of one round of one slot, in the slot's CSR entry
 * order (dropped entries read 0).  out: host float[nnz]. */
fgd_status fgd_get_effective_weights(const fgd_engine *e, int32_t which, int32_t round, float *out);

/* The same computation without an engine, for one round:
 * mask = host uint8[nnz] or NULL.  Pure host code. */
fgd_status fgd_effective_weights(int32_t num_workers, const int32_t *row_ptr, const int32_t *col_idx,
                                 const float *weights, const uint8_t *mask, int32_t reweight, float *out);

/* Algorithmic minimum HBM traffic of one step:
 * M * P * (3 * elem_size(param_dtype) + 2 * 4) bytes (read theta_prev,
 * theta_local, momentum; write theta_prev, momentum). */
fgd_status fgd_min_bytes_per_step(const fgd_engine *e, int64_t *bytes);

/* Where to put the step's arrays inside one device buffer that the caller
 * allocates (the caller still owns it; the engine only computes offsets).
 * This is a placement rule, not part of the paper's method: on MI355X the
 * fused step, which streams theta_prev, theta_local and the momentum
 * together, was measured to run about 17% slower (8 workers x 1.1e9 bf16
 * parameters: 24.0 against 20.3 ms) when the momentum lies in the same one
 * of the three equal ranges of the device's physical memory (96 GiB each
 * for 288 GiB) as the parameter arrays, and to run at the faster rate when
 * it lies one range further.  Separate allocations made one after another
 * usually land in the same range.
 *   spread       0: packed, every array directly after the previous one;
 *                1: theta_prev, theta_local (and x) packed from offset 0 and
 *                the momentum at offset range_bytes, one range further, when
 *                the packed arrays end within the first range_bytes (else
 *                packed).  The gap between them is free for the caller.  A
 *                spread buffer smaller than 4/3 of range_bytes is sized to
 *                exactly 4/3 of it (128 GiB): a power of two, which the
 *                device allocator places as one aligned block (a smaller
 *                buffer may be pieced together from blocks placed anywhere,
 *                and was measured in the slow placement).
 *   with_x       1: also place x, the stored Mix1 output of split execution
 *                ([M][ld] param_dtype, after theta_local); 0: no x
 *   range_bytes  span of one physical-memory range in bytes, a multiple of
 *                2 MiB; 0 derives it from the engine's device (total memory
 *                / 3, rounded to a whole GiB), which a host-only engine
 *                cannot (FGD_ERR_STATE).  Ignored when spread = 0.
 *   offsets      host int64[4]: byte offsets of theta_prev, theta_local, x
 *                (-1 without x) and momentum, each a multiple of 2 MiB; the
 *                arrays are [M][ld] with the engine's ld and dtypes
 *   total_bytes  host int64: size of the buffer to allocate
 * Offsets into a buffer that starts on a 16-byte boundary satisfy every
 * alignment rule of the compute calls.  Pure host arithmetic plus, for
 * range_bytes = 0, one device query. */
fgd_status fgd_state_layout(const fgd_engine *e, int32_t spread, int32_t with_x, int64_t range_bytes,
                            int64_t *offsets, int64_t *total_bytes);

/* Kernel timing.  While enabled, every fgd_outer_step brackets its fused
 * kernel with HIP events on its stream.  fgd_read_timing waits for the
 * recorded events and returns the summed kernel milliseconds and the number
 * of timed kernels since the last reset (enabling, or disabling, resets).
 * At most 4096 kernels are timed between resets; later steps run untimed
 * (count stays at 4096).  The events are created on first use and kept
 * until fgd_destroy. */
fgd_status fgd_enable_timing(fgd_engine *e, int32_t enable);
fgd_status fgd_read_timing(fgd_engine *e, double *total_ms, int64_t *count);

#define FGD_MAX_JS_TOPK 1024    /* largest top_k of fgd_js_distance */
#define FGD_MAX_JS_WORKERS 4096 /* largest num_workers of fgd_js_distance */

/* Jensen--Shannon functional distance (Sec. 4.4; Appendix D.2) between
 * every worker's predicted token distribution and the parameter-averaged
 * model's, from their logits on a fixed batch of tokens.  Per worker m and
 * token u, in float64 and the log domain: log p = z - logsumexp(z) over the
 * full vocabulary for the worker and for the averaged model; T(u) = the
 * top_k tokens of the averaged model (the paper uses 100; equal logits: the
 * lower token index first); JS = 1/2 sum_{i in T} p_m,i log(p_m,i / mix_i)
 * + 1/2 sum_{i in T} pbar_i log(pbar_i / mix_i), mix = (p_m + pbar) / 2;
 * d_m(u) = sqrt(max(JS, 0) / log 2).  The probabilities are those of the full
 * softmax; only the sum is restricted to T (a lower bound of the full JS,
 * equal to it at top_k = vocab).  No engine is needed.
 *   logits_avg      device [U][ldk] dtype: the averaged model's logits
 *   logits_workers  device [M][U][ldk] dtype: worker m's row for token u
 *                   starts at element (m * U + u) * ldk
 *   dtype           FGD_F32 or FGD_BF16; logits must not be NaN or +inf
 *                   (-inf, a masked token, is allowed)
 *   num_workers     M in [1, FGD_MAX_JS_WORKERS]; num_tokens U in [1, 2^31)
 *   vocab, ldk      K <= ldk; ldk * elem_size a multiple of 16 (16-byte
 *                   aligned rows) and below 2^31 bytes; elements [K, ldk)
 *                   are read, never used
 *   top_k           in [1, min(K, FGD_MAX_JS_TOPK)]
 *   d_out           device double[M][U]: d_m(u)
 *   mean_out        device double[M] or NULL: the mean of d_m(u) over u
 *                   (the paper's CD_JS is the mean of these M values)
 *   topk_out        device int32[U][top_k] or NULL: T(u) in ascending order
 *   workspace       device memory of at least fgd_js_workspace_size bytes,
 *                   16-byte aligned, owned by the caller, overlapping none
 *                   of the arrays above; the call leaves it undefined (it
 *                   carries each row's log-sum-exp parts and the averaged
 *                   rows' largest vector maxima per thread from the call's
 *                   first kernel to the next)
 * Enqueued on `stream`; deterministic.  Calls that share a workspace must
 * not run concurrently. */
fgd_status fgd_js_distance(const void *logits_avg, const void *logits_workers, int32_t dtype, int32_t num_workers,
                           int64_t num_tokens, int64_t vocab, int64_t ldk, int32_t top_k, double *d_out,
                           double *mean_out, int32_t *topk_out, void *workspace, int64_t workspace_bytes,
                           void *stream);

/* Device workspace fgd_js_distance needs for these sizes: 64 bytes per row
 * ((M + 1) U rows) and 4 KiB plus 4 bytes per token (either dtype).  Host
 * only. */
fgd_status fgd_js_workspace_size(int32_t dtype, int32_t num_workers, int64_t num_tokens, int64_t *bytes);

/* Streaming reference with the fused step's memory traffic and none of its
 * arithmetic: the tiles, lane vectors, cache hints and launch shape of
 * fgd_outer_step; every theta_prev and theta_local row of a tile is loaded
 * before use, then row by row the momentum is loaded and theta_prev and the
 * momentum are stored back with their own bits (the arrays are left exactly
 * as they were; a lane vector that straddles P is not stored).  Its rate is
 * the practical ceiling of the step's read/write mix on the arrays' placement.
 * It follows the kernel fgd_outer_step would launch for the current
 * topology (fgd_step_variant; the lane-per-parameter layout when the slots
 * are not set).  Same arrays and rules as fgd_outer_step; M in {1, 2, 4, 8,
 * 16, 32, 64} (else FGD_ERR_UNSUPPORTED).  Enqueued on `stream`. */
fgd_status fgd_stream_step_pattern(fgd_engine *e, void *theta_prev, const void *theta_local, float *momentum,
                                   void *stream);

/* Streaming reference for fgd_js_distance: the loads of its row kernel (the
 * same grid, rows, lane elements, cache hints and prefetch) and none of its
 * arithmetic; the logits are only read, and the workspace is left undefined.
 * Its rate is the practical ceiling of that kernel's access pattern.  Same
 * logits, sizes and workspace rules as fgd_js_distance.  Enqueued on
 * `stream`. */
fgd_status fgd_stream_js_pattern(const void *logits_avg, const void *logits_workers, int32_t dtype,
                                 int32_t num_workers, int64_t num_tokens, int64_t vocab, int64_t ldk, void *workspace,
                                 int64_t workspace_bytes, void *stream);

/* Plain device copy of `bytes` bytes (16-byte aligned pointers, bytes % 16 ==
 * 0) on `stream`: the streaming reference against which the step's
 * bandwidth and traffic counters are read. */
fgd_status fgd_stream_copy(void *dst, const void *src, int64_t bytes, void *stream);

/* Static name of a status; never NULL. */
const char *fgd_status_string(int32_t status);

/* Detail of the last failure on the calling thread ("" if none). */
const char *fgd_last_error(void);

/* Hash of the sources this library was built from, 16 hex digits, fixed at
 * build time: component 0 = every library source and this header, 1 = the
 * outer-step sources (every kernel source but the JS distance's), 2 = the JS
 * distance sources; "unstamped" for a build that did not supply them, "" for
 * another component.  A static string, never NULL.  Tools compare it with
 * the source tree to refuse a library built from other sources, and accept
 * recorded counters or timings only for the hash they were taken with. */
const char *fgd_source_hash(int32_t component);

#ifdef __cplusplus
}
#endif

#endif /* FGD_H */
