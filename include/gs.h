/*
 * gs.h -- C ABI of the gs-SGD gradient-compression hot path on one AMD Instinct MI355X.
 *
 * Method: Dai, Diao, Li, Xu, "A Distributed SGD Algorithm with Global Sketching for Deep
 * Learning Training Acceleration" (arXiv 2108.06004). Per training iteration every worker
 * accumulates momentum and error feedback into its flat gradient, compresses the result
 * into a Count Sketch, the P sketches are summed along a binomial tree (Alg. 1), the top-k
 * coordinates are recovered from the summed sketch, and their exact values are fetched
 * and removed from the error accumulators (HEAVYMIX, Alg. 2).
 *
 * One GPU holds all P workers. The gradients are stacked row-major as [P][d]; the workers'
 * momentum and error state (u, v) is stacked either the same way or worker-interleaved,
 * as chosen by gs_config.state_layout (see there).
 *
 * Conventions shared by every call
 *   - Array arguments are DEVICE pointers to memory owned by the caller (for example
 *     torch tensors on the GPU). The library never frees or retains them beyond the call.
 *     fp32 arrays are IEEE binary32; index arrays are int32. Arrays are dense, row-major,
 *     and must not overlap unless a call says it works in place.
 *   - `stream` is a hipStream_t passed as void* (NULL is the default stream). Every call
 *     validates its arguments on the host, enqueues its kernels on `stream` and returns
 *     without waiting; outputs are valid once the stream has been synchronized.
 *   - The return value is the only error channel. GS_ERR_INVALID_ARG is returned before
 *     anything is enqueued; GS_ERR_DEVICE reports a launch or runtime failure (details in
 *     gs_last_error). No call aborts the process or throws across the ABI.
 *   - Calls on one context must not overlap on different streams: the context's scratch
 *     memory (histograms, candidate lists, bitmaps, internal tables) is shared by them.
 *     Different contexts are independent.
 *   - Only gs_create allocates (gs_unsketch_topk_static uses a fixed array instead). The
 *     per-step calls (everything but gs_create, gs_destroy, gs_step_profiled and
 *     gs_timing_*) neither allocate, synchronize nor clear memory with a memset, so they
 *     can be captured in a HIP graph and replayed.
 *   - Inputs must be finite; results for NaN or infinite inputs are unspecified.
 */
#ifndef GS_H
#define GS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gs_status {
  GS_OK = 0,
  GS_ERR_INVALID_ARG = 1,   /* argument check failed; nothing was enqueued            */
  GS_ERR_OUT_OF_MEMORY = 2, /* gs_create could not allocate its device scratch        */
  GS_ERR_DEVICE = 3,        /* a HIP launch or runtime call failed                    */
  GS_ERR_UNSUPPORTED = 4    /* shape outside what this build implements               */
} gs_status;

#define GS_MAX_WORKERS 64
#define GS_MAX_ROWS 16
#define GS_MERSENNE_P 2147483647u /* 2^31 - 1 */

/* Layouts of the per-worker state arrays u and v (gs_config.state_layout).
 *   GS_STATE_WORKER_MAJOR  [P][d]: element (q, i) at q*d + i (the default, 0).
 *   GS_STATE_INTERLEAVED   [d][GS_STATE_STRIDE(P)]: element (q, i) at i*GS_STATE_STRIDE(P) + q,
 *                          rows padded to a multiple of 4 floats (16 bytes). The padding
 *                          entries (q >= P) are never written and never affect a result.
 * The interleaved form keeps the P values of a coordinate in one 16-byte-aligned row, which
 * is what the sketch gathers, so the step needs no interleaved copy of v. */
#define GS_STATE_WORKER_MAJOR 0
#define GS_STATE_INTERLEAVED 1
#define GS_STATE_STRIDE(P) ((((P) + 3) / 4) * 4)

/*
 * Problem description (Alg. 1 inputs: k, P; the Count Sketch of Sec. III-A).
 *   d        coordinates per worker, 1 <= d <= p - 1 (so every index is a valid hash input)
 *   P        workers, 1 <= P <= GS_MAX_WORKERS
 *   r, c     sketch rows and columns, 1 <= r <= GS_MAX_ROWS, 1 <= c <= p - 1
 *   k_max    the largest k any call on this context may request, 1 <= k_max <= d
 *   rho      momentum factor of the accumulation u <- rho*u + g (finite)
 *   reset_momentum  1: the reset after selection zeroes u as well as v; 0: only v
 *   hash_a, hash_b  HOST arrays [r]: bucket hash h_j(i) = ((a_j*i + b_j) mod p) mod c
 *   sign_a, sign_b  HOST arrays [r]: sign s_j(i) = +1 if ((sign_a_j*i + sign_b_j) mod p) is odd,
 *                   else -1; 1 <= a < p and 0 <= b < p for all four arrays; copied by gs_create.
 *   state_layout    GS_STATE_WORKER_MAJOR (0) or GS_STATE_INTERLEAVED: the layout of u and v
 *                   in every call that takes them (gs_accumulate, gs_sketch's v,
 *                   gs_gather_reset, gs_step, gs_step_heavymix, gs_step_profiled). Other
 *                   values are GS_ERR_INVALID_ARG.
 *   options         0, or GS_OPT_ROW_COPY: reserve a worker-interleaved [d][PP] fp32 copy
 *                   (4 PP d bytes) in an interleaved-state context too. A worker-major context
 *                   with P > 1 always has it (its sketch gathers from it); with P = 1 the
 *                   state [1][d] is a plain vector that the sketch gathers directly. An
 *                   interleaved context with P > 1 needs it only for gs_step_sketch_momentum
 *                   (GS_ERR_UNSUPPORTED without it) and for a v that is not 16-byte aligned
 *                   (GS_ERR_INVALID_ARG without it; torch allocations are aligned). Other
 *                   bits are GS_ERR_INVALID_ARG.
 */
typedef struct gs_config {
  int64_t d;
  int32_t P;
  int32_t r;
  int64_t c;
  int64_t k_max;
  float rho;
  int32_t reset_momentum;
  const uint32_t* hash_a;
  const uint32_t* hash_b;
  const uint32_t* sign_a;
  const uint32_t* sign_b;
  int32_t state_layout;
  int32_t options;
} gs_config;

#define GS_OPT_ROW_COPY 1

typedef struct gs_ctx gs_ctx; /* opaque: a copy of the config plus device scratch */

/* Validate `cfg`, copy it, and allocate the device scratch on the current HIP device.
 * This is the only call that allocates. On success *out receives the context.
 * The sketch runs as a gather into LDS tiles from per-tile coordinate lists built here;
 * when those lists cannot be built (more than 40,960 tiles) it runs as fp64 device
 * atomics instead. Setting the environment variable GS_SKETCH_PATH=atomic before the call
 * selects the atomic form for any shape, and GS_SKETCH_PATH=unpacked keeps the gather's
 * lists in their unpacked form (diagnostic overrides; results agree within the table
 * tolerance). A selection without an estimate vector prunes (estimates only coordinates
 * with enough heavy cells) when d*r exceeds 2,000,000 and estimates every coordinate
 * otherwise; GS_SELECT_PATH=pruned or =full fixes that choice (the selected set is the same
 * either way); GS_EMIT_SPIN=n bounds how long the selection's last kernel waits on the
 * counts of its earlier workgroups before counting their bitmap words itself (0 or negative:
 * sooner or always; the same indices either way, for tests).
 * Device scratch is about (16 + 4.1 r) d + 8 S P r c bytes (S list segments per tile, 1
 * unless the sketch is small), plus the 4 PP d bytes of the interleaved copy (PP = P rounded
 * up to 4) in a worker-major context with P > 1 or with GS_OPT_ROW_COPY, plus 2 r d bytes while the
 * lists are built: with the interleaved state and no copy 1.0 GB at d = 25.6M, P = 8, r = 5,
 * c = 256,000 (1.8 GB worker-major) and 61 GB at d = 2^31 - 2, P = 2, r = 3 (95 GB
 * worker-major). The atomic form replaces the lists and the copy with 8 P r c bytes. */
gs_status gs_create(const gs_config* cfg, gs_ctx** out);

/* Free the context's scratch (after synchronizing the device). NULL is accepted. */
gs_status gs_destroy(gs_ctx* ctx);

/* Momentum and error-feedback accumulation (Sec. II, sketching paragraph: momentum and
 * error accumulation carried along with the sketch; Alg. 1 starts from a zero state).
 * For every worker q and coordinate i, in IEEE fp32 with each operation rounded:
 *     u[q][i] = rho * u[q][i] + g[q][i];   v[q][i] = v[q][i] + u[q][i].
 * g: [P][d] input. u, v: state layout (see gs_config), updated in place. */
gs_status gs_accumulate(gs_ctx* ctx, void* stream, const float* g, float* u, float* v);

/* Count Sketch of every worker's accumulator (Sec. III-A; Alg. 1 sketch step):
 *     tables[q][j][col] = sum over i with h_j(i) == col of s_j(i) * v[q][i].
 * v: state layout input. tables: [P][r][c] output (overwritten; each cell is the sum
 * accumulated in double precision and rounded once to fp32). */
gs_status gs_sketch(gs_ctx* ctx, void* stream, const float* v, float* tables);

/* Sum of the P worker sketches in the binomial-tree order of Alg. 1 (in each round the
 * even local rank adds the next rank's sketch; an unpaired highest rank passes through).
 * tables: [P][r][c] input. merged: [r][c] output. Deterministic. */
gs_status gs_merge(gs_ctx* ctx, void* stream, const float* tables, float* merged);

/* HEAVYMIX estimate and selection (Alg. 2). For every coordinate i the estimate is the
 * median over rows of s_j(i) * merged[j][h_j(i)] (even r: mean of the two middle values,
 * fl(fl(m1 + m2) * 0.5)). idx receives the k coordinates with the largest |estimate|,
 * ties broken toward the lower index, in ascending order.
 * merged: [r][c] input. est: [d] output, or NULL when not wanted. idx: [k] output.
 * 1 <= k <= k_max. */
gs_status gs_unsketch_topk(gs_ctx* ctx, void* stream, const float* merged, int64_t k, float* est, int32_t* idx);

/* Exact values of the selected coordinates (Alg. 2, second round) and their reset.
 * For t < k, with i = idx[t]: values[t] = tree-order sum over q of v[q][i] (the merge
 * order above); then v[q][i] = 0 for every q, and u[q][i] = 0 too when reset_momentum.
 * idx: [k] distinct coordinates in [0, d) (e.g. the output of gs_unsketch_topk).
 * u, v: state layout, updated in place. values: [k] output. 1 <= k <= k_max. */
gs_status gs_gather_reset(gs_ctx* ctx, void* stream, const int32_t* idx, int64_t k, float* u, float* v,
                          float* values);

/* One whole step: accumulate, sketch, merge, estimate + top-k, exact values + reset, with
 * the per-worker tables kept in context scratch. Equivalent to the five calls above.
 * g: [P][d] input. u, v: state layout, in place. merged: [r][c] output. idx, values: [k]
 * outputs. */
gs_status gs_step(gs_ctx* ctx, void* stream, const float* g, float* u, float* v, int64_t k, float* merged,
                  int32_t* idx, float* values);

/* HEAVYMIX as printed (Alg. 2): query every estimate, split the coordinates into the heavy
 * set H = { i : est_i^2 >= l2sq / k } and the rest NH, and select H plus a random fill of
 * l = k - |H| coordinates of NH.
 *   est_i   as in gs_unsketch_topk.
 *   l2sq    the l2-norm-squared estimate: the median over rows of sum_col merged[j][col]^2,
 *           in double precision, each row summed in a fixed order -- the squares (exact),
 *           padded with zeros to the next power of two, added in adjacent pairs level by
 *           level; for even r the mean of the two middle row sums, fl(fl(m1 + m2) * 0.5).
 *   heavy   est_i^2 >= fl(l2sq / k), with est_i^2 exact in double precision.
 *   fill    the l coordinates of NH with the largest rnd[i] >> 1, ties to the lower index
 *           (a uniformly random l-subset of NH when the draws are independent and uniform).
 *   |H|>=k  the k members of H with the largest |est_i|, ties to the lower index.
 * merged: [r][c] input. rnd: [d] input, the caller's uniform 32-bit draws for this call (the
 * method's random numbers; pass fresh draws for every step). est: [d] output or NULL.
 * idx: [k] output, ascending. n_heavy: one int64 output (|H|) or NULL. l2sq: one double
 * output or NULL. All pointers are device pointers. 1 <= k <= k_max. */
gs_status gs_heavymix_topk(gs_ctx* ctx, void* stream, const float* merged, int64_t k, const uint32_t* rnd,
                           float* est, int32_t* idx, int64_t* n_heavy, double* l2sq);

/* One whole step with HEAVYMIX as printed in place of the deterministic top-k: accumulate,
 * sketch, merge, gs_heavymix_topk, exact values + reset. Arguments as in gs_step plus rnd
 * ([d] device input, this step's draws) and n_heavy (one int64 device output or NULL). */
gs_status gs_step_heavymix(gs_ctx* ctx, void* stream, const float* g, float* u, float* v, int64_t k,
                           const uint32_t* rnd, float* merged, int32_t* idx, float* values, int64_t* n_heavy);

/* One step with momentum and error accumulation kept in the merged sketch instead of in
 * per-worker d-vectors (the sketch is linear, so both can be carried inside it: Sec. II,
 * sketching paragraph). With S the tree-order merge of the P workers' sketches of g:
 *   U <- fl(fl(rho U) + S), E <- fl(E + U)                      per cell, fp32, no FMA
 *   idx = the k largest |estimate of E|, ties to the lower index, ascending
 *   values[t] = the estimate of E at idx[t] (taken before the correction below)
 *   E <- fl(E - D) on every cell that D touches, with D the sketch of the selection (the
 *        values at idx, signed and bucketed like any sketch), each cell summed in double
 *        precision and rounded once; U <- 0 on those cells when reset_momentum is set.
 * g: [P][d] input. U, E: [r][c] state, updated in place (zero before the first step).
 * merged: [r][c] output (S). idx: [k] output, values: [k] output. 1 <= k <= k_max.
 * Uses the context's per-worker sketch scratch, so calls on one context must not overlap. */
gs_status gs_step_sketch_momentum(gs_ctx* ctx, void* stream, const float* g, float* U, float* E, int64_t k,
                                  float* merged, int32_t* idx, float* values);

/* The weight update (Alg. 1, last step): w <- w - lr * G~, with G~ zero outside the
 * selection: for t < k, w[idx[t]] = fl(w[idx[t]] - fl(lr * values[t])) (no fused
 * multiply-add). idx: [k] distinct coordinates in [0, d) (e.g. from gs_step). values: [k].
 * w: [d] parameters, updated in place. lr finite. 1 <= k <= k_max. */
gs_status gs_apply_update(gs_ctx* ctx, void* stream, const int32_t* idx, const float* values, int64_t k, float lr,
                          float* w);

/* Stage timing for benchmarks and profiling. Runs exactly the kernels of gs_step, records a
 * HIP event on `stream` before the first stage and after each stage, synchronizes the stream
 * and writes the stage durations in milliseconds to the HOST array stage_ms[GS_NUM_STAGES]:
 *   [0] accumulate   [1] sketch   [2] merge   [3] estimate + top-k selection
 *   [4] gather + reset
 * Unlike gs_step this call blocks until the step has finished. */
#define GS_NUM_STAGES 5
gs_status gs_step_profiled(gs_ctx* ctx, void* stream, const float* g, float* u, float* v, int64_t k, float* merged,
                           int32_t* idx, float* values, float* stage_ms);

/* Stage timing over ordinary steps (for benchmarks). gs_timing_start allocates
 * max_steps * (GS_NUM_STAGES + 1) HIP events; while it is active, each of the next max_steps
 * calls of gs_step, gs_step_heavymix or gs_step_sketch_momentum records one event on its
 * stream before its first stage and one after each stage, without synchronizing (stages as
 * for gs_step_profiled; for gs_step_sketch_momentum [0] is the gradient interleave and [4]
 * the estimate correction of the sketch-space state). gs_timing_stop synchronizes, writes the
 * mean stage durations in milliseconds to the HOST array stage_ms[GS_NUM_STAGES] (may be
 * NULL) and the number of timed steps to *n_steps (may be NULL), and frees the events.
 * 1 <= max_steps <= 2^20; starting while active, or stopping while not, is
 * GS_ERR_INVALID_ARG. The calls of one context must come from one host thread. */
gs_status gs_timing_start(gs_ctx* ctx, int32_t max_steps);
gs_status gs_timing_stop(gs_ctx* ctx, float* stage_ms, int32_t* n_steps);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): gs_unsketch_topk without a context.
 * Same results as gs_unsketch_topk on a context with the same d, r, c and hash parameters
 * (it runs that call's kernels with every coordinate estimated): est (when non-NULL) the
 * median estimates, idx the k largest |estimate|, ties to the lower index, ascending.
 *   cfg     host pointer; d, r, c and the four host hash arrays are used, with the ranges
 *           of gs_create and 1 <= d <= GS_STATIC_MAX_D; P, k_max, rho, reset_momentum and
 *           state_layout are ignored. 1 <= k <= d.
 *   merged  [r][c] device input; est [d] device output or NULL; idx [k] device output.
 * Scratch: no call allocates or frees. The selection's scratch is a fixed array of the
 * library in device memory, 12.1 bytes per coordinate of GS_STATIC_MAX_D (48.6 MiB), of
 * which each GPU the library runs on holds its own copy until the process ends; the first
 * call on a device looks up that device's copy. Calls on one GPU share the array and keep
 * the last call's contents: calls that overlap on one GPU (other streams or threads without
 * ordering between them) race. Each call clears what must start at zero with a kernel (no
 * memset), so a call can be captured in a HIP graph once the device has been set up.
 * Errors: GS_ERR_INVALID_ARG before anything is enqueued (a larger d among them),
 * GS_ERR_DEVICE for a failed set-up or launch; gs_last_error(NULL) holds the message. */
#define GS_STATIC_MAX_D 4194304
gs_status gs_unsketch_topk_static(const gs_config* cfg, void* stream, const float* merged, int64_t k, float* est,
                                  int32_t* idx);

/* The form a context computes in, fixed by gs_create (for tests and benchmark reports).
 *   sketch            GS_SKETCH_GATHER: LDS tiles gather their listed coordinates (Sec. III-A,
 *                     S(g) = C g, cell by cell); GS_SKETCH_ATOMIC: fp64 device atomics
 *   tile_width        columns per tile (gather), tiles = r * tiles per row, segments = list
 *                     segments per tile (tiles split so that small sketches fill the GPU)
 *   packed_lists      1: one 32-bit word per list entry (coordinate offset, position, sign)
 *   prune             1: selections without an estimate vector prune (d * r > 2,000,000)
 *   row_copy          1: the context holds the interleaved copy of v ([d][PP] floats)
 * Errors: GS_ERR_INVALID_ARG for a NULL argument. */
#define GS_SKETCH_GATHER 0
#define GS_SKETCH_ATOMIC 1
typedef struct gs_plan {
  int32_t sketch;
  int32_t tile_width;
  int32_t tiles;
  int32_t segments;
  int32_t packed_lists;
  int32_t prune;
  int32_t row_copy;
} gs_plan;
gs_status gs_describe(const gs_ctx* ctx, gs_plan* out);

/* Static description of a status code. */
const char* gs_status_string(gs_status status);

/* Message describing the last failing call on `ctx` ("" if none); valid until the next
 * call on the context. With ctx == NULL: the last failing context-free call (gs_create or
 * gs_unsketch_topk_static) on this thread. */
const char* gs_last_error(const gs_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* GS_H */
