/*
 * mfsgd.h -- C ABI of the MI355X (gfx950) SGD matrix-factorisation library.
 *
 * The library trains R ~ P x Q from sparse ratings with stochastic gradient
 * descent, the method of Xie, Tan, Fong, Liang, "CuMF_SGD: Fast and Scalable
 * Matrix Factorization" (arXiv 1610.05838):
 *   - the per-sample update of section 2.2 (prediction error, then the
 *     regularised update of p_u and q_v, both from their values before the
 *     step),
 *   - the two single-GPU schedules of section 3.2: batch-Hogwild!
 *     (section 3.2.2) and wavefront-update (section 3.2.3),
 *   - the test RMSE used as the convergence measure (section 3.2.4).
 *
 * Conventions for every call:
 *   - Every entry point returns an int status: MFSGD_OK (0) or a negative
 *     MFSGD_E* code; mfsgd_last_error() then describes the failure.  No C++
 *     exception crosses the ABI.
 *   - All calls act on one process-wide context (one model on the current
 *     HIP device).  The library is not thread-safe: calls must not overlap.
 *   - `stream` is a hipStream_t passed as void*; NULL is the default (null)
 *     stream.  Calls documented as asynchronous only enqueue work.
 *   - Sample arrays are caller-owned device memory holding packed 12-byte
 *     mfsgd_sample records; they must stay alive and unchanged until the
 *     work enqueued on them has completed.
 *   - P, Q, the wavefront plan, tickets and all scratch are library-owned
 *     device memory, released by mfsgd_finalize() or by the next mfsgd_init().
 *   - Feature storage: P is m rows of k values and Q is stored transposed,
 *     n rows of k values (row v is the item vector q_v, the paper's column v
 *     of the k x n matrix Q), so both rows are contiguous.  Rows are padded
 *     internally to a supported width with zero columns; the padding stays
 *     exactly zero and is invisible through get/set.
 */
#ifndef MFSGD_H
#define MFSGD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* One observed rating r of user u for item v (0-based), 12 bytes, packed.
 * Section 3.2.2 sizes a sample as two integers and one float. */
typedef struct {
    int32_t u;
    int32_t v;
    float r;
} mfsgd_sample;

enum {
    MFSGD_OK = 0,
    MFSGD_EINVAL = -1,   /* bad argument, option, size or index range       */
    MFSGD_ENOMEM = -2,   /* device or pinned-host allocation failed         */
    MFSGD_EHIP = -3,     /* a HIP runtime call failed (message has details) */
    MFSGD_ESTATE = -4,   /* call not valid in the current state             */
    MFSGD_ETIMEOUT = -5, /* a wavefront ticket wait hit the spin limit      */
    MFSGD_ENUMERIC = -6  /* non-finite RMSE                                 */
};

/* Schedules (section 3.2).
 *
 * MI355X has eight XCDs, each with its own L2 cache; the L2s are not coherent
 * with each other inside a kernel.  Lock-free updates that meet in one L2 see
 * each other at once; updates from different XCDs only when lines are
 * written back and evicted, and of two stores to one row that overlap the
 * later wins.  The block-scheduled forms keep each worker team on one XCD and
 * pass rows between teams only at block hand-over (agent-scope
 * release/acquire), which is the paper's own answer for workers without a
 * shared coherent memory (section 2.3, and the block partition of section
 * 4.1 applied to XCDs instead of GPUs). */
enum {
    /* batch-Hogwild! (section 3.2.2): samples are taken in batches of f
     * consecutive samples, each batch updated serially by one worker, workers
     * never lock.  The form is option "partition":
     *   2 (default) automatic, the form that follows the serial order within
     *     the Hogwild! tolerance for these samples (at most min(m, n) / 20
     *     workers -- the paper's empirical Hogwild! condition, section 5.5.1
     *     -- and one sample in flight per wavefront): batch-Hogwild! inside
     *     one XCD (form 4) when the most popular user or item holds more than
     *     1/64 of the samples (or k <= 32, or binary16 at k <= 64), otherwise
     *     over all XCDs in one address space with every change added
     *     atomically (form 0 with "atomic"), the Hogwild! model of
     *     component-wise atomic updates, so no concurrent update is lost;
     *     atomic adds read from stale rows add up, so their worker count is
     *     also kept at most 1 / (4 lr s) for the most popular row's share s.
     *     The sample array's per-row counts are taken once (synchronously) on
     *     its first such epoch.  Read-only "hogwild_form" and
     *     "hogwild_atomic" report what the last epoch ran.
     *   0 one address space over all XCDs: batch b goes to worker (wavefront;
     *     half-wavefront at k <= 32, see "half_waves") b mod W.  With plain
     *     stores a row that several XCDs keep cached is updated in separate
     *     copies of which the one written back last wins, so on data with
     *     very popular rows the per-epoch convergence trails the serial order
     *     (see "sync_every", "coherent"); with "atomic" the changes are added
     *     atomically instead.
     *   1 partitioned: the rating matrix is cut into an s x s grid (s =
     *     number of XCDs unless "hogwild_grid" says otherwise; planned
     *     internally, once per sample array) and the wavefronts of each XCD
     *     run batch-Hogwild! inside the block the wavefront schedule below
     *     gives that XCD's worker, each claiming the block's next batch when
     *     it is free, so concurrent updates always meet in one L2; the block
     *     order trails the serial order per epoch (section 5.5.2).
     *   3 as 1 without the column tickets (the fastest form): workers that
     *     drift apart may share a column block across XCDs.
     *   4 one XCD: the whole array as one block run by the wavefronts of one
     *     XCD (a 1 x 1 grid), claiming batches in order. */
    MFSGD_BATCH_HOGWILD = 0,
    /* wavefront-update (section 3.2.3) on the s x s grid of the last
     * mfsgd_plan: worker i owns row block i and visits the column blocks in
     * the order sigma_i(w) = C[(i + O[w]) mod s], C and O permutations drawn
     * per epoch from (seed, epoch), so the blocks of one wave share no row and
     * no column.  A 1-D array of column tickets orders the waves: worker i
     * starts wave w once column sigma_i(w) has been released by wave w-1.  A
     * worker lives on one XCD; inside its open block the wavefronts of that
     * XCD claim batches of f samples one at a time and run them as
     * batch-Hogwild!, and a wavefront with nothing to claim for its own
     * worker serves the other workers of its XCD.  Work is claimed, not
     * assigned, so the launch does not depend on every workgroup being
     * resident at once. */
    MFSGD_WAVEFRONT = 1,
    /* the same schedule with one wavefront per worker and each block's
     * samples in their array order: the result then equals the serial
     * update in wave order up to floating-point rounding (deterministic).
     * Option "wave_launch" runs it as one kernel launch per wave instead. */
    MFSGD_WAVEFRONT_DET = 2,
    /* LIBMF's global scheduling table (section 3.2.1), the baseline the two
     * schedules above replace ("LIBMF-GPU" in the paper).  R is cut into a
     * "table_grid" x "table_grid" grid of equal index ranges
     * (floor(u*s/m), floor(v*s/n); planned internally, synchronously, on the
     * first such epoch on a sample array).  Each of "table_workers"
     * wavefronts is one worker: it takes a lock on the one table, picks a
     * block not yet taken in this epoch whose row block and column block no
     * other worker holds, marks both, releases the lock, updates the block's
     * samples serially in array order, then clears its marks.  Every
     * non-empty block is taken once per epoch.  The choice among the free
     * blocks is random: the blocks not yet taken form a list (initially the
     * non-empty block ids, ascending); decision d of epoch t draws a list
     * position from output d of the SplitMix64 stream keyed (seed, 2^40 + t)
     * (high 32 bits times the list length, shifted down 32), takes the first
     * free block at or cyclically after it, and moves the list's last entry
     * into its slot.  With one worker the result therefore equals the
     * serial update in that block order (deterministic).  Needs nnz < 2^32. */
    MFSGD_GLOBAL_TABLE = 3
};

enum { MFSGD_FP32 = 0, MFSGD_FP16 = 1 };

/* Options (integer valued).  Keys:
 *   "dtype"        feature storage: MFSGD_FP32 (default) or MFSGD_FP16
 *                  (binary16 storage, binary32 arithmetic, round to nearest
 *                  even on store; section 3.1 "Half-precision").  Takes
 *                  effect at the next mfsgd_init.
 *   "batch_f"      batch size f, a positive multiple of 64 (default 256, the
 *                  paper's choice in section 3.2.2).
 *   "workers"      batch-Hogwild! wavefronts in total; 0 (default) = as many
 *                  as stay resident on the GPU (the automatic form: at most
 *                  min(m, n) / 20, see MFSGD_BATCH_HOGWILD).
 *   "depth"        samples each wavefront keeps in flight: 1, 2, 4 or 8, or
 *                  0 (default) automatically: 1 for the automatic and the
 *                  one-XCD batch-Hogwild! forms (bound by one XCD's
 *                  bandwidth or by atomics, not by latency, so one in flight
 *                  runs as fast and halves the updates in flight), 2
 *                  elsewhere.  A wavefront forwards
 *                  its own pending updates, so depth never changes the
 *                  serial semantics of one worker; fewer samples in flight
 *                  also means fresher reads of the rows other workers update.
 *   "team_waves"   wavefronts per wavefront-update worker (rounded up to
 *                  whole workgroups of 4); 0 (default) = every workgroup slot
 *                  the occupancy allows, shared among the s workers in
 *                  proportion to the samples of their row blocks (each
 *                  worker on one XCD, the XCDs loaded as evenly as the row
 *                  blocks allow).  A worker's wavefronts prefer its blocks
 *                  but also serve the other workers on their XCD.
 *   "priority"     pooled block-scheduled epochs: 1 (default) a wavefront
 *                  that finds several open blocks takes the one with the
 *                  most work chained behind it (MFSGD_DBG_PRIORITY: the
 *                  epoch's critical path runs through it, e.g. the blocks
 *                  of a column holding far more than its share, and the
 *                  blocks that gate them); among equals, and with 0, its
 *                  own worker's block first.
 *   "tail_claims"  pooled block-scheduled epochs: 1 claims a block's last
 *                  2 units of 64 samples per wavefront of the XCD one unit
 *                  at a time instead of in batches of f; 0 (default).
 *   "partition"    batch-Hogwild! form, 0 to 4 (default 2, automatic; see
 *                  MFSGD_BATCH_HOGWILD).
 *   "atomic"       1: batch-Hogwild! in one address space or in one XCD adds
 *                  the change of every value with an atomic add (binary32
 *                  add, or packed binary16 add; k > 64 for binary16) instead
 *                  of storing the new row, at depth 1; with "hot_log2" = L >
 *                  0 only rows holding at least nnz >> L samples are added,
 *                  the others stored.  0 (default): stores (the automatic
 *                  form decides by itself).
 *   "coherent"     one address space, plain stores: 1 agent-scope
 *                  (write-through) stores, 2 the same plus agent-scope loads,
 *                  3 non-temporal stores, 4 system-scope stores, for every
 *                  row not marked hot by "hot_log2" (hot rows keep plain
 *                  write-back stores); 0 (default) plain.  Measured options:
 *                  they shrink the per-XCD copies but cost time.
 *   "coherent_mat" which matrices "coherent" applies to: bit 0 P, bit 1 Q
 *                  (default 3).
 *   "hot_log2"     hot rows for "coherent" and "atomic": rows with at least
 *                  nnz >> hot_log2 samples (0, the default: none).
 *   "hogwild_grid" grid side of the partitioned batch-Hogwild!; 0 (default)
 *                  = number of XCDs.
 *   "balance"      how a grid is cut: 1 into consecutive index ranges
 *                  holding as equal sample counts as consecutive ranges
 *                  allow (the smallest possible largest range, ranges
 *                  filled greedily at that size); 0 into equal index ranges
 *                  floor(u*s/m), floor(v*s/n); 2 (default) automatic: 1
 *                  when s is at most the number of XCDs (each worker then
 *                  has an XCD to itself, so the largest row block sets the
 *                  epoch time), 0 above (the workers sharing an XCD share
 *                  its wavefronts, and the greedy fill can leave ranges
 *                  empty when one index holds a large share).
 *   "sync_every"   one-address-space batch-Hogwild!: every this many of its
 *                  batches, one wavefront per XCD writes that XCD's L2 back
 *                  and invalidates it, bounding how long an update stays
 *                  invisible to other XCDs; 0 (default) = never.
 *   "sync_l1"      with sync_every: the other wavefronts also drop their CU's
 *                  L1 at those points (default 0).
 *   "spin_limit"   polls of a column ticket before the wait gives up with
 *                  MFSGD_ETIMEOUT (default 2^24, each poll sleeps briefly).
 *   "skip_stores"  block-scheduled epochs: a wavefront that updates a row
 *                  again within its in-flight window writes it back once per
 *                  run (the final values are the same).  0 never, 1 always,
 *                  2 (default) when one user or one item holds more than
 *                  half of the samples of its row or column block (many
 *                  wavefronts then update one row at once), except in
 *                  partitioned batch-Hogwild! at k <= 32 with "half_waves"
 *                  on.  Epochs with debug output never skip.
 *   "stage_samples" samples per chunk of mfsgd_epoch_staged (default 2^25,
 *                  402 MB per buffer; three device buffers, and three
 *                  pinned host buffers for pageable arrays).
 *   "wave_launch"  MFSGD_WAVEFRONT_DET only: 1 runs every wave as a kernel
 *                  launch of its own (worker i of wave w updates block
 *                  (i, sigma_i(w)) serially; the launch boundary orders the
 *                  waves, no tickets), a cross-check of the ticketed kernel
 *                  whose factors it reproduces bit for bit; 0 (default) the
 *                  persistent ticketed kernel.
 *   "half_waves"   two workers per wavefront, one per half of its 64
 *                  lanes, each lane holding (padded k)/32 values.
 *                  1 (default): at k <= 32 (a row of 32 values fills a
 *                  half), and for pooled wavefront-update at wider rows of
 *                  at most 16 bytes per lane when no column block of the
 *                  plan holds more than twice the mean share of the
 *                  samples; 2: everywhere at widths of at most 16 bytes per
 *                  lane (binary32 k <= 128, binary16 k <= 256); 0: never (at
 *                  k <= 32 the upper 32 lanes then idle).  In one address
 *                  space "workers" and the default worker count are then
 *                  counted in half-wavefronts.  Block-scheduled with teams
 *                  of more than one wavefront, a wavefront claims two
 *                  batches of its open block at once and runs one per half:
 *                  at k <= 32 (batch-Hogwild!) instead of skipping stores
 *                  (unless "skip_stores" is 1), at wider rows with skipped
 *                  stores where "skip_stores" calls for them; the automatic
 *                  one-XCD form counts such a wavefront as two workers.  At
 *                  k <= 32 a lone worker computes the same bits either way;
 *                  at wider rows its lane sums run in another order.
 *   "table_grid"   grid side of MFSGD_GLOBAL_TABLE, 1 to 1024 (default 256).
 *   "table_workers" MFSGD_GLOBAL_TABLE workers (wavefronts); 0 (default) =
 *                  table_grid / 2 (at least 1): about twice as many row and
 *                  column blocks as workers, so that a free worker usually
 *                  finds an idle block.
 *   "debug"        bit 0: count visits of every sample (read with
 *                  mfsgd_debug_read(MFSGD_DBG_VISITS)); bit 1: record the
 *                  schedule (MFSGD_DBG_TRACE).  Costs one extra atomic per
 *                  sample; a block-scheduled epoch needs a plan made while
 *                  bit 0 was set.
 * Read-only keys (after mfsgd_init): "resident_waves" (wavefronts of the
 * one-address-space epoch kernel the GPU holds at once), "xcds" (XCDs: the
 * largest hardware XCD id an init probe saw, plus one), "xcd_round_robin" (1
 * if that probe's workgroups were dealt round-robin), "cus",
 * "partitioned" (whether batch-Hogwild! runs block-scheduled: the last
 * epoch's form, or before one the option's), "hogwild_form" (form of the last
 * batch-Hogwild! epoch, values of "partition" other than 2; -1 before one),
 * "hogwild_atomic" (whether it added its updates atomically),
 * "half_workers" (whether its one-address-space form runs two workers per
 * wavefront for this model), "blocked_pairs" (whether the last
 * block-scheduled epoch, wavefront-update or block-scheduled
 * batch-Hogwild!, had each wavefront claim two batches and run one per half;
 * -1 before one),
 * "table_blocks" (non-empty blocks of the last global-table plan, 0 before one),
 * "blocked_per_cu" (workgroups per CU the occupancy query reports for the
 * block-scheduled kernel with one batch per claim; the two-batch variant
 * holds twice the values per lane and may fit fewer), "teams_grid"
 * (workgroups of the last block-scheduled epoch, 0 before one).
 * Returns MFSGD_EINVAL for an unknown key or an out-of-range value. */
int mfsgd_set_option(const char* key, int64_t value);
int mfsgd_get_option(const char* key, int64_t* value);
/* Restore every option to its default (the values listed above).  Host
 * logic only; takes effect like mfsgd_set_option.  Always MFSGD_OK. */
int mfsgd_reset_options(void);

/* Allocate P (m x k) and Q (n x k) in the storage dtype on the current
 * device and initialise every entry uniformly on [0, 1/sqrt(k)): entry j of
 * row u of P is output u*k+j of the SplitMix64 stream keyed (seed, 1) -- the
 * stream's state is output 1 of a SplitMix64 generator seeded with `seed` --
 * whose top 24 bits times 2^-24 are multiplied in binary64 by 1/sqrt(k) and
 * rounded once to the storage type; Q likewise with stream (seed, 2).  The
 * paper fixes no initialisation; this one is reproducible bit for bit.
 * Resets the epoch counter to 0 and drops any plan.  Synchronous.
 * EINVAL: m or n not in [1, 2^31-1], k not in [1, 512]. */
int mfsgd_init(int64_t m, int64_t n, int32_t k, uint64_t seed);

/* Wavefront-update preparation (section 3.2.3): check every sample's indices
 * (0 <= u < m, 0 <= v < n), cut the grid into s x s blocks (see option
 * "balance") and keep a library-owned copy of the samples grouped by block,
 * in array order inside each block.  The plan is tied to (samples, nnz): a
 * wavefront epoch on other samples returns MFSGD_ESTATE.  Synchronises
 * `stream`.  EINVAL: s not in [1, 64], nnz < 0, NULL samples with nnz > 0,
 * or an out-of-range index (nothing is planned then). */
int mfsgd_plan(const mfsgd_sample* samples, int64_t nnz, int32_t s, void* stream);

/* One epoch: every one of the nnz samples is used for exactly one update
 * (section 2.3), under `scheme`, with learning rate lr and regularisation
 * lambda_p, lambda_q (section 2.2).  Asynchronous on `stream`, except that
 * the first partitioned batch-Hogwild! or global-table epoch on a sample
 * array plans it (synchronously, like mfsgd_plan).  Increments the epoch counter, which
 * keys the per-epoch column orders.  Indices are not checked by the
 * one-address-space batch-Hogwild! (use mfsgd_check_samples): an index out
 * of range is undefined behaviour there.
 * EINVAL: nnz < 0, NULL samples with nnz > 0, unknown scheme, non-finite lr
 * or lambda, (planning) an index out of range, or nnz >= 2^32 for
 * MFSGD_GLOBAL_TABLE.  ESTATE: no init, or a
 * wavefront scheme without a plan for these samples. */
int mfsgd_epoch(const mfsgd_sample* samples, int64_t nnz, float lr, float lambda_p, float lambda_q,
                int32_t scheme, void* stream);

/* One batch-Hogwild! epoch over samples that stay in host memory, for sample
 * arrays larger than the GPU's memory: the out-of-core mode of section 4,
 * where the transfer of the next part of R overlaps the computation on the
 * current one.  The array is cut into chunks of "stage_samples" consecutive
 * samples (rounded down to a multiple of f); chunk i is copied into one of
 * three library-owned device buffers on a library-owned stream while the
 * kernel of chunk i-1 runs on `stream`, and each chunk is run like
 * MFSGD_BATCH_HOGWILD in one address space (batch b of the chunk to worker
 * b mod W, chunks in array order).  With one worker this is exactly the
 * serial update in array order.
 * samples: host memory, caller-owned, 12-byte records as for mfsgd_epoch.
 * Pinned memory (hipHostMalloc) is copied directly and must stay valid and
 * unchanged until the work on `stream` completes; pageable memory is copied
 * by this thread into pinned staging buffers, so the call returns once its
 * last chunk has been staged.  Asynchronous on `stream` otherwise;
 * increments the epoch counter.  Indices are not checked (use
 * mfsgd_check_samples on a device copy).  Debug bit 0 counts visits as for
 * mfsgd_epoch.
 * EINVAL: nnz < 0, NULL samples with nnz > 0, a device pointer, non-finite
 * lr or lambda.  ESTATE: no init.  ENOMEM: staging buffers. */
int mfsgd_epoch_staged(const mfsgd_sample* samples, int64_t nnz, float lr, float lambda_p, float lambda_q,
                       void* stream);

/* Test RMSE (section 3.2.4): sqrt(sum over the ntest samples of
 * (r - p_u . q_v)^2 / ntest), dot products in binary32, squares summed in
 * binary64 in a fixed order (the result is reproducible bit for bit); 0 for
 * ntest == 0.  Synchronises `stream` and writes *rmse_out.  Also reports a
 * pending device error (ETIMEOUT) of earlier work on the stream.
 * ENUMERIC: the result is not finite (it is still written). */
int mfsgd_rmse(const mfsgd_sample* test, int64_t ntest, double* rmse_out, void* stream);

/* The same test RMSE for callers that cannot allocate or synchronise: code
 * under HIP graph capture and tight serving loops.  Enqueues the two RMSE
 * kernels on `stream` and returns at once; the result (0 for ntest == 0) is
 * written to *rmse_dev, one binary64 in caller-owned DEVICE memory, when the
 * stream reaches it.  Same kernels and summation order as mfsgd_rmse, hence
 * the same value bit for bit.  It calls no allocation routine: the 2048
 * partial sums go to a fixed 16 KiB array in device memory (one per GPU,
 * held until the process ends; its address is taken at mfsgd_init on the
 * device current then), which every call on that GPU reuses and fully
 * rewrites -- calls that overlap on one GPU (two streams, or two threads)
 * race on it.  ntest is not limited by the scratch (the partial count is
 * fixed).  Errors: ESTATE before mfsgd_init or when the current device is
 * not the one mfsgd_init ran on; EINVAL for a bad array or NULL rmse_dev;
 * EHIP for a launch failure.  Device-side errors and a non-finite result
 * are not reported here (nothing is waited for): mfsgd_sync reports the
 * former, the caller checks the value. */
int mfsgd_rmse_noalloc(const mfsgd_sample* test, int64_t ntest, double* rmse_dev, void* stream);

/* Check that every sample index is in range.  Synchronises `stream`.
 * EINVAL if any is not. */
int mfsgd_check_samples(const mfsgd_sample* samples, int64_t nnz, void* stream);

/* Wait for `stream` and report a device-side error of earlier epochs
 * (MFSGD_ETIMEOUT if a ticket wait gave up; the flag is then cleared). */
int mfsgd_sync(void* stream);

/* Copy the factors out / in, compact m x k and n x k row-major in the
 * storage dtype (4 or 2 bytes per value).  The pointers may be host or
 * device memory.  Synchronise `stream`.  Either pointer may be NULL to skip
 * that matrix. */
int mfsgd_get_factors(void* P, void* Q, void* stream);
int mfsgd_set_factors(const void* P, const void* Q, void* stream);

/* Epoch counter (keys the per-epoch wavefront column orders); saved with the
 * factors for checkpoint/resume. */
int mfsgd_set_epoch(int64_t t);
int64_t mfsgd_get_epoch(void);

/* Debug buffers (see the "debug" option).  Synchronise `stream`.
 *   MFSGD_DBG_VISITS : count = nnz of the last epoch, dst uint32[count] --
 *                      how often each sample was used since the last epoch
 *                      started (wavefront epochs count by position in the
 *                      caller's array).
 *   MFSGD_DBG_TRACE  : batch-Hogwild!: dst int32[ceil(nnz/f)], the worker
 *                      that ran each batch; wavefront and partitioned
 *                      batch-Hogwild!: dst int32[s*s], entry i*s+w = column
 *                      block of worker i in wave w, optionally followed by
 *                      2*s*s values of one event counter (count up to
 *                      3*s*s): entry s*s + 2(i*s+w) = the earliest claim of
 *                      a batch of that block, the next entry = the completion
 *                      of its last batch (the block of wave w+1 in the same
 *                      column is claimed only after that; 0xffffffff where
 *                      not recorded, e.g. per-wave launches), optionally
 *                      followed by 2*s*s clock stamps (count up to 5*s*s):
 *                      the low 32 bits of the 100 MHz realtime counter when
 *                      the block's first batch was claimed and when its last
 *                      batch completed, same order;
 *                      global table: dst int32[3*B], B = "table_blocks": for
 *                      decision d, entry 3d = the block id I*s+J taken, 3d+1
 *                      and 3d+2 = the values of one event counter when the
 *                      block was taken and when it was given back (a block
 *                      that shares a row or column block with another is
 *                      taken only after the other was given back).
 *   MFSGD_DBG_PLAN_STARTS : the wavefront-update plan of the last mfsgd_plan:
 *                      count = s*s+1, dst int64 -- first planned position of
 *                      block (I, J) at entry I*s+J, nnz at entry s*s.
 *   MFSGD_DBG_PLAN_ORDER  : same plan, count <= nnz, dst int64 -- position in
 *                      the caller's array of each planned sample (needs a plan
 *                      made while debug bit 0 was set).
 *   MFSGD_DBG_TEAM_MAP : the team layout of the last block-scheduled epoch:
 *                      count = its workgroup count (read-only option
 *                      "teams_grid"), dst int32 -- team << 16 | member, -1
 *                      for an idle slot.  Teams of several wavefronts: entry
 *                      x * (count / xcds) + j is the j-th workgroup to start
 *                      on XCD x (each workgroup reads its XCD from the
 *                      hardware); one-wavefront teams: entry b is workgroup b.
 *   MFSGD_DBG_TEAM_SIZES : same layout, count = s, dst int32 -- workgroups
 *                      of each team.
 *   MFSGD_DBG_TABLE_STARTS : the global-table plan: count = s*s+1 (s =
 *                      "table_grid" of the plan), dst int64 -- first planned
 *                      position of block (I, J) at entry I*s+J, nnz at s*s.
 *   MFSGD_DBG_TABLE_ORDER  : same plan, count <= nnz, dst int64 -- position in
 *                      the caller's array of each planned sample (needs a plan
 *                      made while debug bit 0 was set).
 *   MFSGD_DBG_PRIORITY : the critical-path weights of the last pooled
 *                      block-scheduled epoch with "priority" on: count = s*s,
 *                      dst uint32 -- entry t*s + w for team t's block of wave
 *                      w: the largest number of 64-sample units (each block
 *                      rounded up) on a chain from that block to the end of
 *                      the epoch, where a block is followed by the same
 *                      team's block of the next wave and by the next wave's
 *                      block in its column.
 * dst may be host or device memory. */
enum {
    MFSGD_DBG_VISITS = 1,
    MFSGD_DBG_TRACE = 2,
    MFSGD_DBG_PLAN_STARTS = 3,
    MFSGD_DBG_PLAN_ORDER = 4,
    MFSGD_DBG_TEAM_MAP = 5,
    MFSGD_DBG_TEAM_SIZES = 6,
    MFSGD_DBG_TABLE_STARTS = 7,
    MFSGD_DBG_TABLE_ORDER = 8,
    MFSGD_DBG_PRIORITY = 9
};
int mfsgd_debug_read(int32_t what, void* dst, int64_t count, void* stream);

/* Release everything; the context returns to the un-initialised state. */
int mfsgd_finalize(void);

/* Text of the last failure in this thread ("" if none). */
const char* mfsgd_last_error(void);

/* Library version string. */
const char* mfsgd_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MFSGD_H */
