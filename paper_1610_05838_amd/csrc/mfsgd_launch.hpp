// mfsgd_launch.hpp -- host-side launch interface between the C-ABI layer and
// the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mfsgd {

struct Sample;

constexpr int kMaxGrid = 64;      // largest wavefront-update grid side s
constexpr int kRmseWaves = 2048;  // fixed, so the RMSE reduction order never changes
constexpr int kSchemeHogwild = 0;
constexpr int kSchemeWavefront = 1;
constexpr int kSchemeWaveLaunch = 2; // one deterministic wavefront-update wave per launch (cross-check)
// block-scheduled claim state: finished units and head claims per (team, wave), cursor per team, event counter,
// workgroups arrived per XCD, unit claims (after the head claims) per (team, wave)
constexpr int kSchedWords = 3 * kMaxGrid * kMaxGrid + kMaxGrid + 1 + kMaxGrid;

struct DebugSink;

struct EpochLaunch {
    int scheme;  // kSchemeHogwild, kSchemeWavefront or kSchemeWaveLaunch
    int KP;      // padded row width
    int depth;   // samples in flight per wavefront
    const Sample* S;
    int64_t nnz;
    int64_t W;   // batch-Hogwild! workers
    int f;       // batch size
    void* P;
    void* Q;
    float lr, lp, lq;
    int sync_every;  // one-address-space batch-Hogwild!: batches between XCD cache flushes (0 = none)
    int sync_l1;     // ... and whether the other wavefronts drop their CU's L1 then
    int nx;          // XCDs (one-address-space batch-Hogwild!: the first nx workgroups lead the flushes)
    int buf;         // every row offset of P and Q fits 31 bits: rows may be addressed through buffer descriptors
    int half;        // batch-Hogwild! at KP = 32: two workers per wavefront
    int atomic;      // block-scheduled epochs at depth 1: rows updated with atomic adds
    int coh;         // one-address-space batch-Hogwild!: coherence policy of rows that are not hot (kCoh*)
    int coh_p, coh_q;                 // ... applied to P's / Q's rows
    const uint32_t* hot_p;            // hot-row bits of P (nullptr: none)
    const uint32_t* hot_q;            // hot-row bits of Q
    // block-scheduled epochs
    const int64_t* bstart;
    int s;           // grid side
    int grid;        // workgroups launched
    int xslots;      // pooled teams: workgroup slots per XCD (tmap rows), 0: one-wavefront teams
    const int32_t* tmap;   // pooled: per (XCD, arrival slot) home team << 16 | member, or -1 (idle);
                           // one-wavefront teams: per workgroup
    const int32_t* xteams; // per XCD x: [x * (kMaxGrid + 1)] = team count, then the teams placed on x
    int pool;              // 1: a wavefront also serves the other teams of its XCD
    const uint32_t* prio;  // pooled: per (team, wave) t*s+w a critical-path weight, or nullptr
    int free_run;          // 1: blocks open without waiting for their column ticket
    int wg_waves;    // wavefronts per workgroup
    void* sink;      // grid * wg_waves * 2 * KP storage elements: rows for skipped stores (nullptr: no skipping)
    uint64_t sigma_c, sigma_o;
    uint32_t tail;   // pooled teams: units (64 samples) of a block claimed one at a time at its end (0: none)
    int wave;        // kSchemeWaveLaunch: the wave this launch runs
    uint32_t* tickets;
    uint32_t* sched; // claim state, kSchedWords entries (see k_blocked)
    uint32_t spin_limit;
    int* err;
    int32_t* trace_wave;
    // debug
    uint32_t* visits;
    const int64_t* orig;
    int32_t* trace_batch;
};

// Global scheduling table (LIBMF's policy, the baseline of section 3.2.1).
// tab, in 32-bit words: [0] ticket now served (the lock), [1] blocks not yet
// taken this epoch, [2] event counter (debug stamps), [3] next ticket,
// [kTableHdr, +s) row block in use,
// [kTableHdr + s, +s) column block in use, [kTableHdr + 2 s, + nb) the blocks
// not yet taken.
constexpr int kMaxTableGrid = 1024; // largest grid side of the table
constexpr int kTableHdr = 64;

struct TableLaunch {
    int KP, depth;
    const Sample* Sp;      // samples grouped by block
    const int64_t* bstart; // s*s+1 block starts
    int s;
    uint32_t nb;           // non-empty blocks (entries of the list)
    uint64_t draw;         // this epoch's stream of list positions
    void* P;
    void* Q;
    float lr, lp, lq;
    int f;
    int64_t W;             // workers (one wavefront each)
    uint32_t* tab;
    uint32_t spin_limit;
    int* err;
    // debug
    uint32_t* visits;
    const int64_t* orig;
    int32_t* trace;        // 3 per decision: block, claim stamp, release stamp
};

// Implemented per storage type in mfsgd_kernels_f32.hip / mfsgd_kernels_f16.hip.
hipError_t epoch_f32(const EpochLaunch& a, hipStream_t st);
hipError_t epoch_f16(const EpochLaunch& a, hipStream_t st);
hipError_t table_epoch_f32(const TableLaunch& a, hipStream_t st);
hipError_t table_epoch_f16(const TableLaunch& a, hipStream_t st);
// wavefronts of the one-address-space batch-Hogwild! kernel per CU (half: two workers per wavefront)
int occupancy_f32(int KP, int depth, int half);
int occupancy_f16(int KP, int depth, int half);
// workgroups per CU (half: the launch runs two batches per claim)
int occupancy_blocked_f32(int KP, int depth, int threads, int half);
int occupancy_blocked_f16(int KP, int depth, int threads, int half);
hipError_t rmse_partial_f32(int KP, const Sample* S, int64_t ntest, const void* P, const void* Q, double* partial,
                            hipStream_t st);
hipError_t rmse_partial_f16(int KP, const Sample* S, int64_t ntest, const void* P, const void* Q, double* partial,
                            hipStream_t st);
hipError_t init_f32(void* A, int64_t rows, int k, int KP, uint64_t stream, double inv_sqrt_k, hipStream_t st);
hipError_t init_f16(void* A, int64_t rows, int k, int KP, uint64_t stream, double inv_sqrt_k, hipStream_t st);

// Implemented in mfsgd_aux.hip (type-independent kernels).
hipError_t rmse_final(const double* partial, int64_t ntest, double* out, hipStream_t st);
hipError_t check_indices(const Sample* S, int64_t nnz, int64_t m, int64_t n, int* bad, hipStream_t st);
// zero the column tickets and the kSchedWords claim counters (a fill kernel, safe under graph capture)
hipError_t reset_tickets(uint32_t* tickets, uint32_t* sched, hipStream_t st);
hipError_t block_priority(const int64_t* bstart, int s, uint64_t sigma_c, uint64_t sigma_o, uint32_t* prio,
                          hipStream_t st);
// XCC id of each of `n` one-wavefront workgroups (to learn the dispatch layout)
hipError_t probe_xcc(int* out, int n, hipStream_t st);
// stable bucketing of samples into the s x s grid
struct PlanBuffers {
    int64_t* counts;     // s*s*chunks, bin-major
    int chunks;          // contiguous sample ranges counted and scattered in parallel (a multiple of 256)
    int64_t* totals;     // s*s
    int64_t* bstart;     // s*s+1
    Sample* Sp;          // planned copy
    int64_t* orig;       // planned position -> caller position (optional)
    int* bad;            // index-range flag
    const int64_t* rbnd; // balanced cut (s+1 user bounds), or nullptr for equal ranges
    const int64_t* cbnd; // s+1 item bounds
};
// per-index sample counts for the balanced cut (indices out of range raise *bad)
hipError_t plan_degrees(const Sample* S, int64_t nnz, int64_t m, int64_t n, unsigned long long* du,
                        unsigned long long* dv, int* bad, hipStream_t st);
// *out = max(*out, deg[0 .. rows-1]) (the caller zeroes *out first)
hipError_t max_degree(const unsigned long long* deg, int64_t rows, unsigned long long* out, hipStream_t st);
// bits[i / 32] bit i % 32 = (deg[i] >= thr), for rows 0 .. rows-1 (the last word's spare bits clear)
hipError_t hot_bits(const unsigned long long* deg, int64_t rows, unsigned long long thr, uint32_t* bits,
                    hipStream_t st);
// chunks of a plan: about one per kPlanChunkSamples samples, between
// kPlanChunksMin and kPlanChunksMax, and at most kPlanCountBytes of counts
constexpr int kPlanChunksMin = 2048;
constexpr int kPlanChunksMax = 16384;
constexpr int64_t kPlanChunkSamples = 65536;
constexpr int64_t kPlanCountBytes = int64_t(512) << 20;
// counts, per-block scans and block starts; raises *b.bad on an index out of range
hipError_t plan_build(const Sample* S, int64_t nnz, int64_t m, int64_t n, int s, const PlanBuffers& b,
                      hipStream_t st);
// scatter into the planned copy (run only after plan_build reported no bad index)
hipError_t plan_scatter(const Sample* S, int64_t nnz, int64_t m, int64_t n, int s, const PlanBuffers& b,
                        hipStream_t st);

// Global-table plan (mfsgd_table.hip): stable grouping of the samples by block
// floor(u*s/m) * s + floor(v*s/n) for s up to kMaxTableGrid, through a radix
// sort of (block id, position) pairs.  Needs nnz < 2^32.
struct TablePlanBuffers {
    uint32_t* keys[2]; // nnz each
    uint32_t* vals[2]; // nnz each
    void* temp;        // table_sort_bytes(nnz, s)
    size_t temp_bytes;
    int64_t* bstart;   // s*s+1
    Sample* Sp;        // planned copy
    int64_t* orig;     // planned position -> caller position (optional)
    int* bad;          // index-range flag
};
size_t table_sort_bytes(int64_t nnz, int s);
// keys, sort and block starts; raises *b.bad on an index out of range
hipError_t table_plan_build(const Sample* S, int64_t nnz, int64_t m, int64_t n, int s, const TablePlanBuffers& b,
                            hipStream_t st);
// gather into the planned copy (run only after table_plan_build reported no bad index)
hipError_t table_plan_gather(const Sample* S, int64_t nnz, const TablePlanBuffers& b, hipStream_t st);
// table state at the start of an epoch: lock free, every flag clear, the list
// = blist[0..nb) (the non-empty blocks, ascending)
hipError_t table_reset(uint32_t* tab, const uint32_t* blist, uint32_t nb, int s, hipStream_t st);

} // namespace mfsgd
