// mfsgd_api.hip -- the C ABI (include/mfsgd.h): context, argument checks,
// buffer ownership, plans, team layout, kernel selection and device-error
// reporting.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "mfsgd.h"
#include "mfsgd_device.hpp"
#include "mfsgd_launch.hpp"

// Scratch of mfsgd_rmse_noalloc: the kRmseWaves binary64 partial sums of the
// RMSE's first pass, in a fixed device array so that the call allocates
// nothing.  In host code `rmse_scratch` names a host-side stand-in; its device
// address, one per GPU, comes from hipGetSymbolAddress at mfsgd_init.
constexpr int kRmseScratchDoubles = 2048;
static __device__ __align__(256) double rmse_scratch[kRmseScratchDoubles];

namespace {

using namespace mfsgd;

static_assert(kRmseWaves <= kRmseScratchDoubles, "the RMSE partial sums must fit the no-alloc scratch");
constexpr int kMaxDevices = 64;
double* g_rmse_scratch[kMaxDevices] = {}; // device address of rmse_scratch per GPU

thread_local std::string g_err;

struct Options {
    int64_t dtype = MFSGD_FP32;
    int64_t batch_f = 256;
    int64_t workers = 0;
    int64_t depth = 0;
    int64_t team_waves = 0;
    int64_t partition = 2;
    int64_t hogwild_grid = 0;
    int64_t balance = 2;
    int64_t sync_every = 0;
    int64_t sync_l1 = 0;
    int64_t spin_limit = int64_t(1) << 24;
    int64_t skip_stores = 2;
    int64_t stage_samples = int64_t(1) << 25;
    int64_t wave_launch = 0;
    int64_t half_waves = 1;
    int64_t table_grid = 256;
    int64_t table_workers = 0;
    int64_t atomic = 0;
    int64_t priority = 1;
    int64_t tail_claims = 0;
    int64_t coherent = 0;
    int64_t coherent_mat = 3;
    int64_t hot_log2 = 0;
    int64_t debug = 0;
};

// Hot-row bits of one sample array (coherent one-address-space batch-Hogwild!):
// row i of P (Q) is hot when it holds at least nnz >> log2 of the samples.
struct HotSet {
    const mfsgd_sample* src = nullptr;
    int64_t nnz = -1;
    int log2 = -1;
    uint32_t* bits = nullptr; // ceil(m/32) words for P, then ceil(n/32) for Q
    int64_t bits_cap = 0;
    int64_t hot_p = 0, hot_q = 0; // rows marked
    bool matches(const mfsgd_sample* p, int64_t n, int l) const
    {
        return src == p && nnz == n && log2 == l && src != nullptr;
    }
};

// A grouping of one sample array into the blocks of an s x s grid.
struct Plan {
    const mfsgd_sample* src = nullptr;
    int64_t nnz = -1;
    int s = 0;
    bool balanced = false;
    bool has_orig = false;
    Sample* Sp = nullptr;
    int64_t Sp_cap = 0;
    int64_t* orig = nullptr;
    int64_t orig_cap = 0;
    int64_t* bstart = nullptr; // kMaxGrid^2 + 1
    std::vector<int64_t> hstart; // host copy of bstart[0 .. s*s]
    double hot_col = 0.0;        // largest share of a column block's samples held by one item
    double col_peak = 0.0;       // samples of the fullest column block over the mean column block
    double hot_row = 0.0;        // largest share of a row block's samples held by one user
    uint64_t version = 0;        // bumped by every build
    bool matches(const mfsgd_sample* p, int64_t n) const { return src == p && nnz == n && src != nullptr; }
    bool valid() const { return nnz >= 0 && bstart != nullptr; }
    void invalidate()
    {
        src = nullptr;
        nnz = -1;
    }
};

// The grouping of one sample array into the blocks of the global scheduling
// table's grid (equal index ranges), and the table's device state.
struct TablePlan {
    const mfsgd_sample* src = nullptr;
    int64_t nnz = -1;
    int s = 0;
    bool has_orig = false;
    Sample* Sp = nullptr;
    int64_t Sp_cap = 0;
    int64_t* orig = nullptr;
    int64_t orig_cap = 0;
    int64_t* bstart = nullptr;
    int64_t bstart_cap = 0;
    uint32_t* blist = nullptr; // the non-empty blocks, ascending
    int64_t blist_cap = 0;
    uint32_t nb = 0;
    uint32_t* tab = nullptr; // lock, counters, row/column marks, list (kTableHdr + 2 s + nb words)
    int64_t tab_cap = 0;
    bool matches(const mfsgd_sample* p, int64_t n) const { return src == p && nnz == n && src != nullptr; }
};

// The most samples any one user and any one item holds, for one sample array
// (the automatic batch-Hogwild! form).
struct RowStats {
    const mfsgd_sample* src = nullptr;
    int64_t nnz = -1;
    unsigned long long du = 0, dv = 0;
    bool matches(const mfsgd_sample* p, int64_t n) const { return src == p && nnz == n && src != nullptr; }
};

struct Context {
    bool inited = false;
    int device = 0;
    int cus = 0;
    int nx = 1;      // XCDs: distinct hardware XCD ids the init probe saw
    bool rr = false; // the probe's workgroups were dealt round-robin (b on XCD (b + o) mod nx)
    int64_t m = 0, n = 0;
    int k = 0, KP = 0, dtype = 0;
    uint64_t seed = 0;
    int64_t epoch = 0;
    void* P = nullptr;
    void* Q = nullptr;
    uint32_t* tickets = nullptr;
    uint32_t* prio = nullptr; // kMaxGrid^2: critical-path weight per (team, wave) of the last pooled epoch
    int prio_s = 0;           // its grid side (0: none yet)
    uint32_t* sched = nullptr; // block-scheduled claim state (kSchedWords)
    int* err = nullptr;
    int* bad = nullptr;
    double* partial = nullptr;
    double* dres = nullptr;
    double* hres = nullptr; // pinned
    int* hflag = nullptr;   // pinned
    Plan wf;                // the caller's wavefront-update plan (mfsgd_plan)
    Plan hw;                // internal plan of the XCD-partitioned batch-Hogwild!
    TablePlan gt;           // internal plan of the global scheduling table
    HotSet hot;             // hot rows of the last coherent batch-Hogwild! sample array
    RowStats stats;         // largest user and item sample counts of the last automatic batch-Hogwild! array
    unsigned long long* maxdeg = nullptr; // 2 device words for them
    int last_form = -1;     // form of the last batch-Hogwild! epoch (values of option "partition"), -1 before one
    int last_atomic = 0;    // whether it added its updates atomically
    int last_pairs = -1;    // whether the last block-scheduled epoch claimed two batches per wavefront, -1 before one
    // planner scratch
    int64_t* counts = nullptr;
    int64_t counts_cap = 0;
    int64_t* totals = nullptr;
    int64_t* bnd = nullptr; // 2 x (kMaxGrid + 1)
    unsigned long long* deg = nullptr;
    int64_t deg_cap = 0;
    // debug
    uint32_t* visits = nullptr;
    int64_t visits_cap = 0, visits_n = 0;
    int32_t* trace = nullptr;
    int64_t trace_cap = 0, trace_n = 0;
    // team layout of the last block-scheduled launch (device copy in tmap/tsize)
    int32_t* tmap = nullptr;
    int64_t tmap_cap = 0;
    int32_t* tsize = nullptr;
    int32_t* xteams = nullptr; // kMaxGrid * (kMaxGrid + 1): per XCD, team count then teams
    unsigned char* sink = nullptr; // rows for skipped stores, 2 per wavefront of the grid
    int64_t sink_cap = 0;
    // staged epochs: a ring of device buffers fed from host memory by a copy stream
    static constexpr int kStages = 3;
    Sample* stage_dev[kStages] = {};
    Sample* stage_host[kStages] = {}; // pinned, only for pageable caller arrays
    int64_t stage_dev_cap = 0, stage_host_cap = 0;
    hipStream_t copy_stream = nullptr;
    hipEvent_t ev_copied[kStages] = {}, ev_used[kStages] = {}, ev_start = nullptr;
    bool copied_pending[kStages] = {};
    const Plan* lay_plan = nullptr;
    uint64_t lay_version = 0;
    int64_t lay_want = -1;
    int lay_grid = 0, lay_waves = 0, lay_depth = 0, lay_half = -1, lay_xslots = 0;
};

Options g_opt;
Context g;

int fail(int code, const std::string& msg)
{
    g_err = msg;
    return code;
}

#define HIPCHK(call)                                                                                               \
    do {                                                                                                           \
        hipError_t e_ = (call);                                                                                    \
        if (e_ != hipSuccess)                                                                                      \
            return fail(MFSGD_EHIP, std::string(#call) + ": " + hipGetErrorString(e_));                          \
    } while (0)

#define CHK(expr)                                                                                                  \
    do {                                                                                                           \
        int rc_ = (expr);                                                                                          \
        if (rc_ != MFSGD_OK)                                                                                       \
            return rc_;                                                                                            \
    } while (0)

template <typename F>
int guarded(F&& f)
{
    try {
        g_err.clear();
        return f();
    } catch (const std::bad_alloc&) {
        return fail(MFSGD_ENOMEM, "host allocation failed");
    } catch (...) {
        return fail(MFSGD_EHIP, "unexpected exception");
    }
}

void dfree(void* p)
{
    if (p)
        (void)hipFree(p);
}

int dalloc(void** p, size_t bytes, const char* what)
{
    *p = nullptr;
    if (bytes == 0)
        bytes = 256;
    hipError_t e = hipMalloc(p, bytes);
    if (e != hipSuccess) {
        *p = nullptr;
        (void)hipGetLastError();
        return fail(MFSGD_ENOMEM, std::string("hipMalloc ") + what + " (" + std::to_string(bytes) +
                                      " bytes): " + hipGetErrorString(e));
    }
    return MFSGD_OK;
}

template <typename T>
int grow(T** p, int64_t* cap, int64_t need, const char* what)
{
    if (*cap >= need && *p)
        return MFSGD_OK;
    dfree(*p);
    *p = nullptr;
    *cap = 0;
    int rc = dalloc((void**)p, sizeof(T) * (size_t)(need > 0 ? need : 1), what);
    if (rc == MFSGD_OK)
        *cap = need;
    return rc;
}

void free_plan(Plan& p)
{
    dfree(p.Sp);
    dfree(p.orig);
    dfree(p.bstart);
    p = Plan();
}

void free_table_plan(TablePlan& p)
{
    dfree(p.Sp);
    dfree(p.orig);
    dfree(p.bstart);
    dfree(p.blist);
    dfree(p.tab);
    p = TablePlan();
}

void release_all()
{
    Context& c = g;
    dfree(c.P);
    dfree(c.Q);
    dfree(c.tickets);
    dfree(c.prio);
    dfree(c.sched);
    dfree(c.err);
    dfree(c.bad);
    dfree(c.partial);
    dfree(c.dres);
    if (c.hres)
        (void)hipHostFree(c.hres);
    if (c.hflag)
        (void)hipHostFree(c.hflag);
    free_plan(c.wf);
    free_plan(c.hw);
    free_table_plan(c.gt);
    dfree(c.counts);
    dfree(c.totals);
    dfree(c.bnd);
    dfree(c.deg);
    dfree(c.hot.bits);
    dfree(c.maxdeg);
    dfree(c.visits);
    dfree(c.trace);
    dfree(c.tmap);
    dfree(c.tsize);
    dfree(c.xteams);
    dfree(c.sink);
    for (int i = 0; i < Context::kStages; ++i) {
        dfree(c.stage_dev[i]);
        if (c.stage_host[i])
            (void)hipHostFree(c.stage_host[i]);
        if (c.ev_copied[i])
            (void)hipEventDestroy(c.ev_copied[i]);
        if (c.ev_used[i])
            (void)hipEventDestroy(c.ev_used[i]);
    }
    if (c.ev_start)
        (void)hipEventDestroy(c.ev_start);
    if (c.copy_stream)
        (void)hipStreamDestroy(c.copy_stream);
    c = Context();
}

size_t elem_size(int dtype) { return dtype == MFSGD_FP16 ? 2 : 4; }

int padded_width(int k)
{
    if (k <= 32)
        return 32;
    if (k <= 64)
        return 64;
    if (k <= 128)
        return 128;
    if (k <= 256)
        return 256;
    return 512;
}

// Whether one-address-space batch-Hogwild! runs two workers per wavefront.
// By default (half_waves = 1) at KP = 32, where one worker per wavefront
// leaves half of the lanes idle.  Wider rows (half_waves = 2: every width of
// at most 16 bytes per half-wavefront lane) were no faster per epoch on the
// Netflix shape except binary16 at KP = 64, and twice the workers converge
// worse per epoch, so they are not the default.  0: never.
bool half_wave_workers(int KP, int dtype)
{
    if (g_opt.half_waves == 0)
        return false;
    if (g_opt.half_waves == 2)
        return (int64_t)KP * (int64_t)elem_size(dtype) <= 16 * 32;
    return KP == 32;
}

int occupancy_waves(int KP, int dtype, int depth)
{
    const int half = half_wave_workers(KP, dtype) ? 1 : 0;
    return dtype == MFSGD_FP16 ? occupancy_f16(KP, depth, half) : occupancy_f32(KP, depth, half);
}

int occupancy_blocked(int KP, int dtype, int depth, int threads, bool half = false)
{
    return dtype == MFSGD_FP16 ? occupancy_blocked_f16(KP, depth, threads, half ? 1 : 0)
                               : occupancy_blocked_f32(KP, depth, threads, half ? 1 : 0);
}

// Read back and clear the device error flag; the stream has been synchronised.
int take_device_error()
{
    if (*g.hflag) {
        *g.hflag = 0;
        int zero = 0;
        HIPCHK(hipMemcpy(g.err, &zero, sizeof(int), hipMemcpyHostToDevice));
        return fail(MFSGD_ETIMEOUT, "a block-schedule ticket wait exceeded spin_limit; the epoch was abandoned");
    }
    return MFSGD_OK;
}

int sync_and_check(hipStream_t st)
{
    HIPCHK(hipMemcpyAsync(g.hflag, g.err, sizeof(int), hipMemcpyDeviceToHost, st));
    HIPCHK(hipStreamSynchronize(st));
    return take_device_error();
}

bool valid_samples(const mfsgd_sample* s, int64_t nnz) { return nnz >= 0 && (nnz == 0 || s != nullptr); }

// whether every row of P and Q starts below 2^31 bytes (buffer addressing)
bool rows_fit_31_bits()
{
    const int64_t row = (int64_t)g.KP * (int64_t)elem_size(g.dtype);
    return std::max(g.m, g.n) * row <= (int64_t(1) << 31);
}

// The batch-Hogwild! forms (option "partition").  Each XCD's L2 is a
// write-back cache the other XCDs do not see inside a kernel, so lock-free
// updates of one row made on two XCDs land in separate copies and the copy
// written back last wins, and inside one L2 two workers that update one row
// at once keep only the later store.  Measured against the serial oracle:
//   * one address space over all XCDs (0): the per-XCD copies of popular rows
//     trail the serial order (Netflix shape, 20 epochs: 0.017 in test RMSE);
//   * XCD-partitioned (1, 3): a coarse block order that trails by 0.05;
//   * one XCD (4): every update meets in one L2; where a few rows hold a
//     large share of the samples and the learning rate decays (Netflix
//     shape) it ends within 1e-3 of the serial oracle, but where many rows
//     are moderately popular and the rate stays constant (Yahoo shape) the
//     stores that overwrite concurrent updates of the same row make it fall
//     behind epoch after epoch;
//   * one address space with atomic adds of every change (0 with option
//     "atomic"): no update is lost -- the Hogwild! model of component-wise
//     atomic updates -- and the Yahoo-shaped run follows the serial oracle to
//     1e-4, but the adds of one row meet at one memory channel, which the
//     hottest Netflix-shaped rows saturate.
// The automatic form (2, the default) therefore takes one XCD when the most
// popular user or item holds more than 1/kOneXcdShareInv of the samples and
// atomic adds over all XCDs otherwise; both run one sample in flight per
// wavefront and at most min(m, n) / 20 workers (the paper's empirical
// Hogwild! condition, section 5.5.1).
constexpr int kOneXcdShareInv = 64;

// Wavefront-update plans whose fullest column block holds at most this many
// times the mean run two batches per claim at rows wider than 32 values.
constexpr double kPairsColumnPeak = 2.0;

bool partitioned_hogwild()
{
    if (g.last_form >= 0)
        return g.last_form != 0;
    return g_opt.partition == 1 || g_opt.partition == 3 || g_opt.partition == 4;
}

// grid side of the block-scheduled batch-Hogwild! plan of form `form`
int hogwild_grid_side(int form)
{
    if (form == 4)
        return 1;
    return g_opt.hogwild_grid > 0 ? (int)g_opt.hogwild_grid : std::max(1, g.nx);
}

// workers of the automatic forms: the paper's Hogwild! condition
int64_t hogwild_condition_workers() { return std::max<int64_t>(1, std::min(g.m, g.n) / 20); }

// samples in flight per wavefront: the option, or automatically 1 for
// batch-Hogwild! in one XCD (bound by that XCD's bandwidth, not by latency:
// depth 1 runs as fast and halves the updates in flight) and 2 elsewhere
int depth_for(bool hogwild_one_xcd)
{
    if (g_opt.depth > 0)
        return (int)g_opt.depth;
    return hogwild_one_xcd ? 1 : 2;
}

// ---------------------------------------------------------------------------
// options
// ---------------------------------------------------------------------------
struct OptSpec {
    const char* key;
    int64_t Options::*field;
    int64_t lo, hi;
    const char* what;
};

const OptSpec kOpts[] = {
    {"dtype", &Options::dtype, 0, 1, "dtype must be 0 (fp32) or 1 (fp16)"},
    {"batch_f", &Options::batch_f, 64, int64_t(1) << 30, "batch_f must be a positive multiple of 64"},
    {"workers", &Options::workers, 0, int64_t(1) << 30, "workers must be in [0, 2^30]"},
    {"depth", &Options::depth, 0, 8, "depth must be 0 (automatic), 1, 2, 4 or 8"},
    {"team_waves", &Options::team_waves, 0, 65536, "team_waves must be in [0, 65536]"},
    {"partition", &Options::partition, 0, 4, "partition must be 0, 1, 2, 3 or 4"},
    {"hogwild_grid", &Options::hogwild_grid, 0, kMaxGrid, "hogwild_grid must be in [0, 64]"},
    {"balance", &Options::balance, 0, 2, "balance must be 0, 1 or 2"},
    {"sync_every", &Options::sync_every, 0, int64_t(1) << 30, "sync_every must be in [0, 2^30]"},
    {"sync_l1", &Options::sync_l1, 0, 1, "sync_l1 must be 0 or 1"},
    {"spin_limit", &Options::spin_limit, 1, 0xffffffffll, "spin_limit must be in [1, 2^32-1]"},
    {"skip_stores", &Options::skip_stores, 0, 2, "skip_stores must be 0, 1 or 2"},
    {"stage_samples", &Options::stage_samples, 64, int64_t(1) << 31, "stage_samples must be in [64, 2^31]"},
    {"wave_launch", &Options::wave_launch, 0, 1, "wave_launch must be 0 or 1"},
    {"half_waves", &Options::half_waves, 0, 2, "half_waves must be 0, 1 or 2"},
    {"table_grid", &Options::table_grid, 1, kMaxTableGrid, "table_grid must be in [1, 1024]"},
    {"table_workers", &Options::table_workers, 0, 65536, "table_workers must be in [0, 65536]"},
    {"atomic", &Options::atomic, 0, 1, "atomic must be 0 or 1"},
    {"priority", &Options::priority, 0, 1, "priority must be 0 or 1"},
    {"tail_claims", &Options::tail_claims, 0, 1, "tail_claims must be 0 or 1"},
    {"coherent", &Options::coherent, 0, 4, "coherent must be in [0, 4]"},
    {"coherent_mat", &Options::coherent_mat, 0, 3, "coherent_mat must be in [0, 3]"},
    {"hot_log2", &Options::hot_log2, 0, 62, "hot_log2 must be in [0, 62]"},
    {"debug", &Options::debug, 0, 3, "debug must be in [0, 3]"},
};

int set_option_impl(const char* key, int64_t value)
{
    if (!key)
        return fail(MFSGD_EINVAL, "option key is NULL");
    for (const OptSpec& o : kOpts) {
        if (std::strcmp(key, o.key) != 0)
            continue;
        bool ok = value >= o.lo && value <= o.hi;
        if (ok && o.field == &Options::batch_f)
            ok = value % 64 == 0;
        if (ok && o.field == &Options::depth)
            ok = value == 0 || value == 1 || value == 2 || value == 4 || value == 8;
        if (!ok)
            return fail(MFSGD_EINVAL, o.what);
        g_opt.*(o.field) = value;
        return MFSGD_OK;
    }
    return fail(MFSGD_EINVAL, std::string("unknown option '") + key + "'");
}

int get_option_impl(const char* key, int64_t* value)
{
    if (!key || !value)
        return fail(MFSGD_EINVAL, "NULL argument");
    for (const OptSpec& o : kOpts)
        if (std::strcmp(key, o.key) == 0) {
            *value = g_opt.*(o.field);
            return MFSGD_OK;
        }
    const bool ro = !std::strcmp(key, "resident_waves") || !std::strcmp(key, "xcds") || !std::strcmp(key, "cus") ||
                    !std::strcmp(key, "blocked_per_cu") || !std::strcmp(key, "partitioned") ||
                    !std::strcmp(key, "teams_grid") || !std::strcmp(key, "table_blocks") ||
                    !std::strcmp(key, "half_workers") || !std::strcmp(key, "hogwild_form") ||
                    !std::strcmp(key, "hogwild_atomic") || !std::strcmp(key, "xcd_round_robin") ||
                    !std::strcmp(key, "blocked_pairs");
    if (!ro)
        return fail(MFSGD_EINVAL, std::string("unknown option '") + key + "'");
    if (!g.inited)
        return fail(MFSGD_ESTATE, std::string("'") + key + "' is read-only and needs mfsgd_init");
    if (!std::strcmp(key, "resident_waves"))
        *value = (int64_t)g.cus * occupancy_waves(g.KP, g.dtype, depth_for(false));
    else if (!std::strcmp(key, "xcds"))
        *value = g.nx;
    else if (!std::strcmp(key, "xcd_round_robin"))
        *value = g.rr ? 1 : 0;
    else if (!std::strcmp(key, "half_workers"))
        *value = half_wave_workers(g.KP, g.dtype) ? 1 : 0;
    else if (!std::strcmp(key, "blocked_per_cu"))
        *value = occupancy_blocked(g.KP, g.dtype, depth_for(g_opt.partition == 2 || g_opt.partition == 4), 256);
    else if (!std::strcmp(key, "partitioned"))
        *value = partitioned_hogwild() ? 1 : 0;
    else if (!std::strcmp(key, "hogwild_form"))
        *value = g.last_form;
    else if (!std::strcmp(key, "hogwild_atomic"))
        *value = g.last_atomic;
    else if (!std::strcmp(key, "blocked_pairs"))
        *value = g.last_pairs;
    else if (!std::strcmp(key, "teams_grid"))
        *value = g.lay_plan ? g.lay_grid : 0;
    else if (!std::strcmp(key, "table_blocks"))
        *value = g.gt.nnz >= 0 ? (int64_t)g.gt.nb : 0;
    else
        *value = g.cus;
    return MFSGD_OK;
}

// ---------------------------------------------------------------------------
// init
// ---------------------------------------------------------------------------
int detect_xcds(Context& c)
{
    // Deal 64 workgroups and read which XCD each runs on; round-robin dealing
    // (workgroup b on XCD b mod nx) is what the team layout relies on.
    constexpr int kProbe = 64;
    int* dev = nullptr;
    CHK(dalloc((void**)&dev, sizeof(int) * kProbe, "xcd probe"));
    std::vector<int> host(kProbe, -1);
    hipError_t e = probe_xcc(dev, kProbe, nullptr);
    if (e == hipSuccess)
        e = hipMemcpy(host.data(), dev, sizeof(int) * kProbe, hipMemcpyDeviceToHost);
    dfree(dev);
    if (e != hipSuccess)
        return fail(MFSGD_EHIP, std::string("XCD probe: ") + hipGetErrorString(e));
    // the number of XCDs: the largest id among 64 one-wavefront workgroups
    // plus one.  The block-scheduled kernel reads each workgroup's XCD from
    // the hardware itself, so it needs only this count, whatever order the
    // dispatcher deals the workgroups in; whether that order was round-robin
    // (starting wherever the previous launch left off) is kept for the
    // epoch kernel's optional periodic cache flushes, led by the first nx
    // workgroups of its grid.
    const int top = *std::max_element(host.begin(), host.end());
    if (*std::min_element(host.begin(), host.end()) < 0 || top >= kMaxGrid)
        return fail(MFSGD_EHIP, "XCD probe: unexpected XCD id");
    c.nx = top + 1;
    bool round_robin = true;
    for (int b = 0; round_robin && b < kProbe; ++b)
        round_robin = host[b] == (host[0] + b) % c.nx;
    c.rr = round_robin;
    return MFSGD_OK;
}

int init_impl(int64_t m, int64_t n, int32_t k, uint64_t seed)
{
    if (m < 1 || n < 1 || m > INT32_MAX || n > INT32_MAX)
        return fail(MFSGD_EINVAL, "m and n must be in [1, 2^31-1]");
    if (k < 1 || k > 512)
        return fail(MFSGD_EINVAL, "k must be in [1, 512]");
    release_all();
    Context& c = g;
    c.last_form = -1;
    c.last_atomic = 0;
    c.last_pairs = -1;
    c.stats = RowStats();
    HIPCHK(hipGetDevice(&c.device));
    if (c.device >= 0 && c.device < kMaxDevices && !g_rmse_scratch[c.device]) {
        void* sp = nullptr;
        HIPCHK(hipGetSymbolAddress(&sp, HIP_SYMBOL(rmse_scratch)));
        g_rmse_scratch[c.device] = (double*)sp;
    }
    HIPCHK(hipDeviceGetAttribute(&c.cus, hipDeviceAttributeMultiprocessorCount, c.device));
    c.m = m;
    c.n = n;
    c.k = k;
    c.KP = padded_width(k);
    c.dtype = (int)g_opt.dtype;
    c.seed = seed;
    c.epoch = 0;
    const size_t es = elem_size(c.dtype);
    int rc;
    if ((rc = dalloc(&c.P, (size_t)m * c.KP * es, "P")) || (rc = dalloc(&c.Q, (size_t)n * c.KP * es, "Q")) ||
        (rc = dalloc((void**)&c.tickets, sizeof(uint32_t) * kMaxGrid, "tickets")) ||
        (rc = dalloc((void**)&c.prio, sizeof(uint32_t) * kMaxGrid * kMaxGrid, "block priorities")) ||
        (rc = dalloc((void**)&c.sched, sizeof(uint32_t) * kSchedWords, "claim counters")) ||
        (rc = dalloc((void**)&c.err, sizeof(int), "flag")) || (rc = dalloc((void**)&c.bad, sizeof(int), "flag")) ||
        (rc = dalloc((void**)&c.partial, sizeof(double) * kRmseWaves, "rmse partials")) ||
        (rc = dalloc((void**)&c.dres, sizeof(double), "rmse result")) ||
        (rc = dalloc((void**)&c.bnd, sizeof(int64_t) * 2 * (kMaxGrid + 1), "plan bounds"))) {
        release_all();
        return rc;
    }
    if (hipHostMalloc((void**)&c.hres, sizeof(double), hipHostMallocDefault) != hipSuccess ||
        hipHostMalloc((void**)&c.hflag, sizeof(int), hipHostMallocDefault) != hipSuccess) {
        (void)hipGetLastError();
        release_all();
        return fail(MFSGD_ENOMEM, "pinned host allocation failed");
    }
    *c.hflag = 0;
    HIPCHK(hipMemset(c.err, 0, sizeof(int)));
    HIPCHK(hipMemset(c.bad, 0, sizeof(int)));
    HIPCHK(reset_tickets(c.tickets, c.sched, nullptr));
    const double inv_sqrt_k = 1.0 / std::sqrt((double)k);
    const uint64_t sp = sm64_at(seed, kTagP), sq = sm64_at(seed, kTagQ);
    if (c.dtype == MFSGD_FP16) {
        HIPCHK(init_f16(c.P, m, k, c.KP, sp, inv_sqrt_k, nullptr));
        HIPCHK(init_f16(c.Q, n, k, c.KP, sq, inv_sqrt_k, nullptr));
    } else {
        HIPCHK(init_f32(c.P, m, k, c.KP, sp, inv_sqrt_k, nullptr));
        HIPCHK(init_f32(c.Q, n, k, c.KP, sq, inv_sqrt_k, nullptr));
    }
    CHK(detect_xcds(c));
    HIPCHK(hipDeviceSynchronize());
    c.inited = true;
    return MFSGD_OK;
}

// ---------------------------------------------------------------------------
// plans
// ---------------------------------------------------------------------------
// Optimal consecutive cut of per-index counts into s ranges: the smallest cap
// on a range's count for which a greedy fill needs at most s ranges, and the
// ranges of that greedy fill.  pre[i] = count of indices 0..i-1; a greedy
// range starting at index b ends before the first e > b with
// pre[e+1] - pre[b] > cap, found by binary search, so one fill costs
// O(s log N) instead of O(N).
int64_t greedy_ranges(const std::vector<int64_t>& pre, int64_t cap, int s, int64_t* bounds)
{
    const int64_t N = (int64_t)pre.size() - 1;
    int64_t k = 0, b = 0;
    if (bounds)
        bounds[0] = 0;
    while (true) {
        // first e in (b, N] with pre[e] - pre[b] > cap ends the range at e - 1 (range = [b, e-1))
        const int64_t lim = pre[b] + cap;
        const int64_t e = std::upper_bound(pre.begin() + b + 1, pre.end(), lim) - pre.begin();
        // indices b .. e-2 fit; index e-1 would overflow (or e = N + 1: all fit)
        const int64_t next = std::max<int64_t>(e - 1, b + 1);
        if (next >= N)
            break;
        ++k;
        if (k > s && !bounds)
            return k + 1; // infeasible; exact count not needed
        if (bounds && k <= s)
            bounds[k] = next;
        b = next;
    }
    if (bounds)
        for (int64_t j = k + 1; j <= s; ++j)
            bounds[j] = N;
    return k + 1;
}

void balanced_cut(const std::vector<unsigned long long>& cnt, int64_t nnz, int s, int64_t* bounds)
{
    std::vector<int64_t> pre(cnt.size() + 1, 0);
    int64_t top = 0;
    for (size_t i = 0; i < cnt.size(); ++i) {
        pre[i + 1] = pre[i] + (int64_t)cnt[i];
        top = std::max<int64_t>(top, (int64_t)cnt[i]);
    }
    int64_t lo = std::max<int64_t>((nnz + s - 1) / s, top);
    int64_t hi = std::max<int64_t>(nnz, lo);
    while (lo < hi) {
        const int64_t mid = lo + (hi - lo) / 2;
        if (greedy_ranges(pre, mid, s, nullptr) <= s)
            hi = mid;
        else
            lo = mid + 1;
    }
    greedy_ranges(pre, lo, s, bounds);
}

// Whether an s x s grid is cut by sample counts (option "balance"; automatic:
// when no XCD hosts two of its workers).
bool balanced_grid(int s)
{
    return g_opt.balance == 1 || (g_opt.balance == 2 && s <= std::max(1, g.nx));
}

int bad_index_error()
{
    return fail(MFSGD_EINVAL, "a sample index is out of range (need 0 <= u < m and 0 <= v < n)");
}

// Largest user and item sample counts of a sample array (cached per array).
int row_stats(const mfsgd_sample* samples, int64_t nnz, hipStream_t st)
{
    Context& c = g;
    if (c.stats.matches(samples, nnz))
        return MFSGD_OK;
    c.stats.src = nullptr;
    CHK(grow(&c.deg, &c.deg_cap, c.m + c.n, "plan degrees"));
    if (!c.maxdeg)
        CHK(dalloc((void**)&c.maxdeg, 2 * sizeof(unsigned long long), "largest degrees"));
    HIPCHK(hipMemsetAsync(c.bad, 0, sizeof(int), st));
    HIPCHK(hipMemsetAsync(c.deg, 0, sizeof(unsigned long long) * (size_t)(c.m + c.n), st));
    HIPCHK(hipMemsetAsync(c.maxdeg, 0, 2 * sizeof(unsigned long long), st));
    HIPCHK(plan_degrees((const Sample*)samples, nnz, c.m, c.n, c.deg, c.deg + c.m, c.bad, st));
    HIPCHK(max_degree(c.deg, c.m, c.maxdeg, st));
    HIPCHK(max_degree(c.deg + c.m, c.n, c.maxdeg + 1, st));
    unsigned long long h[2] = {0, 0};
    HIPCHK(hipMemcpyAsync(h, c.maxdeg, sizeof(h), hipMemcpyDeviceToHost, st));
    HIPCHK(hipMemcpyAsync(c.hflag, c.bad, sizeof(int), hipMemcpyDeviceToHost, st));
    HIPCHK(hipStreamSynchronize(st));
    if (*c.hflag) {
        *c.hflag = 0;
        return bad_index_error();
    }
    c.stats.du = h[0];
    c.stats.dv = h[1];
    c.stats.src = samples;
    c.stats.nnz = nnz;
    return MFSGD_OK;
}

// Hot-row bits of a sample array: per-index sample counts (the planner's
// degree kernel), then one bit per row of P and of Q.
int build_hot(const mfsgd_sample* samples, int64_t nnz, int log2, hipStream_t st)
{
    Context& c = g;
    HotSet& h = c.hot;
    h.src = nullptr;
    const int64_t wp = (c.m + 31) / 32, wq = (c.n + 31) / 32;
    CHK(grow(&h.bits, &h.bits_cap, wp + wq, "hot-row bits"));
    CHK(grow(&c.deg, &c.deg_cap, c.m + c.n, "plan degrees"));
    HIPCHK(hipMemsetAsync(c.bad, 0, sizeof(int), st));
    HIPCHK(hipMemsetAsync(c.deg, 0, sizeof(unsigned long long) * (size_t)(c.m + c.n), st));
    HIPCHK(plan_degrees((const Sample*)samples, nnz, c.m, c.n, c.deg, c.deg + c.m, c.bad, st));
    const unsigned long long thr = std::max<unsigned long long>(1ull, (unsigned long long)nnz >> log2);
    HIPCHK(hot_bits(c.deg, c.m, thr, h.bits, st));
    HIPCHK(hot_bits(c.deg + c.m, c.n, thr, h.bits + wp, st));
    HIPCHK(hipMemcpyAsync(c.hflag, c.bad, sizeof(int), hipMemcpyDeviceToHost, st));
    HIPCHK(hipStreamSynchronize(st));
    if (*c.hflag) {
        *c.hflag = 0;
        return bad_index_error();
    }
    h.src = samples;
    h.nnz = nnz;
    h.log2 = log2;
    return MFSGD_OK;
}

int build_plan(Plan& pl, const mfsgd_sample* samples, int64_t nnz, int s, bool balanced, bool keep_orig,
               hipStream_t st)
{
    Context& c = g;
    pl.invalidate();
    // chunks: enough wavefronts to hide the scatter's latency on large sample arrays
    int64_t chunks = (nnz + kPlanChunkSamples - 1) / kPlanChunkSamples;
    chunks = std::min<int64_t>(std::max<int64_t>(chunks, kPlanChunksMin), kPlanChunksMax);
    chunks = std::min<int64_t>(chunks, kPlanCountBytes / (int64_t)(sizeof(int64_t) * s * s));
    chunks = std::max<int64_t>(256, chunks / 256 * 256);
    CHK(grow(&c.counts, &c.counts_cap, (int64_t)s * s * chunks, "plan counts"));
    if (!c.totals)
        CHK(dalloc((void**)&c.totals, sizeof(int64_t) * kMaxGrid * kMaxGrid, "plan totals"));
    if (!pl.bstart)
        CHK(dalloc((void**)&pl.bstart, sizeof(int64_t) * (kMaxGrid * kMaxGrid + 1), "plan starts"));
    CHK(grow(&pl.Sp, &pl.Sp_cap, nnz, "planned samples"));
    if (keep_orig)
        CHK(grow(&pl.orig, &pl.orig_cap, nnz, "plan positions"));
    const Sample* S = (const Sample*)samples;
    HIPCHK(hipMemsetAsync(c.bad, 0, sizeof(int), st));
    const int64_t* rbnd = nullptr;
    const int64_t* cbnd = nullptr;
    // per-index sample counts: the balanced cut and the hot-row and
    // hot-column measures below need both
    CHK(grow(&c.deg, &c.deg_cap, c.m + c.n, "plan degrees"));
    HIPCHK(hipMemsetAsync(c.deg, 0, sizeof(unsigned long long) * (size_t)(c.m + c.n), st));
    HIPCHK(plan_degrees(S, nnz, c.m, c.n, c.deg, c.deg + c.m, c.bad, st));
    std::vector<unsigned long long> du((size_t)c.m), dv((size_t)c.n);
    HIPCHK(hipMemcpyAsync(du.data(), c.deg, sizeof(unsigned long long) * du.size(), hipMemcpyDeviceToHost, st));
    HIPCHK(hipMemcpyAsync(dv.data(), c.deg + c.m, sizeof(unsigned long long) * dv.size(), hipMemcpyDeviceToHost, st));
    HIPCHK(hipMemcpyAsync(c.hflag, c.bad, sizeof(int), hipMemcpyDeviceToHost, st));
    HIPCHK(hipStreamSynchronize(st));
    if (*c.hflag) {
        *c.hflag = 0;
        return bad_index_error();
    }
    std::vector<int64_t> cut(2 * (kMaxGrid + 1));
    int64_t* ccut = cut.data() + kMaxGrid + 1;
    if (balanced) {
        balanced_cut(du, nnz, s, cut.data());
        balanced_cut(dv, nnz, s, ccut);
        HIPCHK(hipMemcpy(c.bnd, cut.data(), sizeof(int64_t) * cut.size(), hipMemcpyHostToDevice));
        rbnd = c.bnd;
        cbnd = c.bnd + kMaxGrid + 1;
    } else {
        for (int j = 0; j <= s; ++j) { // first index of each equal range floor(x*s/N) = j
            cut[j] = (int64_t)((j * c.m + s - 1) / s);
            ccut[j] = (int64_t)((j * c.n + s - 1) / s);
        }
    }
    // Largest share of one block row's (column's) samples that a single user
    // (item) holds.
    auto hottest = [s](const std::vector<unsigned long long>& d, const int64_t* bnd) {
        double h = 0.0;
        for (int j = 0; j < s; ++j) {
            unsigned long long tot = 0, top = 0;
            for (int64_t x = bnd[j]; x < bnd[j + 1]; ++x) {
                tot += d[(size_t)x];
                top = std::max(top, d[(size_t)x]);
            }
            if (tot > 0)
                h = std::max(h, (double)top / (double)tot);
        }
        return h;
    };
    pl.hot_row = hottest(du, cut.data());
    pl.hot_col = hottest(dv, ccut);
    PlanBuffers b{c.counts, (int)chunks, c.totals, pl.bstart, pl.Sp, keep_orig ? pl.orig : nullptr, c.bad, rbnd, cbnd};
    HIPCHK(plan_build(S, nnz, c.m, c.n, s, b, st));
    HIPCHK(hipMemcpyAsync(c.hflag, c.bad, sizeof(int), hipMemcpyDeviceToHost, st));
    HIPCHK(hipStreamSynchronize(st));
    const int bad = *c.hflag;
    *c.hflag = 0;
    if (bad)
        return bad_index_error();
    HIPCHK(plan_scatter(S, nnz, c.m, c.n, s, b, st));
    pl.hstart.assign((size_t)s * s + 1, 0);
    HIPCHK(hipMemcpyAsync(pl.hstart.data(), pl.bstart, sizeof(int64_t) * pl.hstart.size(), hipMemcpyDeviceToHost,
                          st));
    HIPCHK(hipStreamSynchronize(st));
    {
        int64_t top = 0;
        for (int j = 0; j < s; ++j) {
            int64_t col = 0;
            for (int t = 0; t < s; ++t)
                col += pl.hstart[(size_t)t * s + j + 1] - pl.hstart[(size_t)t * s + j];
            top = std::max(top, col);
        }
        pl.col_peak = nnz > 0 ? (double)top * s / (double)nnz : 0.0;
    }
    pl.version += 1;
    pl.src = samples;
    pl.nnz = nnz;
    pl.s = s;
    pl.balanced = balanced;
    pl.has_orig = keep_orig;
    return MFSGD_OK;
}

// Group the samples by block of the table's s x s grid (equal index ranges),
// keep the non-empty block list, size the table.  Synchronous.
int build_table_plan(TablePlan& pl, const mfsgd_sample* samples, int64_t nnz, int s, bool keep_orig, hipStream_t st)
{
    Context& c = g;
    pl.src = nullptr;
    pl.nnz = -1;
    const int64_t nblocks = (int64_t)s * s;
    CHK(grow(&pl.Sp, &pl.Sp_cap, nnz, "table samples"));
    if (keep_orig)
        CHK(grow(&pl.orig, &pl.orig_cap, nnz, "table positions"));
    CHK(grow(&pl.bstart, &pl.bstart_cap, nblocks + 1, "table block starts"));
    TablePlanBuffers b{};
    b.bstart = pl.bstart;
    b.Sp = pl.Sp;
    b.orig = keep_orig ? pl.orig : nullptr;
    b.bad = c.bad;
    // sort scratch, released again below
    std::vector<void*> scratch;
    auto take = [&](void** p, size_t bytes, const char* what) {
        int rc = dalloc(p, bytes, what);
        if (rc == MFSGD_OK)
            scratch.push_back(*p);
        return rc;
    };
    auto drop = [&]() {
        for (void* p : scratch)
            dfree(p);
        scratch.clear();
    };
    int rc = MFSGD_OK;
    const size_t words = sizeof(uint32_t) * (size_t)std::max<int64_t>(nnz, 1);
    b.temp_bytes = table_sort_bytes(nnz, s);
    if (nnz > 0 && b.temp_bytes == 0)
        rc = fail(MFSGD_EHIP, "radix sort size query failed");
    for (int i = 0; rc == MFSGD_OK && i < 2; ++i) {
        rc = take((void**)&b.keys[i], words, "table sort keys");
        if (rc == MFSGD_OK)
            rc = take((void**)&b.vals[i], words, "table sort values");
    }
    if (rc == MFSGD_OK)
        rc = take(&b.temp, b.temp_bytes, "table sort scratch");
    hipError_t e = hipSuccess;
    if (rc == MFSGD_OK) {
        e = hipMemsetAsync(c.bad, 0, sizeof(int), st);
        if (e == hipSuccess)
            e = table_plan_build((const Sample*)samples, nnz, c.m, c.n, s, b, st);
        if (e == hipSuccess)
            e = hipMemcpyAsync(c.hflag, c.bad, sizeof(int), hipMemcpyDeviceToHost, st);
        if (e == hipSuccess)
            e = hipStreamSynchronize(st);
        if (e == hipSuccess && *c.hflag) {
            *c.hflag = 0;
            rc = bad_index_error();
        } else if (e == hipSuccess) {
            e = table_plan_gather((const Sample*)samples, nnz, b, st);
            if (e == hipSuccess)
                e = hipStreamSynchronize(st);
        }
        if (e != hipSuccess)
            rc = fail(MFSGD_EHIP, std::string("table plan: ") + hipGetErrorString(e));
    }
    drop();
    if (rc != MFSGD_OK)
        return rc;
    std::vector<int64_t> hstart((size_t)nblocks + 1);
    HIPCHK(hipMemcpy(hstart.data(), pl.bstart, sizeof(int64_t) * hstart.size(), hipMemcpyDeviceToHost));
    std::vector<uint32_t> blist;
    for (int64_t x = 0; x < nblocks; ++x)
        if (hstart[(size_t)x + 1] > hstart[(size_t)x])
            blist.push_back((uint32_t)x);
    CHK(grow(&pl.blist, &pl.blist_cap, (int64_t)blist.size(), "table block list"));
    if (!blist.empty())
        HIPCHK(hipMemcpy(pl.blist, blist.data(), sizeof(uint32_t) * blist.size(), hipMemcpyHostToDevice));
    CHK(grow(&pl.tab, &pl.tab_cap, kTableHdr + 2 * (int64_t)s + (int64_t)blist.size(), "scheduling table"));
    pl.nb = (uint32_t)blist.size();
    pl.src = samples;
    pl.nnz = nnz;
    pl.s = s;
    pl.has_orig = keep_orig;
    return MFSGD_OK;
}

// One epoch under the global scheduling table (see k_table).
int table_epoch(const mfsgd_sample* samples, int64_t nnz, float lr, float lp, float lq, hipStream_t st)
{
    Context& c = g;
    const int64_t dbg = g_opt.debug;
    if (nnz >= (int64_t(1) << 32))
        return fail(MFSGD_EINVAL, "the global scheduling table handles fewer than 2^32 samples");
    const int s = (int)g_opt.table_grid;
    const bool keep = (dbg & 1) != 0;
    TablePlan& pl = c.gt;
    if (!pl.matches(samples, nnz) || pl.s != s || (keep && !pl.has_orig))
        CHK(build_table_plan(pl, samples, nnz, s, keep, st));
    TableLaunch a{};
    a.KP = c.KP;
    a.depth = depth_for(false);
    a.Sp = pl.Sp;
    a.bstart = pl.bstart;
    a.s = s;
    a.nb = pl.nb;
    a.draw = sm64_at(c.seed, kTagTable + (uint64_t)c.epoch);
    a.P = c.P;
    a.Q = c.Q;
    a.lr = lr;
    a.lp = lp;
    a.lq = lq;
    a.f = (int)g_opt.batch_f;
    a.W = g_opt.table_workers > 0 ? g_opt.table_workers : std::max(1, s / 2);
    a.tab = pl.tab;
    a.spin_limit = (uint32_t)g_opt.spin_limit;
    a.err = c.err;
    if (dbg & 1) {
        CHK(grow(&c.visits, &c.visits_cap, nnz, "visit counters"));
        c.visits_n = nnz;
        HIPCHK(hipMemsetAsync(c.visits, 0, sizeof(uint32_t) * (size_t)(nnz > 0 ? nnz : 1), st));
        a.visits = c.visits;
        a.orig = pl.orig;
    }
    if (dbg & 2) {
        const int64_t words = 3 * (int64_t)pl.nb;
        CHK(grow(&c.trace, &c.trace_cap, words, "trace"));
        c.trace_n = words;
        HIPCHK(hipMemsetAsync(c.trace, 0xff, sizeof(int32_t) * (size_t)(words > 0 ? words : 1), st));
        a.trace = c.trace;
    }
    HIPCHK(table_reset(pl.tab, pl.blist, pl.nb, s, st));
    if (c.dtype == MFSGD_FP16)
        HIPCHK(table_epoch_f16(a, st));
    else
        HIPCHK(table_epoch_f32(a, st));
    c.epoch += 1;
    return MFSGD_OK;
}

int plan_impl(const mfsgd_sample* samples, int64_t nnz, int32_t s, hipStream_t st)
{
    if (!g.inited)
        return fail(MFSGD_ESTATE, "mfsgd_init has not been called");
    if (!valid_samples(samples, nnz))
        return fail(MFSGD_EINVAL, "bad sample array");
    if (s < 1 || s > kMaxGrid)
        return fail(MFSGD_EINVAL, "grid side s must be in [1, 64]");
    return build_plan(g.wf, samples, nnz, s, balanced_grid(s), (g_opt.debug & 1) != 0, st);
}

int check_impl(const mfsgd_sample* samples, int64_t nnz, hipStream_t st)
{
    if (!g.inited)
        return fail(MFSGD_ESTATE, "mfsgd_init has not been called");
    if (!valid_samples(samples, nnz))
        return fail(MFSGD_EINVAL, "bad sample array");
    if (nnz == 0)
        return MFSGD_OK;
    HIPCHK(hipMemsetAsync(g.bad, 0, sizeof(int), st));
    HIPCHK(check_indices((const Sample*)samples, nnz, g.m, g.n, g.bad, st));
    HIPCHK(hipMemcpyAsync(g.hflag, g.bad, sizeof(int), hipMemcpyDeviceToHost, st));
    HIPCHK(hipStreamSynchronize(st));
    const int bad = *g.hflag;
    *g.hflag = 0;
    return bad ? bad_index_error() : MFSGD_OK;
}

// ---------------------------------------------------------------------------
// epochs
// ---------------------------------------------------------------------------
// Team layout of a block-scheduled launch: which workgroup serves which
// team.  Teams go to XCDs largest row block first, each onto the XCD with the
// fewest samples so far; then each XCD's workgroup slots are shared among its
// teams: one each, the rest in proportion to the samples of the team's row
// block (largest remainders first), or `uniform` per team if uniform > 0.
// Slot j of XCD x is the j-th workgroup that starts on XCD x (the kernel
// reads its XCD from the hardware and counts arrivals).
struct TeamLayout {
    std::vector<int32_t> tmap, tsize;
    std::vector<int32_t> xteams; // per XCD: team count, then the teams placed there
    int64_t grid = 0;
    int64_t xslots = 0; // pooled: workgroup slots per XCD (0: one-wavefront teams, mapped by workgroup)
};

int build_team_layout(const std::vector<int64_t>& load, int nx, int64_t slots, int64_t uniform, TeamLayout& L)
{
    const int s = (int)load.size();
    std::vector<int> order(s), xcd(s);
    for (int t = 0; t < s; ++t)
        order[t] = t;
    std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return load[x] > load[y]; });
    std::vector<int64_t> xl(nx, 0), xc(nx, 0);
    for (int t : order) {
        int best = 0;
        for (int x = 1; x < nx; ++x)
            if (xl[x] < xl[best] || (xl[x] == xl[best] && xc[x] < xc[best]))
                best = x;
        xcd[t] = best;
        xl[best] += load[t];
        xc[best] += 1;
    }
    for (int x = 0; x < nx; ++x)
        if (xc[x] > slots)
            return fail(MFSGD_EINVAL, "grid side exceeds the co-resident workgroup count");
    L.tsize.assign(s, 1);
    if (uniform > 0) {
        int64_t G = uniform;
        for (int x = 0; x < nx; ++x)
            if (xc[x] > 0)
                G = std::min<int64_t>(G, slots / xc[x]);
        for (int t = 0; t < s; ++t)
            L.tsize[t] = (int32_t)G;
    } else {
        for (int x = 0; x < nx; ++x) {
            if (xc[x] == 0)
                continue;
            const int64_t spare = slots - xc[x];
            std::vector<std::pair<double, int>> rem;
            int64_t used = 0;
            for (int t = 0; t < s; ++t) {
                if (xcd[t] != x)
                    continue;
                const double share = xl[x] > 0 ? (double)spare * (double)load[t] / (double)xl[x]
                                               : (double)spare / (double)xc[x];
                const int64_t gi = std::min<int64_t>((int64_t)share, spare - used);
                L.tsize[t] = (int32_t)(1 + gi);
                used += gi;
                rem.push_back({share - (double)gi, t});
            }
            std::stable_sort(rem.begin(), rem.end(),
                             [](const std::pair<double, int>& p, const std::pair<double, int>& q) {
                                 return p.first > q.first;
                             });
            for (size_t i = 0; used < spare && i < rem.size(); ++i, ++used)
                L.tsize[rem[i].second] += 1;
        }
    }
    L.xteams.assign((size_t)nx * (kMaxGrid + 1), 0);
    for (int t = 0; t < s; ++t) {
        int32_t* xt = &L.xteams[(size_t)xcd[t] * (kMaxGrid + 1)];
        xt[1 + xt[0]++] = t;
    }
    // tmap[x * rows + j]: the team of the j-th workgroup that starts on XCD x
    // (the kernel reads its XCD from the hardware and counts arrivals); the
    // grid holds rows workgroups per XCD, which the dispatcher deals out
    // round-robin, and any surplus on one XCD leaves at once
    std::vector<int64_t> fill(nx, 0);
    for (int t = 0; t < s; ++t)
        fill[xcd[t]] += L.tsize[t];
    const int64_t rows = *std::max_element(fill.begin(), fill.end());
    L.grid = rows * nx;
    L.xslots = rows;
    L.tmap.assign((size_t)L.grid, -1);
    std::fill(fill.begin(), fill.end(), 0);
    for (int t = 0; t < s; ++t)
        for (int m = 0; m < L.tsize[t]; ++m) {
            const int x = xcd[t];
            L.tmap[(size_t)(x * rows + fill[x])] = (t << 16) | m;
            fill[x] += 1;
        }
    return MFSGD_OK;
}

// Whether a block-scheduled epoch on plan pl redirects the stores of rows
// that the same wavefront updates again within its in-flight window.
// Automatic: when one user or one item holds most of some row or column
// block's samples.  Many wavefronts then work on the same row at once (a
// hot row block's batches are claimed concurrently; every team passes
// through a hot column), and its L2 lines become the bottleneck; otherwise
// the variant's extra register pressure costs more than it saves.
bool skip_stores(const Plan& pl)
{
    if (g_opt.skip_stores != 2)
        return g_opt.skip_stores != 0;
    return pl.hot_col > 0.5 || pl.hot_row > 0.5;
}

// Team shape of a block-scheduled launch on plan pl with `want` wavefronts per
// team (1: one-wavefront teams placed anywhere, each serving only its own
// team; 0: every workgroup slot the occupancy allows, home teams shared in
// proportion to the row blocks' samples, every wavefront also serving the
// other teams of its XCD).
int team_layout(const Plan& pl, int64_t want, bool half, EpochLaunch& a)
{
    Context& c = g;
    const int s = pl.s;
    const int waves = want == 1 ? 1 : 4;
    const int nx = std::max(1, c.nx);
    if (c.lay_plan != &pl || c.lay_version != pl.version || c.lay_want != want || c.lay_waves != waves ||
        c.lay_depth != a.depth || c.lay_half != (int)half) {
        TeamLayout L;
        if (want == 1) {
            L.grid = s;
            L.tsize.assign(s, 1);
            L.tmap.resize(s);
            for (int t = 0; t < s; ++t)
                L.tmap[t] = t << 16;
            L.xteams.assign((size_t)nx * (kMaxGrid + 1), 0);
        } else {
            const int per_cu = occupancy_blocked(c.KP, c.dtype, a.depth, 64 * waves, half);
            if (per_cu <= 0)
                return fail(MFSGD_EHIP, "occupancy query failed for the block-scheduled kernel");
            // Work is claimed, not assigned, so no workgroup has to be
            // resident for the others to progress (one per XCD is enough, and
            // the first nx workgroups of the grid are on distinct XCDs): the
            // grid takes every slot the occupancy query reports.
            const int64_t cap = (int64_t)per_cu * c.cus;
            std::vector<int64_t> load(s);
            for (int t = 0; t < s; ++t)
                load[t] = pl.hstart[(size_t)(t + 1) * s] - pl.hstart[(size_t)t * s];
            CHK(build_team_layout(load, nx, cap / nx, want > 0 ? (want + 3) / 4 : 0, L));
        }
        CHK(grow(&c.tmap, &c.tmap_cap, L.grid, "team map"));
        CHK(grow(&c.sink, &c.sink_cap, L.grid * waves * 4 * c.KP * (int64_t)elem_size(c.dtype), "store sink"));
        if (!c.tsize)
            CHK(dalloc((void**)&c.tsize, sizeof(int32_t) * kMaxGrid, "team sizes"));
        if (!c.xteams)
            CHK(dalloc((void**)&c.xteams, sizeof(int32_t) * kMaxGrid * (kMaxGrid + 1), "XCD team lists"));
        HIPCHK(hipMemcpy(c.tmap, L.tmap.data(), sizeof(int32_t) * L.tmap.size(), hipMemcpyHostToDevice));
        HIPCHK(hipMemcpy(c.xteams, L.xteams.data(), sizeof(int32_t) * L.xteams.size(), hipMemcpyHostToDevice));
        HIPCHK(hipMemcpy(c.tsize, L.tsize.data(), sizeof(int32_t) * L.tsize.size(), hipMemcpyHostToDevice));
        c.lay_plan = &pl;
        c.lay_version = pl.version;
        c.lay_want = want;
        c.lay_waves = waves;
        c.lay_depth = a.depth;
        c.lay_half = (int)half;
        c.lay_grid = (int)L.grid;
        c.lay_xslots = (int)L.xslots;
    }
    a.grid = c.lay_grid;
    a.xslots = c.lay_xslots;
    a.tmap = c.tmap;
    a.xteams = c.xteams;
    a.nx = nx;
    a.pool = want == 1 ? 0 : 1;
    a.wg_waves = waves;
    a.sink = skip_stores(pl) ? c.sink : nullptr;
    // the last 2 units per wavefront of the XCD go one unit per claim
    a.tail = a.pool && g_opt.tail_claims ? (uint32_t)std::min<int64_t>(2 * (int64_t)c.lay_xslots * waves, 1 << 30) : 0u;
    a.half = 0;
    return MFSGD_OK;
}

int epoch_impl(const mfsgd_sample* samples, int64_t nnz, float lr, float lp, float lq, int32_t scheme,
               hipStream_t st)
{
    Context& c = g;
    if (!c.inited)
        return fail(MFSGD_ESTATE, "mfsgd_init has not been called");
    if (!valid_samples(samples, nnz))
        return fail(MFSGD_EINVAL, "bad sample array");
    if (!std::isfinite(lr) || !std::isfinite(lp) || !std::isfinite(lq))
        return fail(MFSGD_EINVAL, "lr and lambdas must be finite");
    if (scheme != MFSGD_BATCH_HOGWILD && scheme != MFSGD_WAVEFRONT && scheme != MFSGD_WAVEFRONT_DET &&
        scheme != MFSGD_GLOBAL_TABLE)
        return fail(MFSGD_EINVAL, "unknown scheme");
    if (scheme == MFSGD_GLOBAL_TABLE)
        return table_epoch(samples, nnz, lr, lp, lq, st);
    const int64_t dbg = g_opt.debug;
    const bool hog = scheme == MFSGD_BATCH_HOGWILD;
    const bool automatic = hog && g_opt.partition == 2;
    int form = hog ? (int)g_opt.partition : -1;
    bool atomic = hog && g_opt.atomic != 0;
    if (automatic) {
        // the serial-tracking form for these samples
        CHK(row_stats(samples, nnz, st));
        const unsigned long long top = std::max(c.stats.du, c.stats.dv);
        const bool skewed = nnz > 0 && (double)top * kOneXcdShareInv > (double)nnz;
        // atomic adds need one worker per wavefront and, in binary16, value pairs
        const bool no_atomic = c.KP == 32 || (c.dtype == MFSGD_FP16 && c.KP < 128);
        form = skewed || no_atomic ? 4 : 0;
        atomic = form == 0;
    }
    const bool blocked = !hog || form != 0;
    Plan* pl = nullptr;
    if (!hog) {
        if (!c.wf.matches(samples, nnz))
            return fail(MFSGD_ESTATE, "wavefront-update needs mfsgd_plan on these samples first");
        pl = &c.wf;
    } else if (blocked) {
        const int s_h = hogwild_grid_side(form);
        const bool keep = (dbg & 1) != 0;
        if (!c.hw.matches(samples, nnz) || c.hw.s != s_h || c.hw.balanced != balanced_grid(s_h) ||
            (keep && !c.hw.has_orig))
            CHK(build_plan(c.hw, samples, nnz, s_h, balanced_grid(s_h), keep, st));
        pl = &c.hw;
    }
    if (blocked && (dbg & 1) && !pl->has_orig)
        return fail(MFSGD_ESTATE, "visit counting needs a plan made with debug bit 0 set");

    EpochLaunch a{};
    a.KP = c.KP;
    // the automatic form always runs one sample in flight (atomic adds need it)
    a.depth = automatic ? 1 : depth_for(hog && (form == 4 || atomic));
    a.nnz = nnz;
    a.f = (int)g_opt.batch_f;
    a.P = c.P;
    a.Q = c.Q;
    a.lr = lr;
    a.lp = lp;
    a.lq = lq;
    a.spin_limit = (uint32_t)g_opt.spin_limit;
    a.err = c.err;
    a.buf = rows_fit_31_bits() ? 1 : 0;
    if (dbg & 1) {
        CHK(grow(&c.visits, &c.visits_cap, nnz, "visit counters"));
        c.visits_n = nnz;
        HIPCHK(hipMemsetAsync(c.visits, 0, sizeof(uint32_t) * (size_t)(nnz > 0 ? nnz : 1), st));
        a.visits = c.visits;
    }
    if (!blocked) {
        const int64_t nbatch = (nnz + a.f - 1) / a.f;
        int64_t W = g_opt.workers;
        if (W == 0) {
            const int per_cu = occupancy_waves(c.KP, c.dtype, a.depth);
            if (per_cu <= 0)
                return fail(MFSGD_EHIP, "occupancy query failed for the epoch kernel");
            W = (int64_t)c.cus * per_cu * (half_wave_workers(c.KP, c.dtype) ? 2 : 1);
            if (automatic) {
                // atomic adds computed from stale reads add up: keep the
                // concurrent updates of the most popular row times the rate
                // at most 1/4 (the summed steps of one row stay small)
                const double top = (double)std::max(c.stats.du, c.stats.dv) / (double)std::max<int64_t>(nnz, 1);
                const double cap = top > 0 && lr > 0 ? 0.25 / ((double)lr * top) : 1e18;
                W = std::min(W, std::min(hogwild_condition_workers(), std::max<int64_t>(1, (int64_t)std::min(cap, 1e18))));
            }
        }
        W = std::min(W, nbatch);
        a.scheme = kSchemeHogwild;
        a.half = half_wave_workers(c.KP, c.dtype) ? 1 : 0;
        a.S = (const Sample*)samples;
        a.W = W;
        a.sync_every = (int)g_opt.sync_every;
        a.sync_l1 = (int)g_opt.sync_l1;
        a.nx = c.nx;
        if (atomic) {
            if (a.depth != 1 || a.half || (c.dtype == MFSGD_FP16 && c.KP < 128))
                return fail(MFSGD_EINVAL, "atomic updates need depth 1, one worker per wavefront and, for binary16, "
                                          "k > 64");
            a.atomic = 1;
            a.coh = g_opt.coherent == kCohBoth ? kCohBoth : kCohOff;
            const int l2 = (int)g_opt.hot_log2;
            if (l2 > 0 && nnz > 0) {
                if (!c.hot.matches(samples, nnz, l2))
                    CHK(build_hot(samples, nnz, l2, st));
                a.hot_p = c.hot.bits;
                a.hot_q = c.hot.bits + (c.m + 31) / 32;
            }
        } else if (g_opt.coherent != kCohOff && !a.half) {
            a.coh = (int)g_opt.coherent;
            a.coh_p = (g_opt.coherent_mat & 1) ? 1 : 0;
            a.coh_q = (g_opt.coherent_mat & 2) ? 1 : 0;
            const int l2 = (int)g_opt.hot_log2;
            if (l2 > 0 && nnz > 0) {
                if (!c.hot.matches(samples, nnz, l2))
                    CHK(build_hot(samples, nnz, l2, st));
                a.hot_p = c.hot.bits;
                a.hot_q = c.hot.bits + (c.m + 31) / 32;
            }
        }
        if (dbg & 2) {
            CHK(grow(&c.trace, &c.trace_cap, nbatch, "trace"));
            c.trace_n = nbatch;
            HIPCHK(hipMemsetAsync(c.trace, 0xff, sizeof(int32_t) * (size_t)(nbatch > 0 ? nbatch : 1), st));
            a.trace_batch = c.trace;
        }
        if (nnz > 0) {
            if (c.dtype == MFSGD_FP16)
                HIPCHK(epoch_f16(a, st));
            else
                HIPCHK(epoch_f32(a, st));
        }
    } else {
        const int s = pl->s;
        int64_t want;
        if (scheme == MFSGD_WAVEFRONT_DET)
            want = 1;
        else if (hog && g_opt.workers > 0)
            want = std::max<int64_t>(1, g_opt.workers / s);
        else if (automatic) {
            // one XCD: the paper's empirical Hogwild! condition caps the
            // workers; the team never exceeds the XCD's resident slots.  At
            // k <= 32 a wavefront runs two batches at once (below), i.e. two
            // workers, so it takes half as many wavefronts.
            want = hogwild_condition_workers();
            if ((c.KP == 32 && half_wave_workers(c.KP, c.dtype) && g_opt.skip_stores != 1) ||
                (g_opt.half_waves == 2 && c.KP > 32 && half_wave_workers(c.KP, c.dtype)))
                want = std::max<int64_t>(2, (want + 1) / 2);
        }
        else if (hog)
            want = 0;
        else
            want = g_opt.team_waves;
        a.scheme = kSchemeWavefront;
        a.S = pl->Sp;
        a.bstart = pl->bstart;
        a.s = s;
        // Pooled wavefronts that claim two batches at a time and run one per
        // half: block-scheduled batch-Hogwild! at k <= 32, in place of
        // skipped stores (measured faster on the Netflix shape at k = 32); at
        // wider rows, with skipped stores where the plan calls for them, for
        // both schedules with option half_waves = 2 and, by default, for
        // wavefront-update on a plan whose column blocks hold at most twice
        // their mean share (on the Hugewiki shape about 8 % shorter epochs;
        // where one column block bounds the epoch, the coarser claims
        // lengthen its chain, on the Netflix shape about 10 % longer ones).
        // One-wavefront teams keep one batch per wavefront: their blocks run
        // in order.
        const bool narrow_pairs = hog && c.KP == 32 && half_wave_workers(c.KP, c.dtype) && g_opt.skip_stores != 1;
        const bool wide_fit = c.KP > 32 && (int64_t)c.KP * (int64_t)elem_size(c.dtype) <= 16 * 32;
        const bool wide_pairs = wide_fit && (g_opt.half_waves == 2 || (g_opt.half_waves == 1 && !hog &&
                                                                       pl->col_peak <= kPairsColumnPeak));
        const bool pairs = want != 1 && (narrow_pairs || wide_pairs);
        CHK(team_layout(*pl, want, pairs, a));
        if (pairs) {
            a.half = 1;
            if (narrow_pairs)
                a.sink = nullptr;
        }
        if (atomic) {
            if (a.depth != 1 || a.half || (c.dtype == MFSGD_FP16 && c.KP < 128))
                return fail(MFSGD_EINVAL, "atomic updates need depth 1, one batch per wavefront and, for binary16, "
                                          "k > 64");
            a.atomic = 1;
            a.sink = nullptr;
            const int l2 = (int)g_opt.hot_log2;
            if (l2 > 0 && nnz > 0) {
                // atomic adds for the hot rows only
                if (!c.hot.matches(samples, nnz, l2))
                    CHK(build_hot(samples, nnz, l2, st));
                a.hot_p = c.hot.bits;
                a.hot_q = c.hot.bits + (c.m + 31) / 32;
            }
        }
        a.sigma_c = sm64_at(c.seed, kTagColPerm + 2ull * (uint64_t)c.epoch);
        a.sigma_o = sm64_at(c.seed, kTagWaveOffset + 2ull * (uint64_t)c.epoch);
        a.prio = nullptr;
        if (a.pool && g_opt.priority) {
            HIPCHK(block_priority(a.bstart, s, a.sigma_c, a.sigma_o, c.prio, st));
            a.prio = c.prio;
            c.prio_s = s;
        }
        a.tickets = c.tickets;
        a.sched = c.sched;
        a.free_run = hog && form == 3 ? 1 : 0;
        a.orig = (dbg & 1) ? pl->orig : nullptr;
        if (dbg & 2) {
            // columns, then two event stamps and two clock stamps per (team, wave)
            const int64_t words = 5 * (int64_t)s * s;
            CHK(grow(&c.trace, &c.trace_cap, words, "trace"));
            c.trace_n = words;
            HIPCHK(hipMemsetAsync(c.trace, 0xff, sizeof(int32_t) * (size_t)words, st));
            a.trace_wave = c.trace;
        }
        if (scheme == MFSGD_WAVEFRONT_DET && g_opt.wave_launch) {
            // the cross-check form: one launch per wave, ordered by the stream
            a.scheme = kSchemeWaveLaunch;
            for (int w = 0; w < s; ++w) {
                a.wave = w;
                if (c.dtype == MFSGD_FP16)
                    HIPCHK(epoch_f16(a, st));
                else
                    HIPCHK(epoch_f32(a, st));
            }
        } else {
            HIPCHK(reset_tickets(c.tickets, c.sched, st));
            if (c.dtype == MFSGD_FP16)
                HIPCHK(epoch_f16(a, st));
            else
                HIPCHK(epoch_f32(a, st));
        }
        c.last_pairs = a.half ? 1 : 0;
    }
    if (hog) {
        c.last_form = form;
        c.last_atomic = atomic ? 1 : 0;
    }
    c.epoch += 1;
    return MFSGD_OK;
}

// ---------------------------------------------------------------------------
// staged epochs (samples in host memory)
// ---------------------------------------------------------------------------
// The sample array is cut into chunks of C consecutive samples (C = option
// "stage_samples" rounded down to a multiple of f).  Chunk i is copied into
// device buffer i mod 3 on the library's copy stream while the caller's
// stream runs the batch-Hogwild! kernel (one address space) over chunk i-1;
// events order each copy after the kernel that last read its buffer and
// each kernel after its copy.  A pinned caller array is copied directly; a
// pageable one passes through pinned staging buffers, filled by this thread
// once the copy that last read them has finished.
int staged_buffers(int64_t C, bool pageable)
{
    Context& c = g;
    if (!c.copy_stream) {
        HIPCHK(hipStreamCreateWithFlags(&c.copy_stream, hipStreamNonBlocking));
        HIPCHK(hipEventCreateWithFlags(&c.ev_start, hipEventDisableTiming));
        for (int i = 0; i < Context::kStages; ++i) {
            HIPCHK(hipEventCreateWithFlags(&c.ev_copied[i], hipEventDisableTiming));
            HIPCHK(hipEventCreateWithFlags(&c.ev_used[i], hipEventDisableTiming));
        }
    }
    if (c.stage_dev_cap < C) {
        HIPCHK(hipDeviceSynchronize()); // no kernel may still read the old buffers
        for (int i = 0; i < Context::kStages; ++i) {
            dfree(c.stage_dev[i]);
            c.stage_dev[i] = nullptr;
        }
        c.stage_dev_cap = 0;
        for (int i = 0; i < Context::kStages; ++i)
            CHK(dalloc((void**)&c.stage_dev[i], sizeof(Sample) * (size_t)C, "staging buffers"));
        c.stage_dev_cap = C;
    }
    if (pageable && c.stage_host_cap < C) {
        for (int i = 0; i < Context::kStages; ++i) {
            if (c.copied_pending[i])
                HIPCHK(hipEventSynchronize(c.ev_copied[i]));
            c.copied_pending[i] = false;
            if (c.stage_host[i])
                (void)hipHostFree(c.stage_host[i]);
            c.stage_host[i] = nullptr;
        }
        c.stage_host_cap = 0;
        for (int i = 0; i < Context::kStages; ++i)
            if (hipHostMalloc((void**)&c.stage_host[i], sizeof(Sample) * (size_t)C, hipHostMallocDefault) !=
                hipSuccess) {
                (void)hipGetLastError();
                return fail(MFSGD_ENOMEM, "pinned staging allocation failed");
            }
        c.stage_host_cap = C;
    }
    return MFSGD_OK;
}

int epoch_staged_impl(const mfsgd_sample* samples, int64_t nnz, float lr, float lp, float lq, hipStream_t st)
{
    Context& c = g;
    if (!c.inited)
        return fail(MFSGD_ESTATE, "mfsgd_init has not been called");
    if (!valid_samples(samples, nnz))
        return fail(MFSGD_EINVAL, "bad sample array");
    if (!std::isfinite(lr) || !std::isfinite(lp) || !std::isfinite(lq))
        return fail(MFSGD_EINVAL, "lr and lambdas must be finite");
    bool pinned = false;
    if (nnz > 0) {
        hipPointerAttribute_t attr{};
        if (hipPointerGetAttributes(&attr, samples) == hipSuccess) {
            if (attr.type == hipMemoryTypeDevice || attr.type == hipMemoryTypeArray)
                return fail(MFSGD_EINVAL, "mfsgd_epoch_staged takes host memory; use mfsgd_epoch for device samples");
            pinned = attr.type == hipMemoryTypeHost;
        } else {
            (void)hipGetLastError(); // plain pageable memory is unknown to the runtime
        }
    }
    const int64_t f = g_opt.batch_f;
    const int64_t C = std::max<int64_t>(f, g_opt.stage_samples / f * f);
    const int64_t dbg = g_opt.debug;
    EpochLaunch a{};
    a.scheme = kSchemeHogwild;
    a.KP = c.KP;
    a.depth = depth_for(false);
    a.f = (int)f;
    a.P = c.P;
    a.Q = c.Q;
    a.lr = lr;
    a.lp = lp;
    a.lq = lq;
    a.nx = c.nx;
    a.buf = rows_fit_31_bits() ? 1 : 0;
    int64_t W = g_opt.workers;
    if (W == 0) {
        const int per_cu = occupancy_waves(c.KP, c.dtype, a.depth);
        if (per_cu <= 0)
            return fail(MFSGD_EHIP, "occupancy query failed for the epoch kernel");
        W = (int64_t)c.cus * per_cu * (half_wave_workers(c.KP, c.dtype) ? 2 : 1);
    }
    a.half = half_wave_workers(c.KP, c.dtype) ? 1 : 0;
    if (dbg & 1) {
        CHK(grow(&c.visits, &c.visits_cap, nnz, "visit counters"));
        c.visits_n = nnz;
        HIPCHK(hipMemsetAsync(c.visits, 0, sizeof(uint32_t) * (size_t)(nnz > 0 ? nnz : 1), st));
    }
    if (nnz > 0) {
        CHK(staged_buffers(std::min(C, nnz), !pinned));
        // copies start after everything already queued on the caller's stream
        // (a previous epoch's kernels may still read the device buffers)
        HIPCHK(hipEventRecord(c.ev_start, st));
        HIPCHK(hipStreamWaitEvent(c.copy_stream, c.ev_start, 0));
        const char* src = (const char*)samples;
        for (int64_t i = 0, off = 0; off < nnz; ++i, off += C) {
            const int64_t cnt = std::min(C, nnz - off);
            const int b = (int)(i % Context::kStages);
            if (i >= Context::kStages)
                HIPCHK(hipStreamWaitEvent(c.copy_stream, c.ev_used[b], 0));
            const void* from = src + (size_t)off * sizeof(Sample);
            if (!pinned) {
                if (c.copied_pending[b])
                    HIPCHK(hipEventSynchronize(c.ev_copied[b]));
                std::memcpy(c.stage_host[b], from, sizeof(Sample) * (size_t)cnt);
                from = c.stage_host[b];
            }
            HIPCHK(hipMemcpyAsync(c.stage_dev[b], from, sizeof(Sample) * (size_t)cnt, hipMemcpyHostToDevice,
                                  c.copy_stream));
            HIPCHK(hipEventRecord(c.ev_copied[b], c.copy_stream));
            c.copied_pending[b] = !pinned;
            HIPCHK(hipStreamWaitEvent(st, c.ev_copied[b], 0));
            a.S = c.stage_dev[b];
            a.nnz = cnt;
            a.W = std::min(W, (cnt + f - 1) / f);
            a.visits = (dbg & 1) ? c.visits + off : nullptr;
            if (c.dtype == MFSGD_FP16)
                HIPCHK(epoch_f16(a, st));
            else
                HIPCHK(epoch_f32(a, st));
            HIPCHK(hipEventRecord(c.ev_used[b], st));
        }
    }
    c.epoch += 1;
    return MFSGD_OK;
}

int rmse_impl(const mfsgd_sample* test, int64_t ntest, double* out, hipStream_t st)
{
    Context& c = g;
    if (!c.inited)
        return fail(MFSGD_ESTATE, "mfsgd_init has not been called");
    if (!valid_samples(test, ntest) || !out)
        return fail(MFSGD_EINVAL, "bad test array or NULL output");
    if (ntest > 0) {
        if (c.dtype == MFSGD_FP16)
            HIPCHK(rmse_partial_f16(c.KP, (const Sample*)test, ntest, c.P, c.Q, c.partial, st));
        else
            HIPCHK(rmse_partial_f32(c.KP, (const Sample*)test, ntest, c.P, c.Q, c.partial, st));
        HIPCHK(rmse_final(c.partial, ntest, c.dres, st));
        HIPCHK(hipMemcpyAsync(c.hres, c.dres, sizeof(double), hipMemcpyDeviceToHost, st));
    } else {
        *c.hres = 0.0;
    }
    int rc = sync_and_check(st);
    *out = *c.hres;
    if (rc)
        return rc;
    if (!std::isfinite(*out))
        return fail(MFSGD_ENUMERIC, "RMSE is not finite (diverged training?)");
    return MFSGD_OK;
}

// RMSE into a caller-owned device double, asynchronously, with the partial
// sums in the device's rmse_scratch array: no allocation, no host copy, no
// synchronisation (so it can be captured in a HIP graph).
int rmse_noalloc_impl(const mfsgd_sample* test, int64_t ntest, double* out, hipStream_t st)
{
    Context& c = g;
    if (!c.inited)
        return fail(MFSGD_ESTATE, "mfsgd_init has not been called");
    if (!valid_samples(test, ntest) || !out)
        return fail(MFSGD_EINVAL, "bad test array or NULL output");
    int dev = -1;
    HIPCHK(hipGetDevice(&dev));
    if (dev != c.device)
        return fail(MFSGD_ESTATE, "the current device is not the one mfsgd_init ran on");
    if (dev < 0 || dev >= kMaxDevices || !g_rmse_scratch[dev])
        return fail(MFSGD_ESTATE, "no RMSE scratch address for this device");
    double* scr = g_rmse_scratch[dev];
    if (ntest > 0) {
        if (c.dtype == MFSGD_FP16)
            HIPCHK(rmse_partial_f16(c.KP, (const Sample*)test, ntest, c.P, c.Q, scr, st));
        else
            HIPCHK(rmse_partial_f32(c.KP, (const Sample*)test, ntest, c.P, c.Q, scr, st));
    }
    HIPCHK(rmse_final(scr, ntest, out, st));
    return MFSGD_OK;
}

int factors_impl(void* P, void* Q, const void* Pin, const void* Qin, hipStream_t st)
{
    Context& c = g;
    if (!c.inited)
        return fail(MFSGD_ESTATE, "mfsgd_init has not been called");
    const size_t es = elem_size(c.dtype);
    const size_t row = (size_t)c.k * es, pitch = (size_t)c.KP * es;
    if (P)
        HIPCHK(hipMemcpy2DAsync(P, row, c.P, pitch, row, (size_t)c.m, hipMemcpyDefault, st));
    if (Q)
        HIPCHK(hipMemcpy2DAsync(Q, row, c.Q, pitch, row, (size_t)c.n, hipMemcpyDefault, st));
    if (Pin)
        HIPCHK(hipMemcpy2DAsync(c.P, pitch, Pin, row, row, (size_t)c.m, hipMemcpyDefault, st));
    if (Qin)
        HIPCHK(hipMemcpy2DAsync(c.Q, pitch, Qin, row, row, (size_t)c.n, hipMemcpyDefault, st));
    return sync_and_check(st);
}

int debug_read_impl(int32_t what, void* dst, int64_t count, hipStream_t st)
{
    Context& c = g;
    if (!c.inited)
        return fail(MFSGD_ESTATE, "mfsgd_init has not been called");
    if (!dst || count < 0)
        return fail(MFSGD_EINVAL, "bad destination");
    if (what == MFSGD_DBG_VISITS) {
        if (!c.visits || count > c.visits_n)
            return fail(MFSGD_ESTATE, "no visit counts recorded for that many samples (set debug bit 0)");
        if (count)
            HIPCHK(hipMemcpyAsync(dst, c.visits, sizeof(uint32_t) * (size_t)count, hipMemcpyDefault, st));
    } else if (what == MFSGD_DBG_TRACE) {
        if (!c.trace || count > c.trace_n)
            return fail(MFSGD_ESTATE, "no schedule trace recorded for that many entries (set debug bit 1)");
        if (count)
            HIPCHK(hipMemcpyAsync(dst, c.trace, sizeof(int32_t) * (size_t)count, hipMemcpyDefault, st));
    } else if (what == MFSGD_DBG_PLAN_STARTS) {
        if (!c.wf.valid() || count != (int64_t)c.wf.s * c.wf.s + 1)
            return fail(MFSGD_ESTATE, "no wavefront plan, or count is not s*s+1");
        HIPCHK(hipMemcpyAsync(dst, c.wf.bstart, sizeof(int64_t) * (size_t)count, hipMemcpyDefault, st));
    } else if (what == MFSGD_DBG_PLAN_ORDER) {
        if (!c.wf.valid() || !c.wf.has_orig || count > c.wf.nnz)
            return fail(MFSGD_ESTATE, "no wavefront plan with positions (plan with debug bit 0 set)");
        if (count)
            HIPCHK(hipMemcpyAsync(dst, c.wf.orig, sizeof(int64_t) * (size_t)count, hipMemcpyDefault, st));
    } else if (what == MFSGD_DBG_TABLE_STARTS) {
        if (c.gt.nnz < 0 || count != (int64_t)c.gt.s * c.gt.s + 1)
            return fail(MFSGD_ESTATE, "no global-table plan, or count is not s*s+1");
        HIPCHK(hipMemcpyAsync(dst, c.gt.bstart, sizeof(int64_t) * (size_t)count, hipMemcpyDefault, st));
    } else if (what == MFSGD_DBG_TABLE_ORDER) {
        if (c.gt.nnz < 0 || !c.gt.has_orig || count > c.gt.nnz)
            return fail(MFSGD_ESTATE, "no global-table plan with positions (run it with debug bit 0 set)");
        if (count)
            HIPCHK(hipMemcpyAsync(dst, c.gt.orig, sizeof(int64_t) * (size_t)count, hipMemcpyDefault, st));
    } else if (what == MFSGD_DBG_TEAM_MAP || what == MFSGD_DBG_TEAM_SIZES) {
        if (!c.lay_plan)
            return fail(MFSGD_ESTATE, "no block-scheduled epoch has run");
        const int64_t have = what == MFSGD_DBG_TEAM_MAP ? c.lay_grid : c.lay_plan->s;
        if (count > have)
            return fail(MFSGD_ESTATE, "count exceeds the team layout");
        if (count)
            HIPCHK(hipMemcpyAsync(dst, what == MFSGD_DBG_TEAM_MAP ? c.tmap : c.tsize, sizeof(int32_t) * (size_t)count,
                                  hipMemcpyDefault, st));
    } else if (what == MFSGD_DBG_PRIORITY) {
        if (c.prio_s == 0)
            return fail(MFSGD_ESTATE, "no block-scheduled epoch with priorities has run");
        if (count != (int64_t)c.prio_s * c.prio_s)
            return fail(MFSGD_EINVAL, "count must be s*s of the last epoch with priorities");
        HIPCHK(hipMemcpyAsync(dst, c.prio, sizeof(uint32_t) * (size_t)count, hipMemcpyDefault, st));
    } else {
        return fail(MFSGD_EINVAL, "unknown debug buffer");
    }
    return sync_and_check(st);
}

} // namespace

extern "C" {

int mfsgd_set_option(const char* key, int64_t value)
{
    return guarded([&]() -> int { return set_option_impl(key, value); });
}

int mfsgd_get_option(const char* key, int64_t* value)
{
    return guarded([&]() -> int { return get_option_impl(key, value); });
}

int mfsgd_reset_options(void)
{
    return guarded([&]() -> int {
        g_opt = Options();
        return MFSGD_OK;
    });
}

int mfsgd_init(int64_t m, int64_t n, int32_t k, uint64_t seed)
{
    return guarded([&]() -> int { return init_impl(m, n, k, seed); });
}

int mfsgd_plan(const mfsgd_sample* samples, int64_t nnz, int32_t s, void* stream)
{
    return guarded([&]() -> int { return plan_impl(samples, nnz, s, (hipStream_t)stream); });
}

int mfsgd_epoch(const mfsgd_sample* samples, int64_t nnz, float lr, float lambda_p, float lambda_q, int32_t scheme,
                void* stream)
{
    return guarded(
        [&]() -> int { return epoch_impl(samples, nnz, lr, lambda_p, lambda_q, scheme, (hipStream_t)stream); });
}

int mfsgd_epoch_staged(const mfsgd_sample* samples, int64_t nnz, float lr, float lambda_p, float lambda_q,
                       void* stream)
{
    return guarded(
        [&]() -> int { return epoch_staged_impl(samples, nnz, lr, lambda_p, lambda_q, (hipStream_t)stream); });
}

int mfsgd_rmse(const mfsgd_sample* test, int64_t ntest, double* rmse_out, void* stream)
{
    return guarded([&]() -> int { return rmse_impl(test, ntest, rmse_out, (hipStream_t)stream); });
}

int mfsgd_rmse_noalloc(const mfsgd_sample* test, int64_t ntest, double* rmse_dev, void* stream)
{
    return guarded([&]() -> int { return rmse_noalloc_impl(test, ntest, rmse_dev, (hipStream_t)stream); });
}

int mfsgd_check_samples(const mfsgd_sample* samples, int64_t nnz, void* stream)
{
    return guarded([&]() -> int { return check_impl(samples, nnz, (hipStream_t)stream); });
}

int mfsgd_sync(void* stream)
{
    return guarded([&]() -> int {
        if (!g.inited)
            return fail(MFSGD_ESTATE, "mfsgd_init has not been called");
        return sync_and_check((hipStream_t)stream);
    });
}

int mfsgd_get_factors(void* P, void* Q, void* stream)
{
    return guarded([&]() -> int { return factors_impl(P, Q, nullptr, nullptr, (hipStream_t)stream); });
}

int mfsgd_set_factors(const void* P, const void* Q, void* stream)
{
    return guarded([&]() -> int { return factors_impl(nullptr, nullptr, P, Q, (hipStream_t)stream); });
}

int mfsgd_set_epoch(int64_t t)
{
    return guarded([&]() -> int {
        if (!g.inited)
            return fail(MFSGD_ESTATE, "mfsgd_init has not been called");
        if (t < 0)
            return fail(MFSGD_EINVAL, "epoch must be >= 0");
        g.epoch = t;
        return MFSGD_OK;
    });
}

int64_t mfsgd_get_epoch(void) { return g.inited ? g.epoch : -1; }

int mfsgd_debug_read(int32_t what, void* dst, int64_t count, void* stream)
{
    return guarded([&]() -> int { return debug_read_impl(what, dst, count, (hipStream_t)stream); });
}

int mfsgd_finalize(void)
{
    return guarded([&]() -> int {
        if (g.inited)
            (void)hipDeviceSynchronize();
        release_all();
        return MFSGD_OK;
    });
}

const char* mfsgd_last_error(void) { return g_err.c_str(); }

const char* mfsgd_version(void) { return "mfsgd 0.2 (gfx950)"; }

} // extern "C"
