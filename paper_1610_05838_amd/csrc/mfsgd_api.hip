// mfsgd_api.hip -- the C ABI (include/mfsgd.h): context, argument checks,
// buffer ownership, kernel selection and device-error reporting.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>

#include "mfsgd.h"
#include "mfsgd_device.hpp"
#include "mfsgd_launch.hpp"

namespace {

using namespace mfsgd;

thread_local std::string g_err;

struct Options {
    int64_t dtype = MFSGD_FP32;
    int64_t batch_f = 256;
    int64_t workers = 0;
    int64_t depth = 4;
    int64_t waves_per_block = 8;
    int64_t spin_limit = int64_t(1) << 24;
    int64_t debug = 0;
};

struct Context {
    bool inited = false;
    int device = 0;
    int cus = 0;
    int64_t m = 0, n = 0;
    int k = 0, KP = 0, dtype = 0;
    uint64_t seed = 0;
    int64_t epoch = 0;
    void* P = nullptr;
    void* Q = nullptr;
    // small device/pinned buffers
    uint32_t* tickets = nullptr;
    int* err = nullptr;
    int* bad = nullptr;
    double* partial = nullptr;
    double* dres = nullptr;
    double* hres = nullptr; // pinned
    int* hflag = nullptr;   // pinned
    // plan
    const mfsgd_sample* plan_src = nullptr;
    int64_t plan_nnz = -1;
    int plan_s = 0;
    bool plan_orig = false;
    Sample* Sp = nullptr;
    int64_t Sp_cap = 0;
    int64_t* orig = nullptr;
    int64_t orig_cap = 0;
    int32_t* counts = nullptr;
    int64_t* totals = nullptr;
    int64_t* bstart = nullptr;
    // debug
    uint32_t* visits = nullptr;
    int64_t visits_cap = 0, visits_n = 0;
    int32_t* trace = nullptr;
    int64_t trace_cap = 0, trace_n = 0;
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

int dfree(void* p)
{
    if (p)
        (void)hipFree(p);
    return 0;
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

void release_all()
{
    Context& c = g;
    dfree(c.P);
    dfree(c.Q);
    dfree(c.tickets);
    dfree(c.err);
    dfree(c.bad);
    dfree(c.partial);
    dfree(c.dres);
    if (c.hres)
        (void)hipHostFree(c.hres);
    if (c.hflag)
        (void)hipHostFree(c.hflag);
    dfree(c.Sp);
    dfree(c.orig);
    dfree(c.counts);
    dfree(c.totals);
    dfree(c.bstart);
    dfree(c.visits);
    dfree(c.trace);
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

int occupancy_waves(int KP, int dtype, int depth)
{
    return dtype == MFSGD_FP16 ? occupancy_f16(KP, depth) : occupancy_f32(KP, depth);
}

// Read back and clear the device error flag; the stream has been synchronised.
int take_device_error()
{
    if (*g.hflag) {
        *g.hflag = 0;
        int zero = 0;
        HIPCHK(hipMemcpy(g.err, &zero, sizeof(int), hipMemcpyHostToDevice));
        return fail(MFSGD_ETIMEOUT, "a wavefront-update ticket wait exceeded spin_limit; the epoch was abandoned");
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

int set_option_impl(const char* key, int64_t value)
{
    if (!key)
        return fail(MFSGD_EINVAL, "option key is NULL");
    std::string k(key);
    if (k == "dtype") {
        if (value != MFSGD_FP32 && value != MFSGD_FP16)
            return fail(MFSGD_EINVAL, "dtype must be 0 (fp32) or 1 (fp16)");
        g_opt.dtype = value;
    } else if (k == "batch_f") {
        if (value <= 0 || value % 64 != 0 || value > (int64_t(1) << 30))
            return fail(MFSGD_EINVAL, "batch_f must be a positive multiple of 64");
        g_opt.batch_f = value;
    } else if (k == "workers") {
        if (value < 0 || value > (int64_t(1) << 30))
            return fail(MFSGD_EINVAL, "workers must be in [0, 2^30]");
        g_opt.workers = value;
    } else if (k == "depth") {
        if (value != 1 && value != 2 && value != 4 && value != 8)
            return fail(MFSGD_EINVAL, "depth must be 1, 2, 4 or 8");
        g_opt.depth = value;
    } else if (k == "waves_per_block") {
        if (value < 1 || value > 16)
            return fail(MFSGD_EINVAL, "waves_per_block must be in [1, 16]");
        g_opt.waves_per_block = value;
    } else if (k == "spin_limit") {
        if (value < 1 || value > 0xffffffffll)
            return fail(MFSGD_EINVAL, "spin_limit must be in [1, 2^32-1]");
        g_opt.spin_limit = value;
    } else if (k == "debug") {
        if (value < 0 || value > 3)
            return fail(MFSGD_EINVAL, "debug must be in [0, 3]");
        g_opt.debug = value;
    } else {
        return fail(MFSGD_EINVAL, "unknown option '" + k + "'");
    }
    return MFSGD_OK;
}

int get_option_impl(const char* key, int64_t* value)
{
    if (!key || !value)
        return fail(MFSGD_EINVAL, "NULL argument");
    std::string k(key);
    if (k == "dtype")
        *value = g_opt.dtype;
    else if (k == "batch_f")
        *value = g_opt.batch_f;
    else if (k == "workers")
        *value = g_opt.workers;
    else if (k == "depth")
        *value = g_opt.depth;
    else if (k == "waves_per_block")
        *value = g_opt.waves_per_block;
    else if (k == "spin_limit")
        *value = g_opt.spin_limit;
    else if (k == "debug")
        *value = g_opt.debug;
    else if (k == "resident_waves") { // read-only: wavefronts of the epoch kernel the GPU holds at once
        if (!g.inited)
            return fail(MFSGD_ESTATE, "resident_waves needs mfsgd_init");
        *value = (int64_t)g.cus * occupancy_waves(g.KP, g.dtype, (int)g_opt.depth);
    } else
        return fail(MFSGD_EINVAL, "unknown option '" + k + "'");
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
    HIPCHK(hipGetDevice(&c.device));
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
        (rc = dalloc((void**)&c.err, sizeof(int), "flag")) || (rc = dalloc((void**)&c.bad, sizeof(int), "flag")) ||
        (rc = dalloc((void**)&c.partial, sizeof(double) * kRmseWaves, "rmse partials")) ||
        (rc = dalloc((void**)&c.dres, sizeof(double), "rmse result"))) {
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
    HIPCHK(hipMemset(c.tickets, 0, sizeof(uint32_t) * kMaxGrid));
    const double inv_sqrt_k = 1.0 / std::sqrt((double)k);
    const uint64_t sp = sm64_at(seed, kTagP), sq = sm64_at(seed, kTagQ);
    if (c.dtype == MFSGD_FP16) {
        HIPCHK(init_f16(c.P, m, k, c.KP, sp, inv_sqrt_k, nullptr));
        HIPCHK(init_f16(c.Q, n, k, c.KP, sq, inv_sqrt_k, nullptr));
    } else {
        HIPCHK(init_f32(c.P, m, k, c.KP, sp, inv_sqrt_k, nullptr));
        HIPCHK(init_f32(c.Q, n, k, c.KP, sq, inv_sqrt_k, nullptr));
    }
    HIPCHK(hipDeviceSynchronize());
    c.inited = true;
    return MFSGD_OK;
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
    int bad = *g.hflag;
    *g.hflag = 0;
    if (bad)
        return fail(MFSGD_EINVAL, "a sample index is out of range (need 0 <= u < m and 0 <= v < n)");
    return MFSGD_OK;
}

int plan_impl(const mfsgd_sample* samples, int64_t nnz, int32_t s, hipStream_t st)
{
    Context& c = g;
    if (!c.inited)
        return fail(MFSGD_ESTATE, "mfsgd_init has not been called");
    if (!valid_samples(samples, nnz))
        return fail(MFSGD_EINVAL, "bad sample array");
    if (s < 1 || s > kMaxGrid)
        return fail(MFSGD_EINVAL, "grid side s must be in [1, 64]");
    c.plan_src = nullptr;
    c.plan_nnz = -1;
    int rc;
    const int64_t nb = (int64_t)s * s;
    if (!c.counts) {
        if ((rc = dalloc((void**)&c.counts, sizeof(int32_t) * kMaxGrid * kMaxGrid * kPlanChunks, "plan counts")) ||
            (rc = dalloc((void**)&c.totals, sizeof(int64_t) * kMaxGrid * kMaxGrid, "plan totals")) ||
            (rc = dalloc((void**)&c.bstart, sizeof(int64_t) * (kMaxGrid * kMaxGrid + 1), "plan starts")))
            return rc;
    }
    if ((rc = grow(&c.Sp, &c.Sp_cap, nnz, "planned samples")))
        return rc;
    const bool keep_orig = (g_opt.debug & 1) != 0;
    if (keep_orig && (rc = grow(&c.orig, &c.orig_cap, nnz, "plan positions")))
        return rc;
    PlanBuffers b{c.counts, c.totals, c.bstart, c.Sp, keep_orig ? c.orig : nullptr, c.bad};
    HIPCHK(hipMemsetAsync(c.bad, 0, sizeof(int), st));
    HIPCHK(plan_build((const Sample*)samples, nnz, c.m, c.n, s, b, st));
    HIPCHK(hipMemcpyAsync(c.hflag, c.bad, sizeof(int), hipMemcpyDeviceToHost, st));
    HIPCHK(hipStreamSynchronize(st));
    const int bad = *c.hflag;
    *c.hflag = 0;
    if (bad)
        return fail(MFSGD_EINVAL, "a sample index is out of range (need 0 <= u < m and 0 <= v < n)");
    HIPCHK(plan_scatter((const Sample*)samples, nnz, c.m, c.n, s, b, st));
    HIPCHK(hipStreamSynchronize(st));
    (void)nb;
    c.plan_src = samples;
    c.plan_nnz = nnz;
    c.plan_s = s;
    c.plan_orig = keep_orig;
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
    if (scheme != MFSGD_BATCH_HOGWILD && scheme != MFSGD_WAVEFRONT && scheme != MFSGD_WAVEFRONT_DET)
        return fail(MFSGD_EINVAL, "unknown scheme");
    const bool wavefront = scheme != MFSGD_BATCH_HOGWILD;
    if (wavefront && (c.plan_src != samples || c.plan_nnz != nnz))
        return fail(MFSGD_ESTATE, "wavefront-update needs mfsgd_plan on these samples first");
    const int64_t dbg = g_opt.debug;
    if (wavefront && (dbg & 1) && !c.plan_orig)
        return fail(MFSGD_ESTATE, "visit counting in wavefront-update needs a plan made with debug bit 0 set");

    EpochLaunch a{};
    a.KP = c.KP;
    a.depth = (int)g_opt.depth;
    a.nnz = nnz;
    a.f = (int)g_opt.batch_f;
    a.P = c.P;
    a.Q = c.Q;
    a.lr = lr;
    a.lp = lp;
    a.lq = lq;
    a.spin_limit = (uint32_t)g_opt.spin_limit;
    a.err = c.err;
    int rc;
    if (dbg & 1) {
        if ((rc = grow(&c.visits, &c.visits_cap, nnz, "visit counters")))
            return rc;
        c.visits_n = nnz;
        HIPCHK(hipMemsetAsync(c.visits, 0, sizeof(uint32_t) * (size_t)(nnz > 0 ? nnz : 1), st));
        a.visits = c.visits;
    }
    if (!wavefront) {
        const int64_t nbatch = (nnz + a.f - 1) / a.f;
        int64_t W = g_opt.workers;
        if (W == 0) {
            const int per_cu = occupancy_waves(c.KP, c.dtype, a.depth);
            if (per_cu <= 0)
                return fail(MFSGD_EHIP, "occupancy query failed for the epoch kernel");
            W = (int64_t)c.cus * per_cu;
        }
        if (W > nbatch)
            W = nbatch;
        a.scheme = kSchemeHogwild;
        a.S = (const Sample*)samples;
        a.W = W;
        if (dbg & 2) {
            if ((rc = grow(&c.trace, &c.trace_cap, nbatch, "trace")))
                return rc;
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
        const int s = c.plan_s;
        a.scheme = kSchemeWavefront;
        a.S = c.Sp;
        a.bstart = c.bstart;
        a.s = s;
        a.team_waves = scheme == MFSGD_WAVEFRONT_DET ? 1 : (int)g_opt.waves_per_block;
        a.sigma_c = sm64_at(c.seed, kTagColPerm + 2ull * (uint64_t)c.epoch);
        a.sigma_o = sm64_at(c.seed, kTagWaveOffset + 2ull * (uint64_t)c.epoch);
        a.tickets = c.tickets;
        a.orig = (dbg & 1) ? c.orig : nullptr;
        if (dbg & 2) {
            if ((rc = grow(&c.trace, &c.trace_cap, (int64_t)s * s, "trace")))
                return rc;
            c.trace_n = (int64_t)s * s;
            HIPCHK(hipMemsetAsync(c.trace, 0xff, sizeof(int32_t) * (size_t)s * s, st));
            a.trace_wave = c.trace;
        }
        HIPCHK(reset_tickets(c.tickets, s, c.err, st));
        if (c.dtype == MFSGD_FP16)
            HIPCHK(epoch_f16(a, st));
        else
            HIPCHK(epoch_f32(a, st));
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
    return guarded([&]() -> int { return epoch_impl(samples, nnz, lr, lambda_p, lambda_q, scheme, (hipStream_t)stream); });
}

int mfsgd_rmse(const mfsgd_sample* test, int64_t ntest, double* rmse_out, void* stream)
{
    return guarded([&]() -> int { return rmse_impl(test, ntest, rmse_out, (hipStream_t)stream); });
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

const char* mfsgd_version(void) { return "mfsgd 0.1 (gfx950)"; }

} // extern "C"
