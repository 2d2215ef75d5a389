// mfsgd_kernels.hpp -- the gfx950 kernels and their launchers, instantiated
// once per storage type (mfsgd_kernels_f32.hip, mfsgd_kernels_f16.hip).
#pragma once

#include "mfsgd_device.hpp"
#include "mfsgd_launch.hpp"

namespace mfsgd {

constexpr int kHogwildBlock = 256; // 4 wavefronts per workgroup, each an independent worker

// batch-Hogwild! over the whole GPU in one address space (section 3.2.2):
// wavefront w of the grid is worker w.  The XCDs' L2 caches are not coherent
// with each other, so rows that several XCDs touch are updated in per-XCD
// copies until evicted; the block-scheduled kernel below is the coherent form.
template <int KP, typename T, int D, bool DBG>
__global__ __launch_bounds__(kHogwildBlock) void k_hogwild(const Sample* __restrict__ S, int64_t nnz, int64_t W,
                                                           int f, T* __restrict__ P, T* __restrict__ Q, float lr,
                                                           float lp, float lq, DebugSink dbg, int sync_every,
                                                           int sync_l1, int nx)
{
    const int64_t worker = uniform64((int64_t)blockIdx.x * (kHogwildBlock / 64) + (threadIdx.x >> 6));
    if (worker >= W)
        return;
    // workgroups are dealt to XCDs round-robin: the first wavefront of each of
    // the first nx workgroups leads its XCD's cache flushes
    const CacheSync sync{sync_every, (int)blockIdx.x < nx && (threadIdx.x >> 6) == 0, sync_l1 != 0};
    run_worker<KP, T, D, DBG>(S, nnz, W, worker, f, P, Q, lr, lp, lq, dbg, sync);
}

// Block-scheduled epoch: wavefront-update (section 3.2.3), and
// batch-Hogwild! partitioned over the GPU's coherence domains.
//
// The s x s grid of blocks is processed in s waves.  Worker (team) i owns row
// block i and in wave w takes column block sigma_i(w) = C[(i + O[w]) mod s],
// so the blocks of one wave share no row and no column.  Column tickets order
// the waves: team i starts wave w once ticket[sigma_i(w)] reads w, and the
// last member to finish releases it with w+1 (every column is used by exactly
// one team per wave, so a ticket counts the waves completed on its column).
//
// A team is a set of workgroups; inside a block its wavefronts run
// batch-Hogwild! (run_worker) over the block's samples.  Members do not wait
// for each other between waves (they share the team's row block, which no
// other team touches); the last one to finish a wave releases its column.
// tmap[b] gives the team and member index of workgroup b (-1: idle), tsize[i]
// the workgroup count of team i.  The host builds the map so that every
// member of a team sits on one XCD (workgroup b runs on XCD b mod nx, checked
// at init) and teams get workgroups in proportion to their row block's
// samples; the team's unsynchronised updates then meet in that XCD's shared
// L2.  Feature rows move between teams only at block hand-over, through an
// agent-scope release (L2 write-back) and acquire (L1/L2 invalidate),
// whichever XCDs the two teams run on.
//
// A ticket wait that exceeds spin_limit polls raises *err; every waiting
// workgroup then leaves, so the grid always drains.
template <int KP, typename T, int D, bool DBG, bool SKIP>
__global__ __launch_bounds__(1024) void k_blocked(const Sample* __restrict__ Sp, const int64_t* __restrict__ bstart,
                                                  int s, const int32_t* __restrict__ tmap,
                                                  const int32_t* __restrict__ tsize, uint64_t sigma_c, uint64_t sigma_o,
                                                  T* __restrict__ P, T* __restrict__ Q, float lr, float lp, float lq,
                                                  int f, uint32_t* tickets, uint32_t* done, uint32_t spin_limit,
                                                  int* err, DebugSink dbg, int32_t* trace, T* __restrict__ sink)
{
    __shared__ int Cperm[kMaxGrid], Ooff[kMaxGrid];
    __shared__ int abort_all;
    const int tm = tmap[blockIdx.x];
    if (tm < 0)
        return;
    const int team = tm >> 16;
    const int member = tm & 0xffff;
    const int G = tsize[team];
    const int waves = blockDim.x >> 6;
    const int wv = uniform(threadIdx.x >> 6);
    const int64_t W = (int64_t)G * waves;
    const int64_t worker = (int64_t)member * waves + wv;
    // two private rows per wavefront of the grid for skipped stores
    T* const my_sink = SKIP ? sink + ((int64_t)blockIdx.x * waves + wv) * 2 * KP : nullptr;
    if (threadIdx.x == 0) {
        shuffle_perm(sigma_c, s, Cperm);
        shuffle_perm(sigma_o, s, Ooff);
        abort_all = 0;
    }
    __syncthreads();
    DebugSink inner = dbg;
    inner.trace = nullptr;
    for (int w = 0; w < s; ++w) {
        const int col = Cperm[(team + Ooff[w]) % s];
        if (threadIdx.x == 0) {
            // Poll with an atomic read-modify-write: it is resolved at the
            // device's coherence point, whereas a plain (even agent-scope) load
            // may keep hitting a stale copy in this XCD's L2.  Acquire once the
            // ticket has come round, which invalidates this CU's L1 and this
            // XCD's L2 before the block's rows are read.
            uint32_t polls = 0;
            while (__hip_atomic_fetch_or(tickets + col, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) !=
                   (uint32_t)w) {
                if (++polls > spin_limit ||
                    __hip_atomic_fetch_or(err, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
                    __hip_atomic_fetch_or(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    abort_all = 1;
                    break;
                }
                __builtin_amdgcn_s_sleep(4);
            }
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            if (trace && member == 0)
                trace[(int64_t)team * s + w] = col;
        }
        __syncthreads();
        if (abort_all)
            return;
        const int64_t b = (int64_t)team * s + col;
        const int64_t lo = bstart[b], hi = bstart[b + 1];
        if (hi > lo) {
            DebugSink blk = inner;
            if (blk.orig)
                blk.orig += lo;
            run_worker<KP, T, D, DBG, SKIP>(Sp + lo, hi - lo, W, worker, f, P, Q, lr, lp, lq, blk,
                                            CacheSync{0, false, false}, my_sink);
        }
        __syncthreads(); // every wavefront of this workgroup is done with the block
        if (threadIdx.x == 0) {
            if (G == 1) {
                __hip_atomic_store(tickets + col, (uint32_t)(w + 1), __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
            } else {
                // one counter per (team, wave): a member may already be in the
                // next wave (its next column can come free first) while another
                // is still finishing this one
                const uint32_t before = __hip_atomic_fetch_add(done + (int64_t)team * s + w, 1u, __ATOMIC_ACQ_REL,
                                                               __HIP_MEMORY_SCOPE_AGENT);
                if (before == (uint32_t)(G - 1)) // last member of the team to finish this wave
                    __hip_atomic_store(tickets + col, (uint32_t)(w + 1), __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
    }
}

template <int KP, typename T, int D>
static int occupancy_blocked_t(int threads)
{
    int blocks = 0;
    // the co-residency cap must hold for both variants the launcher may pick
    int plain = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_blocked<KP, T, D, false, true>, threads, 0) !=
            hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&plain, k_blocked<KP, T, D, false, false>, threads, 0) !=
            hipSuccess)
        return 0;
    return blocks < plain ? blocks : plain;
}

template <int KP, typename T>
static int occupancy_blocked_kp(int depth, int threads)
{
    switch (depth) {
    case 1: return occupancy_blocked_t<KP, T, 1>(threads);
    case 2: return occupancy_blocked_t<KP, T, 2>(threads);
    case 4: return occupancy_blocked_t<KP, T, 4>(threads);
    case 8: return occupancy_blocked_t<KP, T, 8>(threads);
    default: return 0;
    }
}

// Test RMSE, pass 1 (section 3.2.4): wavefront w of kRmseWaves sums the
// squared errors of its contiguous share of the test samples in binary64.
// Samples are independent here, so 8 are fetched before any is reduced.
template <int KP, typename T>
__global__ __launch_bounds__(256) void k_rmse_partial(const Sample* __restrict__ S, int64_t ntest,
                                                      const T* __restrict__ P, const T* __restrict__ Q,
                                                      double* __restrict__ partial)
{
    constexpr int E = Geo<KP>::E;
    constexpr int A = Geo<KP>::A;
    constexpr int U = 8;
    typedef Row<T, E> R;
    const int lane = lane_id();
    const bool holds = (A == 64) || (lane < A);
    const int col = lane * E;
    const int64_t wave = uniform64((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6));
    const int64_t share = (ntest + kRmseWaves - 1) / kRmseWaves;
    const int64_t lo = wave * share;
    const int64_t hi = lo + share < ntest ? lo + share : ntest;
    double acc = 0.0;
    for (int64_t c0 = lo; c0 < hi; c0 += 64) {
        const int cnt = (int)(hi - c0 >= 64 ? 64 : hi - c0);
        int cu = 0, cv = 0;
        float cr = 0.f;
        if (lane < cnt) {
            cu = __builtin_nontemporal_load(&S[c0 + lane].u);
            cv = __builtin_nontemporal_load(&S[c0 + lane].v);
            cr = __builtin_nontemporal_load(&S[c0 + lane].r);
        }
        for (int i0 = 0; i0 < cnt; i0 += U) {
            float p[U][E], q[U][E];
#pragma unroll
            for (int j = 0; j < U; ++j) {
                const int i = i0 + j;
#pragma unroll
                for (int e = 0; e < E; ++e)
                    p[j][e] = q[j][e] = 0.f;
                if (i < cnt && holds) {
                    const int u = __builtin_amdgcn_readlane(cu, i);
                    const int v = __builtin_amdgcn_readlane(cv, i);
                    R::load(P + (int64_t)u * KP + col, p[j]);
                    R::load(Q + (int64_t)v * KP + col, q[j]);
                }
            }
#pragma unroll
            for (int j = 0; j < U; ++j) {
                const int i = i0 + j;
                float dot = 0.f;
#pragma unroll
                for (int e = 0; e < E; ++e)
                    dot += p[j][e] * q[j][e];
                dot = wave_sum(dot);
                if (i < cnt) {
                    const float r = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cr), i));
                    const double e = (double)(r - dot);
                    acc += e * e;
                }
            }
        }
    }
    if (lane == 0)
        partial[wave] = acc;
}

template <int KP, typename T, int D, bool DBG>
static hipError_t launch_epoch_d(const EpochLaunch& a, hipStream_t st)
{
    T* P = (T*)a.P;
    T* Q = (T*)a.Q;
    if (a.scheme == kSchemeHogwild) {
        const int64_t blocks = (a.W + 3) / 4;
        const DebugSink dbg{a.visits, nullptr, a.trace_batch};
        hipLaunchKernelGGL((k_hogwild<KP, T, D, DBG>), dim3((unsigned)blocks), dim3(kHogwildBlock), 0, st, a.S,
                           a.nnz, a.W, a.f, P, Q, a.lr, a.lp, a.lq, dbg, a.sync_every, a.sync_l1, a.nx);
    } else {
        const DebugSink dbg{a.visits, a.orig, nullptr};
        // skipped stores only in epochs without debug output (they never change results)
        if (!DBG && a.sink)
            hipLaunchKernelGGL((k_blocked<KP, T, D, false, true>), dim3((unsigned)a.grid), dim3(64 * a.wg_waves), 0,
                               st, a.S, a.bstart, a.s, a.tmap, a.tsize, a.sigma_c, a.sigma_o, P, Q, a.lr, a.lp, a.lq,
                               a.f, a.tickets, a.done, a.spin_limit, a.err, dbg, a.trace_wave, (T*)a.sink);
        else
            hipLaunchKernelGGL((k_blocked<KP, T, D, DBG, false>), dim3((unsigned)a.grid), dim3(64 * a.wg_waves), 0,
                               st, a.S, a.bstart, a.s, a.tmap, a.tsize, a.sigma_c, a.sigma_o, P, Q, a.lr, a.lp, a.lq,
                               a.f, a.tickets, a.done, a.spin_limit, a.err, dbg, a.trace_wave, (T*)nullptr);
    }
    return hipGetLastError();
}

template <int KP, typename T, int D>
static hipError_t launch_epoch_t(const EpochLaunch& a, hipStream_t st)
{
    if (a.visits || a.trace_batch)
        return launch_epoch_d<KP, T, D, true>(a, st);
    return launch_epoch_d<KP, T, D, false>(a, st);
}

template <int KP, typename T>
static hipError_t launch_epoch_kp(const EpochLaunch& a, hipStream_t st)
{
    switch (a.depth) {
    case 1: return launch_epoch_t<KP, T, 1>(a, st);
    case 2: return launch_epoch_t<KP, T, 2>(a, st);
    case 4: return launch_epoch_t<KP, T, 4>(a, st);
    case 8: return launch_epoch_t<KP, T, 8>(a, st);
    default: return hipErrorInvalidValue;
    }
}

template <int KP, typename T, int D>
static int occupancy_t()
{
    int blocks = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_hogwild<KP, T, D, false>, kHogwildBlock, 0) != hipSuccess)
        return 0;
    return blocks * (kHogwildBlock / 64);
}

template <int KP, typename T>
static int occupancy_kp(int depth)
{
    switch (depth) {
    case 1: return occupancy_t<KP, T, 1>();
    case 2: return occupancy_t<KP, T, 2>();
    case 4: return occupancy_t<KP, T, 4>();
    case 8: return occupancy_t<KP, T, 8>();
    default: return 0;
    }
}

template <typename T>
__global__ void k_init(T* __restrict__ A, int64_t rows, int k, int KP, uint64_t stream, double inv_sqrt_k)
{
    const int64_t total = rows * KP;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = i / KP;
        const int j = (int)(i - row * KP);
        double val = 0.0;
        if (j < k) {
            const uint64_t x = sm64_at(stream, (uint64_t)(row * k + j));
            val = (double)(x >> 40) * 0x1p-24 * inv_sqrt_k;
        }
        A[i] = from_f64<T>(val);
    }
}

template <typename T>
struct Dispatch {
    static hipError_t epoch(const EpochLaunch& a, hipStream_t st)
    {
        switch (a.KP) {
        case 32: return launch_epoch_kp<32, T>(a, st);
        case 64: return launch_epoch_kp<64, T>(a, st);
        case 128: return launch_epoch_kp<128, T>(a, st);
        case 256: return launch_epoch_kp<256, T>(a, st);
        case 512: return launch_epoch_kp<512, T>(a, st);
        default: return hipErrorInvalidValue;
        }
    }
    static int occupancy(int KP, int depth)
    {
        switch (KP) {
        case 32: return occupancy_kp<32, T>(depth);
        case 64: return occupancy_kp<64, T>(depth);
        case 128: return occupancy_kp<128, T>(depth);
        case 256: return occupancy_kp<256, T>(depth);
        case 512: return occupancy_kp<512, T>(depth);
        default: return 0;
        }
    }
    static int occupancy_blocked(int KP, int depth, int threads)
    {
        switch (KP) {
        case 32: return occupancy_blocked_kp<32, T>(depth, threads);
        case 64: return occupancy_blocked_kp<64, T>(depth, threads);
        case 128: return occupancy_blocked_kp<128, T>(depth, threads);
        case 256: return occupancy_blocked_kp<256, T>(depth, threads);
        case 512: return occupancy_blocked_kp<512, T>(depth, threads);
        default: return 0;
        }
    }
    static hipError_t rmse(int KP, const Sample* S, int64_t ntest, const void* P, const void* Q, double* partial,
                           hipStream_t st)
    {
        const dim3 grid(kRmseWaves / 4), block(256);
        switch (KP) {
        case 32: hipLaunchKernelGGL((k_rmse_partial<32, T>), grid, block, 0, st, S, ntest, (const T*)P, (const T*)Q, partial); break;
        case 64: hipLaunchKernelGGL((k_rmse_partial<64, T>), grid, block, 0, st, S, ntest, (const T*)P, (const T*)Q, partial); break;
        case 128: hipLaunchKernelGGL((k_rmse_partial<128, T>), grid, block, 0, st, S, ntest, (const T*)P, (const T*)Q, partial); break;
        case 256: hipLaunchKernelGGL((k_rmse_partial<256, T>), grid, block, 0, st, S, ntest, (const T*)P, (const T*)Q, partial); break;
        case 512: hipLaunchKernelGGL((k_rmse_partial<512, T>), grid, block, 0, st, S, ntest, (const T*)P, (const T*)Q, partial); break;
        default: return hipErrorInvalidValue;
        }
        return hipGetLastError();
    }
    static hipError_t init(void* A, int64_t rows, int k, int KP, uint64_t stream, double inv_sqrt_k, hipStream_t st)
    {
        const int64_t total = rows * KP;
        int64_t blocks = (total + 255) / 256;
        if (blocks > 65536)
            blocks = 65536;
        hipLaunchKernelGGL((k_init<T>), dim3((unsigned)blocks), dim3(256), 0, st, (T*)A, rows, k, KP, stream,
                           inv_sqrt_k);
        return hipGetLastError();
    }
};

} // namespace mfsgd
