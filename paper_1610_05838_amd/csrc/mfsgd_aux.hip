// mfsgd_aux.hip -- storage-type independent kernels: RMSE final reduction,
// index checks, ticket reset and the wavefront-update planner.
#include "mfsgd_device.hpp"
#include "mfsgd_launch.hpp"

namespace mfsgd {

// Pass 2 of the test RMSE: one workgroup adds the kRmseWaves partial sums in
// a fixed order (strided per thread, then a fixed tree), so the result does
// not depend on timing.
__global__ __launch_bounds__(256) void k_rmse_final(const double* __restrict__ partial, int64_t ntest,
                                                    double* __restrict__ out)
{
    __shared__ double red[256];
    double acc = 0.0;
    for (int i = threadIdx.x; i < kRmseWaves; i += 256)
        acc += partial[i];
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w)
            red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0)
        out[0] = ntest > 0 ? sqrt(red[0] / (double)ntest) : 0.0;
}

hipError_t rmse_final(const double* partial, int64_t ntest, double* out, hipStream_t st)
{
    hipLaunchKernelGGL(k_rmse_final, dim3(1), dim3(256), 0, st, partial, ntest, out);
    return hipGetLastError();
}

__global__ void k_check(const Sample* __restrict__ S, int64_t nnz, int64_t m, int64_t n, int* bad)
{
    int found = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nnz; i += (int64_t)gridDim.x * blockDim.x) {
        const int u = __builtin_nontemporal_load(&S[i].u);
        const int v = __builtin_nontemporal_load(&S[i].v);
        found |= (u < 0) | (u >= m) | (v < 0) | (v >= n);
    }
    if (found)
        atomicOr(bad, 1);
}

hipError_t check_indices(const Sample* S, int64_t nnz, int64_t m, int64_t n, int* bad, hipStream_t st)
{
    if (nnz <= 0)
        return hipSuccess;
    int64_t blocks = (nnz + 255) / 256;
    if (blocks > 8192)
        blocks = 8192;
    hipLaunchKernelGGL(k_check, dim3((unsigned)blocks), dim3(256), 0, st, S, nnz, m, n, bad);
    return hipGetLastError();
}

__global__ void k_reset_tickets(uint32_t* tickets, uint32_t* sched)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < kMaxGrid)
        tickets[i] = 0u;
    if (i < kSchedWords)
        sched[i] = 0u;
}

hipError_t reset_tickets(uint32_t* tickets, uint32_t* sched, hipStream_t st)
{
    hipLaunchKernelGGL(k_reset_tickets, dim3((kSchedWords + 255) / 256), dim3(256), 0, st, tickets, sched);
    return hipGetLastError();
}

// Critical-path priorities of a block-scheduled epoch.  Block (t, w) is team
// t's block of wave w, column C[(t + O[w]) mod s]; it must be exhausted
// before the same team's block of wave w+1 can be claimed, and completed
// before the column's block of wave w+1 (team (t + O[w] - O[w+1]) mod s)
// opens.  prio[t*s + w] = the largest number of 64-sample units on a chain
// of such successors from (t, w) to the end of the epoch, its own included:
// the work that still has to follow this block one step at a time.  One
// workgroup, lane t for team t, waves from the last to the first.
__global__ __launch_bounds__(kMaxGrid) void k_block_priority(const int64_t* __restrict__ bstart, int s,
                                                            uint64_t sigma_c, uint64_t sigma_o,
                                                            uint32_t* __restrict__ prio)
{
    __shared__ int Cperm[kMaxGrid], Ooff[kMaxGrid];
    __shared__ uint64_t chain[kMaxGrid];
    const int t = threadIdx.x;
    if (t == 0) {
        shuffle_perm(sigma_c, s, Cperm);
        shuffle_perm(sigma_o, s, Ooff);
    }
    chain[t] = 0;
    __syncthreads();
    for (int w = s - 1; w >= 0; --w) {
        uint64_t v = 0;
        if (t < s) {
            const int64_t b = (int64_t)t * s + Cperm[(t + Ooff[w]) % s];
            v = (uint64_t)((bstart[b + 1] - bstart[b] + 63) / 64);
            if (w + 1 < s) {
                const int tc = ((t + Ooff[w] - Ooff[w + 1]) % s + s) % s;
                v += chain[t] > chain[tc] ? chain[t] : chain[tc];
            }
        }
        __syncthreads();
        if (t < s) {
            chain[t] = v;
            prio[(int64_t)t * s + w] = v > 0xffffffffull ? 0xffffffffu : (uint32_t)v;
        }
        __syncthreads();
    }
}

hipError_t block_priority(const int64_t* bstart, int s, uint64_t sigma_c, uint64_t sigma_o, uint32_t* prio,
                          hipStream_t st)
{
    hipLaunchKernelGGL(k_block_priority, dim3(1), dim3(kMaxGrid), 0, st, bstart, s, sigma_c, sigma_o, prio);
    return hipGetLastError();
}

// Which XCD (accelerator complex die) runs each workgroup: the hardware
// register XCC_ID of gfx94x/gfx950.
__global__ void k_probe_xcc(int* out)
{
    unsigned xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    if (threadIdx.x == 0)
        out[blockIdx.x] = (int)(xcc & 0xf);
}

hipError_t probe_xcc(int* out, int n, hipStream_t st)
{
    hipLaunchKernelGGL(k_probe_xcc, dim3(n), dim3(64), 0, st, out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Planner: a stable counting sort of the samples by block id
// (row block floor(u*s/m)) * s + (column block floor(v*s/n)).
//   1. each of kPlanChunks wavefronts counts its contiguous chunk per block
//      (and flags indices out of range);
//   2. per block, an exclusive scan over the chunks;
//   3. an exclusive scan over the blocks gives the block starts;
//   4. each wavefront walks its chunk in order, 64 samples at a time, ranks
//      equal blocks by lane (ballot peeling) and scatters the samples.
// Chunks, steps and lanes are all taken in array order, so every block keeps
// its samples in array order.
// ---------------------------------------------------------------------------
// Block cut: equal index ranges (floor(i*s/N)) when no bounds are given,
// else the consecutive ranges bounds[0..s] (index i is in the last range
// whose first index is <= i).
struct Cut {
    int64_t rb[kMaxGrid + 1];
    int64_t cb[kMaxGrid + 1];
    bool bounded;
};

__device__ __forceinline__ void load_cut(Cut& c, const int64_t* rbnd, const int64_t* cbnd, int s)
{
    c.bounded = rbnd != nullptr;
    if (c.bounded)
        for (int i = threadIdx.x; i <= s; i += blockDim.x) {
            c.rb[i] = rbnd[i];
            c.cb[i] = cbnd[i];
        }
}

__device__ __forceinline__ int range_of(int64_t i, const int64_t* b, int s)
{
    int lo = 0, hi = s - 1; // largest k in [0, s-1] with b[k] <= i
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (b[mid] <= i)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

__device__ __forceinline__ int block_of(int u, int v, int64_t m, int64_t n, int s, const Cut& c)
{
    if (c.bounded)
        return range_of(u, c.rb, s) * s + range_of(v, c.cb, s);
    const int rb = (int)(((int64_t)u * s) / m);
    const int cb = (int)(((int64_t)v * s) / n);
    return rb * s + cb;
}

// Per-index sample counts (users and items) for the balanced cut and the
// hot-row/column measures; indices out of range are skipped and flagged.
// A workgroup counts a tile of kDegTile samples into open-addressed LDS
// tables (kDegSlots slots each, so at most half full: every probe sequence
// ends), then adds each distinct index's count to global memory once.  Under
// Zipf-like popularity one index can hold several percent of all samples;
// per-sample global atomics on its counter would serialise.
constexpr int kDegTile = 2048;
constexpr int kDegSlots = 4096;
static_assert(kDegSlots >= 2 * kDegTile, "degree tables must stay at most half full");

__device__ __forceinline__ void deg_insert(int* keys, unsigned* cnt, int key)
{
    unsigned h = ((unsigned)key * 2654435761u) >> 20; // 12 bits: kDegSlots = 4096
    for (;;) {
        const int old = atomicCAS(&keys[h], -1, key);
        if (old == -1 || old == key) {
            atomicAdd(&cnt[h], 1u);
            return;
        }
        h = (h + 1) & (kDegSlots - 1);
    }
}

__global__ __launch_bounds__(256) void k_degrees(const Sample* __restrict__ S, int64_t nnz, int64_t m, int64_t n,
                                                 unsigned long long* __restrict__ du,
                                                 unsigned long long* __restrict__ dv, int* bad)
{
    __shared__ int ku[kDegSlots], kv[kDegSlots];
    __shared__ unsigned cu[kDegSlots], cv[kDegSlots];
    for (int j = threadIdx.x; j < kDegSlots; j += blockDim.x) {
        ku[j] = kv[j] = -1;
        cu[j] = cv[j] = 0u;
    }
    __syncthreads();
    int found = 0;
    const int64_t tiles = (nnz + kDegTile - 1) / kDegTile;
    for (int64_t t = blockIdx.x; t < tiles; t += gridDim.x) {
        const int64_t lo = t * kDegTile;
        const int64_t hi = lo + kDegTile < nnz ? lo + kDegTile : nnz;
        for (int64_t i = lo + threadIdx.x; i < hi; i += blockDim.x) {
            const int u = __builtin_nontemporal_load(&S[i].u);
            const int v = __builtin_nontemporal_load(&S[i].v);
            if (u < 0 || u >= m || v < 0 || v >= n) {
                found = 1;
                continue;
            }
            deg_insert(ku, cu, u);
            deg_insert(kv, cv, v);
        }
        __syncthreads();
        for (int j = threadIdx.x; j < kDegSlots; j += blockDim.x) {
            if (ku[j] >= 0) {
                atomicAdd(du + ku[j], (unsigned long long)cu[j]);
                ku[j] = -1;
                cu[j] = 0u;
            }
            if (kv[j] >= 0) {
                atomicAdd(dv + kv[j], (unsigned long long)cv[j]);
                kv[j] = -1;
                cv[j] = 0u;
            }
        }
        __syncthreads();
    }
    if (found)
        atomicOr(bad, 1);
}

// One thread per 32 rows: no atomics, every word written once.
__global__ void k_hot_bits(const unsigned long long* __restrict__ deg, int64_t rows, unsigned long long thr,
                           uint32_t* __restrict__ bits)
{
    const int64_t words = (rows + 31) / 32;
    for (int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; w < words; w += (int64_t)gridDim.x * blockDim.x) {
        uint32_t b = 0;
        for (int i = 0; i < 32; ++i) {
            const int64_t r = w * 32 + i;
            if (r < rows && deg[r] >= thr)
                b |= 1u << i;
        }
        bits[w] = b;
    }
}

hipError_t hot_bits(const unsigned long long* deg, int64_t rows, unsigned long long thr, uint32_t* bits,
                    hipStream_t st)
{
    const int64_t words = (rows + 31) / 32;
    if (words == 0)
        return hipSuccess;
    int64_t blocks = (words + 255) / 256;
    if (blocks > 4096)
        blocks = 4096;
    hipLaunchKernelGGL(k_hot_bits, dim3((unsigned)blocks), dim3(256), 0, st, deg, rows, thr, bits);
    return hipGetLastError();
}

// Largest entry of deg[0 .. rows-1], atomically folded into *out (which the
// caller zeroes).
__global__ void k_max_u64(const unsigned long long* __restrict__ deg, int64_t rows, unsigned long long* out)
{
    unsigned long long mx = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < rows; i += (int64_t)gridDim.x * blockDim.x)
        mx = deg[i] > mx ? deg[i] : mx;
    for (int o = 32; o > 0; o >>= 1) {
        const unsigned long long y = __shfl_xor(mx, o);
        mx = y > mx ? y : mx;
    }
    if ((threadIdx.x & 63) == 0 && mx > 0)
        atomicMax(out, mx);
}

hipError_t max_degree(const unsigned long long* deg, int64_t rows, unsigned long long* out, hipStream_t st)
{
    if (rows <= 0)
        return hipSuccess;
    int64_t blocks = (rows + 255) / 256;
    if (blocks > 1024)
        blocks = 1024;
    hipLaunchKernelGGL(k_max_u64, dim3((unsigned)blocks), dim3(256), 0, st, deg, rows, out);
    return hipGetLastError();
}

hipError_t plan_degrees(const Sample* S, int64_t nnz, int64_t m, int64_t n, unsigned long long* du,
                        unsigned long long* dv, int* bad, hipStream_t st)
{
    if (nnz <= 0)
        return hipSuccess;
    int64_t blocks = (nnz + kDegTile - 1) / kDegTile;
    if (blocks > 2048)
        blocks = 2048;
    hipLaunchKernelGGL(k_degrees, dim3((unsigned)blocks), dim3(256), 0, st, S, nnz, m, n, du, dv, bad);
    return hipGetLastError();
}

__global__ __launch_bounds__(64) void k_plan_count(const Sample* __restrict__ S, int64_t nnz, int64_t m, int64_t n,
                                                   int s, const int64_t* rbnd, const int64_t* cbnd,
                                                   int64_t* __restrict__ counts, int chunks, int* bad)
{
    __shared__ int hist[kMaxGrid * kMaxGrid];
    __shared__ Cut cut;
    const int nb = s * s;
    for (int i = threadIdx.x; i < nb; i += 64)
        hist[i] = 0;
    load_cut(cut, rbnd, cbnd, s);
    __syncthreads();
    const int64_t cs = (nnz + chunks - 1) / chunks;
    const int64_t lo = (int64_t)blockIdx.x * cs;
    const int64_t hi = lo + cs < nnz ? lo + cs : nnz;
    int found = 0;
    for (int64_t i = lo + threadIdx.x; i < hi; i += 64) {
        const int u = __builtin_nontemporal_load(&S[i].u);
        const int v = __builtin_nontemporal_load(&S[i].v);
        if (u < 0 || u >= m || v < 0 || v >= n) {
            found = 1;
            continue;
        }
        atomicAdd(&hist[block_of(u, v, m, n, s, cut)], 1);
    }
    if (found)
        atomicOr(bad, 1);
    __syncthreads();
    for (int b = threadIdx.x; b < nb; b += 64)
        counts[(int64_t)b * chunks + blockIdx.x] = hist[b];
}

// exclusive scan of counts[b][0..chunks) in place, total to totals[b]
// (chunks is a multiple of 256; thread j scans chunks j*per .. j*per+per-1)
__global__ __launch_bounds__(256) void k_plan_scan_chunks(int64_t* __restrict__ counts, int chunks,
                                                          int64_t* __restrict__ totals)
{
    const int per = chunks / 256;
    __shared__ int64_t part[256];
    int64_t* row = counts + (int64_t)blockIdx.x * chunks + (int64_t)threadIdx.x * per;
    int64_t acc = 0;
    for (int i = 0; i < per; ++i)
        acc += row[i];
    part[threadIdx.x] = acc;
    __syncthreads();
    // inclusive Hillis-Steele scan of the 256 thread sums
    for (int off = 1; off < 256; off <<= 1) {
        int64_t add = (int)threadIdx.x >= off ? part[threadIdx.x - off] : 0;
        __syncthreads();
        part[threadIdx.x] += add;
        __syncthreads();
    }
    int64_t run = threadIdx.x > 0 ? part[threadIdx.x - 1] : 0;
    for (int i = 0; i < per; ++i) {
        const int64_t x = row[i];
        row[i] = run;
        run += x;
    }
    if (threadIdx.x == 255)
        totals[blockIdx.x] = part[255];
}

// exclusive scan of the block totals: bstart[0..nb]
__global__ __launch_bounds__(1024) void k_plan_scan_blocks(const int64_t* __restrict__ totals, int nb,
                                                           int64_t* __restrict__ bstart)
{
    constexpr int per = (kMaxGrid * kMaxGrid) / 1024;
    __shared__ int64_t part[1024];
    int64_t local[per];
    int64_t acc = 0;
#pragma unroll
    for (int i = 0; i < per; ++i) {
        const int b = threadIdx.x * per + i;
        local[i] = b < nb ? totals[b] : 0;
        acc += local[i];
    }
    part[threadIdx.x] = acc;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
        int64_t add = (int)threadIdx.x >= off ? part[threadIdx.x - off] : 0;
        __syncthreads();
        part[threadIdx.x] += add;
        __syncthreads();
    }
    int64_t run = threadIdx.x > 0 ? part[threadIdx.x - 1] : 0;
#pragma unroll
    for (int i = 0; i < per; ++i) {
        const int b = threadIdx.x * per + i;
        if (b < nb)
            bstart[b] = run;
        run += local[i];
    }
    if (threadIdx.x == 1023)
        bstart[nb] = part[1023];
}

__global__ __launch_bounds__(64) void k_plan_scatter(const Sample* __restrict__ S, int64_t nnz, int64_t m, int64_t n,
                                                     int s, const int64_t* rbnd, const int64_t* cbnd,
                                                     const int64_t* __restrict__ counts, int chunks,
                                                     const int64_t* __restrict__ bstart, Sample* __restrict__ Sp,
                                                     int64_t* __restrict__ orig)
{
    __shared__ int64_t base[kMaxGrid * kMaxGrid];
    __shared__ Cut cut;
    const int nb = s * s;
    for (int b = threadIdx.x; b < nb; b += 64)
        base[b] = bstart[b] + counts[(int64_t)b * chunks + blockIdx.x];
    load_cut(cut, rbnd, cbnd, s);
    __syncthreads();
    const int lane = threadIdx.x;
    const uint64_t below = (lane == 0) ? 0ull : ((~0ull) >> (64 - lane));
    const int64_t cs = (nnz + chunks - 1) / chunks;
    const int64_t lo = (int64_t)blockIdx.x * cs;
    const int64_t hi = lo + cs < nnz ? lo + cs : nnz;
    for (int64_t c0 = lo; c0 < hi; c0 += 64) {
        const int64_t i = c0 + lane;
        bool valid = i < hi;
        Sample x{0, 0, 0.f};
        int b = -1;
        if (valid) {
            x.u = __builtin_nontemporal_load(&S[i].u);
            x.v = __builtin_nontemporal_load(&S[i].v);
            x.r = __builtin_nontemporal_load(&S[i].r);
            valid = x.u >= 0 && x.u < m && x.v >= 0 && x.v < n; // the host never scatters a plan with bad indices
            if (valid)
                b = block_of(x.u, x.v, m, n, s, cut);
        }
        uint64_t pending = __ballot(valid);
        int64_t dest = -1;
        while (pending) {
            const int leader = __ffsll((unsigned long long)pending) - 1;
            const int lb = __builtin_amdgcn_readlane(b, leader);
            const uint64_t same = __ballot(b == lb) & pending;
            const int64_t at = base[lb];
            if ((same >> lane) & 1ull)
                dest = at + __popcll(same & below);
            __syncthreads();
            if (lane == leader)
                base[lb] = at + __popcll(same);
            __syncthreads();
            pending &= ~same;
        }
        if (valid) {
            Sp[dest] = x;
            if (orig)
                orig[dest] = i;
        }
    }
}

hipError_t plan_build(const Sample* S, int64_t nnz, int64_t m, int64_t n, int s, const PlanBuffers& b,
                      hipStream_t st)
{
    const int nb = s * s;
    if (b.chunks < 256 || b.chunks % 256 != 0)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_plan_count, dim3(b.chunks), dim3(64), 0, st, S, nnz, m, n, s, b.rbnd, b.cbnd, b.counts,
                       b.chunks, b.bad);
    hipLaunchKernelGGL(k_plan_scan_chunks, dim3(nb), dim3(256), 0, st, b.counts, b.chunks, b.totals);
    hipLaunchKernelGGL(k_plan_scan_blocks, dim3(1), dim3(1024), 0, st, b.totals, nb, b.bstart);
    return hipGetLastError();
}

hipError_t plan_scatter(const Sample* S, int64_t nnz, int64_t m, int64_t n, int s, const PlanBuffers& b,
                        hipStream_t st)
{
    hipLaunchKernelGGL(k_plan_scatter, dim3(b.chunks), dim3(64), 0, st, S, nnz, m, n, s, b.rbnd, b.cbnd,
                       b.counts, b.chunks, b.bstart, b.Sp, b.orig);
    return hipGetLastError();
}

} // namespace mfsgd
