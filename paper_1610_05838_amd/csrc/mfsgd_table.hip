// mfsgd_table.hip -- the plan and the per-epoch state of the global
// scheduling table (LIBMF's policy, the baseline of section 3.2.1).
//
// The table's grid is finer than the wavefront-update grid (its side is a few
// times the number of workers, up to kMaxTableGrid = 1024, i.e. up to 2^20
// blocks), too many bins for the LDS-histogram planner of mfsgd_aux.hip.
// Here the samples are grouped by a stable radix sort of (block id, position)
// pairs: LSD radix sorting keeps equal keys in input order, so every block
// keeps its samples in array order, as the single-worker schedule requires.
#include <rocprim/device/device_radix_sort.hpp>

#include "mfsgd_device.hpp"
#include "mfsgd_launch.hpp"

namespace mfsgd {

static int key_bits(int s)
{
    const uint64_t nb = (uint64_t)s * (uint64_t)s;
    int bits = 1;
    while ((uint64_t(1) << bits) < nb)
        ++bits;
    return bits;
}

// key = block id floor(u*s/m) * s + floor(v*s/n), value = position; an index
// out of range raises *bad (its key is then meaningless and the plan is
// dropped by the caller).
__global__ void k_table_keys(const Sample* __restrict__ S, int64_t nnz, int64_t m, int64_t n, int s,
                             uint32_t* __restrict__ keys, uint32_t* __restrict__ vals, int* bad)
{
    int found = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nnz; i += (int64_t)gridDim.x * blockDim.x) {
        const int u = __builtin_nontemporal_load(&S[i].u);
        const int v = __builtin_nontemporal_load(&S[i].v);
        const bool ok = u >= 0 && u < m && v >= 0 && v < n;
        found |= !ok;
        const uint32_t rb = ok ? (uint32_t)(((int64_t)u * s) / m) : 0u;
        const uint32_t cb = ok ? (uint32_t)(((int64_t)v * s) / n) : 0u;
        keys[i] = rb * (uint32_t)s + cb;
        vals[i] = (uint32_t)i;
    }
    if (found)
        atomicOr(bad, 1);
}

// bstart[b] = first sorted position whose key is >= b, for b in [0, s*s];
// thread i (0 <= i <= nnz) fills the ids in (key[i-1], key[i]], with
// key[-1] = -1 and key[nnz] = s*s.
__global__ void k_table_starts(const uint32_t* __restrict__ keys, int64_t nnz, int64_t nblocks,
                               int64_t* __restrict__ bstart)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i <= nnz; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t prev = i == 0 ? -1 : (int64_t)keys[i - 1];
        const int64_t cur = i == nnz ? nblocks : (int64_t)keys[i];
        for (int64_t b = prev + 1; b <= cur; ++b)
            bstart[b] = i;
    }
}

__global__ void k_table_gather(const Sample* __restrict__ S, int64_t nnz, const uint32_t* __restrict__ pos,
                               Sample* __restrict__ Sp, int64_t* __restrict__ orig)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nnz; i += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t j = pos[i];
        Sp[i] = S[j];
        if (orig)
            orig[i] = (int64_t)j;
    }
}

static unsigned grid_for(int64_t items)
{
    int64_t blocks = (items + 255) / 256;
    if (blocks < 1)
        blocks = 1;
    if (blocks > 16384)
        blocks = 16384;
    return (unsigned)blocks;
}

size_t table_sort_bytes(int64_t nnz, int s)
{
    size_t bytes = 0;
    if (nnz <= 0)
        return 0;
    if (rocprim::radix_sort_pairs(nullptr, bytes, (uint32_t*)nullptr, (uint32_t*)nullptr, (uint32_t*)nullptr,
                                  (uint32_t*)nullptr, (size_t)nnz, 0, key_bits(s)) != hipSuccess)
        return 0;
    return bytes;
}

hipError_t table_plan_build(const Sample* S, int64_t nnz, int64_t m, int64_t n, int s, const TablePlanBuffers& b,
                            hipStream_t st)
{
    const int64_t nblocks = (int64_t)s * s;
    if (nnz > 0) {
        hipLaunchKernelGGL(k_table_keys, dim3(grid_for(nnz)), dim3(256), 0, st, S, nnz, m, n, s, b.keys[0], b.vals[0],
                           b.bad);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
        size_t bytes = b.temp_bytes;
        e = rocprim::radix_sort_pairs(b.temp, bytes, b.keys[0], b.keys[1], b.vals[0], b.vals[1], (size_t)nnz, 0,
                                      key_bits(s), st);
        if (e != hipSuccess)
            return e;
    }
    hipLaunchKernelGGL(k_table_starts, dim3(grid_for(nnz + 1)), dim3(256), 0, st, b.keys[1], nnz, nblocks, b.bstart);
    return hipGetLastError();
}

hipError_t table_plan_gather(const Sample* S, int64_t nnz, const TablePlanBuffers& b, hipStream_t st)
{
    if (nnz <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_table_gather, dim3(grid_for(nnz)), dim3(256), 0, st, S, nnz, b.vals[1], b.Sp, b.orig);
    return hipGetLastError();
}

__global__ void k_table_reset(uint32_t* __restrict__ tab, const uint32_t* __restrict__ blist, uint32_t nb, int s)
{
    const int64_t words = kTableHdr + 2 * (int64_t)s + nb;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < words; i += (int64_t)gridDim.x * blockDim.x) {
        uint32_t x = 0u;
        if (i == 1)
            x = nb;
        else if (i >= kTableHdr + 2 * (int64_t)s)
            x = blist[i - kTableHdr - 2 * (int64_t)s];
        tab[i] = x;
    }
}

hipError_t table_reset(uint32_t* tab, const uint32_t* blist, uint32_t nb, int s, hipStream_t st)
{
    hipLaunchKernelGGL(k_table_reset, dim3(grid_for(kTableHdr + 2 * (int64_t)s + nb)), dim3(256), 0, st, tab, blist,
                       nb, s);
    return hipGetLastError();
}

} // namespace mfsgd
