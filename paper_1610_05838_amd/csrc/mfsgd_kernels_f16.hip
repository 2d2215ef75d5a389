// mfsgd_kernels_f16.hip -- kernel instantiations for binary16 feature storage.
#include "mfsgd_kernels.hpp"

namespace mfsgd {

hipError_t epoch_f16(const EpochLaunch& a, hipStream_t st) { return Dispatch<half_t>::epoch(a, st); }

hipError_t table_epoch_f16(const TableLaunch& a, hipStream_t st) { return Dispatch<half_t>::table_epoch(a, st); }

int occupancy_f16(int KP, int depth, int half) { return Dispatch<half_t>::occupancy(KP, depth, half != 0); }

int occupancy_blocked_f16(int KP, int depth, int threads, int half)
{
    return Dispatch<half_t>::occupancy_blocked(KP, depth, threads, half != 0);
}

hipError_t rmse_partial_f16(int KP, const Sample* S, int64_t ntest, const void* P, const void* Q, double* partial,
                           hipStream_t st)
{
    return Dispatch<half_t>::rmse(KP, S, ntest, P, Q, partial, st);
}

hipError_t init_f16(void* A, int64_t rows, int k, int KP, uint64_t stream, double inv_sqrt_k, hipStream_t st)
{
    return Dispatch<half_t>::init(A, rows, k, KP, stream, inv_sqrt_k, st);
}

} // namespace mfsgd
