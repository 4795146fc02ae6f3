// Wavefront-per-row copy shared by the gather and pipelined kernels.
#pragma once

#include "scone_internal.h"

namespace scone {

// One wavefront copies the row of ids[r] (64*U 16-byte units: 1, 2, 4 or 8 KiB)
// into row r of `out`.  The id is wave-uniform, so every load is a scalar row
// base plus the lane offset; all U loads are issued before the U stores, which
// are non-temporal (the output is not re-read by this path).  An id outside
// [0, n_rows) writes a zero row and raises SCONE_EROW.  All 64 lanes call it.
template <int U>
__device__ __forceinline__ void copy_row_wave(const int32_t* __restrict__ ids, int64_t r,
                                              const u32x4* __restrict__ rows, int64_t n_rows,
                                              u32x4* __restrict__ out,
                                              unsigned* __restrict__ err) {
    const int lane = threadIdx.x & 63;
    const int64_t id = ids[r];
    const bool ok = (id >= 0) & (id < n_rows);
    const u32x4* src = rows + (ok ? id : 0) * (64 * U);
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = src[u * 64 + lane];
    u32x4* dst = out + r * (64 * U);
#pragma unroll
    for (int u = 0; u < U; ++u)
        __builtin_nontemporal_store(ok ? v[u] : u32x4{}, dst + u * 64 + lane);
    if (!ok && lane == 0) atomicOr(err, err_bit(SCONE_EROW));
}

// Units per row (16 bytes each) that copy_row_wave handles, as its U; 0 otherwise.
__host__ __device__ constexpr int wave_row_units(int64_t row_bytes) {
    return row_bytes == 1024 ? 1 : row_bytes == 2048 ? 2 : row_bytes == 4096 ? 4
                                                       : row_bytes == 8192 ? 8 : 0;
}

}  // namespace scone
