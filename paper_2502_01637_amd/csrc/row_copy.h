// Wavefront-per-row copy shared by the gather and pipelined kernels.
#pragma once

#include "scone_internal.h"

namespace scone {

// One wavefront copies part `part` of W equal parts of the row of ids[r]
// (64*U 16-byte units in all: 1, 2, 4 or 8 KiB) into row r of `out`.  The
// id is wave-uniform, so every load is a scalar row base plus the lane
// offset; all U/W loads are issued before the U/W stores, which are
// non-temporal (the output is not re-read by this path).  An id outside
// [0, n_rows) writes zeros and raises SCONE_EROW.  All 64 lanes call it.
template <int U, int W>
__device__ __forceinline__ void copy_row_part(const int32_t* __restrict__ ids, int64_t r,
                                              int part, const u32x4* __restrict__ rows,
                                              int64_t n_rows, u32x4* __restrict__ out,
                                              unsigned* __restrict__ err) {
    static_assert(W >= 1 && U % W == 0, "W must divide the row's units");
    constexpr int UW = U / W;
    const int lane = threadIdx.x & 63;
    const int64_t id = ids[r];
    const bool ok = (id >= 0) & (id < n_rows);
    const u32x4* src = rows + (ok ? id : 0) * (64 * U) + part * (64 * UW);
    u32x4 v[UW];
#pragma unroll
    for (int u = 0; u < UW; ++u) v[u] = src[u * 64 + lane];
    u32x4* dst = out + r * (64 * U) + part * (64 * UW);
#pragma unroll
    for (int u = 0; u < UW; ++u)
        __builtin_nontemporal_store(ok ? v[u] : u32x4{}, dst + u * 64 + lane);
    if (!ok && lane == 0 && part == 0) atomicOr(err, err_bit(SCONE_EROW));
}

// Wavefronts per row of 64*U units for the standalone gather and for the
// gather half of the pipelined step.  Measured on rows of 4 KiB over a 41 GB
// table: the standalone gather with 1 KiB per wavefront is 2% faster on the
// Zipf workload and 8% faster on uniform random ids than with whole rows;
// inside the pipelined step, next to the lookup workgroups, 2 KiB per
// wavefront is the fastest (whole rows and 1 KiB parts are 3-4% slower).
// Rows of 1 and 2 KiB stay whole: on the 2 KiB-row workload, 1 KiB parts
// cost 15% on its Zipf ids, which mostly hit the caches.
__host__ __device__ constexpr int gather_row_waves(int U) { return U >= 4 ? U : 1; }
__host__ __device__ constexpr int pipelined_row_waves(int U) { return U >= 4 ? U / 2 : 1; }

// Units per row (16 bytes each) that copy_row_part handles, as its U; 0 otherwise.
__host__ __device__ constexpr int wave_row_units(int64_t row_bytes) {
    return row_bytes == 1024 ? 1 : row_bytes == 2048 ? 2 : row_bytes == 4096 ? 4
                                                       : row_bytes == 8192 ? 8 : 0;
}

}  // namespace scone
