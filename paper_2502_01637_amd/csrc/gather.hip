// Row gather: out[k, :] = rows[ids[k], :] as raw bytes.
//
// The embedding fetch is a pure memory copy (Section 1), so the kernel is an
// HBM-bound streaming copy whose source rows are chosen by the ids.  Rows of
// 1 or 2 KiB (16-byte aligned) take one wavefront per row, rows of 4 or 8 KiB
// one wavefront per KiB (gather_row_waves).  Any other
// width views the output as a flat array of V-sized units (16 bytes when the
// row width and the pointers allow).  Consecutive lanes own consecutive units, so
// one wavefront reads 64 * 16 B = 1 KiB of one row per instruction and writes
// the same 1 KiB of the output; each thread issues all of its U loads before
// its U stores to keep enough bytes in flight.  Output stores are
// non-temporal: the output is not re-read by this path, and keeping it out of
// the caches leaves them to the table rows that repeat (frequent tokens).
// The same kernel reads a host-mapped pinned table over PCIe when the rows
// live off the accelerator.
#include "row_copy.h"

namespace scone {
namespace {

constexpr int kGatherThreads = 256;

template <typename V, int U, bool kPow2>
__global__ __launch_bounds__(kGatherThreads) void k_gather(
    const int32_t* __restrict__ ids, int64_t total, const V* __restrict__ rows, int64_t n_rows,
    int64_t upr, int shift, V* __restrict__ out, unsigned* __restrict__ err, int64_t block0) {
    const int64_t base = block_index(block0) * (kGatherThreads * U) + threadIdx.x;
    V v[U];
    bool ok[U];
    if (base + (int64_t)(U - 1) * kGatherThreads < total) {
        // Whole block in range: every load is unconditional so that all U
        // id loads, then all U row loads, are in flight together.  A bad id
        // reads row 0 instead and its unit is zeroed afterwards.
        int64_t id[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = base + (int64_t)u * kGatherThreads;
            id[u] = ids[kPow2 ? (i >> shift) : (i / upr)];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = base + (int64_t)u * kGatherThreads;
            const int64_t r = kPow2 ? (i >> shift) : (i / upr);
            const int64_t c = i - r * upr;
            ok[u] = (id[u] >= 0) & (id[u] < n_rows);
            const int64_t src = ok[u] ? id[u] : 0;
            v[u] = rows[(kPow2 ? (src << shift) : src * upr) + c];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (!ok[u]) v[u] = V{};
            __builtin_nontemporal_store(v[u], out + base + (int64_t)u * kGatherThreads);
        }
    } else {
        // Ragged last block.
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = base + (int64_t)u * kGatherThreads;
            ok[u] = true;
            if (i < total) {
                const int64_t r = kPow2 ? (i >> shift) : (i / upr);
                const int64_t c = i - r * upr;
                const int64_t id = ids[r];
                ok[u] = (id >= 0) & (id < n_rows);
                v[u] = ok[u] ? rows[id * upr + c] : V{};
                __builtin_nontemporal_store(v[u], out + i);
            }
        }
    }
    bool bad = false;
#pragma unroll
    for (int u = 0; u < U; ++u) bad |= !ok[u];
    if (bad) atomicOr(err, err_bit(SCONE_EROW));
}

// Rows of 64*U 16-byte units (1, 2, 4 or 8 KiB): W = gather_row_waves(U) wavefronts
// per row, each copying one W-th of it; consecutive wavefronts of a workgroup
// take consecutive parts.
template <int U>
__global__ __launch_bounds__(kGatherThreads) void k_gather_rows(
    const int32_t* __restrict__ ids, int64_t n_tok, const u32x4* __restrict__ rows,
    int64_t n_rows, u32x4* __restrict__ out, unsigned* __restrict__ err, int64_t block0) {
    constexpr int W = gather_row_waves(U);
    const int64_t w = block_index(block0) * (kGatherThreads / 64) +
                      __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t r = w / W;
    if (r >= n_tok) return;  // wave-uniform
    copy_row_part<U, W>(ids, r, (int)(w - r * W), rows, n_rows, out, err);
}

// Every id is out of range when the table has no rows: zero the output.
template <typename V>
__global__ __launch_bounds__(kGatherThreads) void k_zero(int64_t total, V* __restrict__ out,
                                                         unsigned* __restrict__ err,
                                                         int64_t block0) {
    const int64_t i = block_index(block0) * kGatherThreads + threadIdx.x;
    if (i < total) out[i] = V{};
    if (i == 0) atomicOr(err, err_bit(SCONE_EROW));
}

template <typename V>
hipError_t launch_zero(int64_t total, V* out, unsigned* err, hipStream_t st) {
    return launch_blocks((total + kGatherThreads - 1) / kGatherThreads, kGatherThreads,
                         [&](int64_t b0, dim3 grid) {
                             hipLaunchKernelGGL(k_zero<V>, grid, dim3(kGatherThreads), 0, st,
                                                total, out, err, b0);
                         });
}

template <typename V, int U>
hipError_t launch_gather(const int32_t* ids, int64_t n_tok, const void* rows, int64_t n_rows,
                         int64_t row_bytes, void* out, unsigned* err, hipStream_t st) {
    const int64_t upr = row_bytes / (int64_t)sizeof(V);
    const int64_t total = n_tok * upr;
    if (n_rows == 0) return launch_zero(total, static_cast<V*>(out), err, st);
    const int64_t blocks = (total + kGatherThreads * U - 1) / (kGatherThreads * U);
    const bool pow2 = (upr & (upr - 1)) == 0;
    int shift = 0;
    while (((int64_t)1 << shift) < upr) ++shift;
    return launch_blocks(blocks, kGatherThreads, [&](int64_t b0, dim3 grid) {
        if (pow2)
            hipLaunchKernelGGL((k_gather<V, U, true>), grid, dim3(kGatherThreads), 0, st, ids,
                               total, static_cast<const V*>(rows), n_rows, upr, shift,
                               static_cast<V*>(out), err, b0);
        else
            hipLaunchKernelGGL((k_gather<V, U, false>), grid, dim3(kGatherThreads), 0, st, ids,
                               total, static_cast<const V*>(rows), n_rows, upr, shift,
                               static_cast<V*>(out), err, b0);
    });
}

}  // namespace

hipError_t launch_zero_rows(void* out, int64_t bytes, unsigned* err, hipStream_t st) {
    return launch_zero(bytes, static_cast<uint8_t*>(out), err, st);
}

hipError_t launch_gather_any(const int32_t* ids, int64_t n_tok, const void* rows, int64_t n_rows,
                             int64_t row_bytes, void* out, unsigned* err, hipStream_t st) {
    // Widest unit that divides the row width and both base addresses.
    const uintptr_t align = (uintptr_t)rows | (uintptr_t)out | (uintptr_t)row_bytes;
    const int64_t upr16 = row_bytes / 16;
    if ((align & 15) == 0 && n_rows > 0 &&
        (upr16 == 64 || upr16 == 128 || upr16 == 256 || upr16 == 512)) {
        const int64_t waves = n_tok * gather_row_waves((int)upr16 / 64);
        const int64_t blocks = (waves + kGatherThreads / 64 - 1) / (kGatherThreads / 64);
        const u32x4* R = static_cast<const u32x4*>(rows);
        u32x4* O = static_cast<u32x4*>(out);
        return launch_blocks(blocks, kGatherThreads, [&](int64_t b0, dim3 grid) {
            const dim3 block(kGatherThreads);
            switch (upr16) {
                case 64: hipLaunchKernelGGL(k_gather_rows<1>, grid, block, 0, st, ids, n_tok, R, n_rows, O, err, b0); break;
                case 128: hipLaunchKernelGGL(k_gather_rows<2>, grid, block, 0, st, ids, n_tok, R, n_rows, O, err, b0); break;
                case 256: hipLaunchKernelGGL(k_gather_rows<4>, grid, block, 0, st, ids, n_tok, R, n_rows, O, err, b0); break;
                default: hipLaunchKernelGGL(k_gather_rows<8>, grid, block, 0, st, ids, n_tok, R, n_rows, O, err, b0); break;
            }
        });
    }
    if ((align & 15) == 0)
        return launch_gather<u32x4, 4>(ids, n_tok, rows, n_rows, row_bytes, out, err, st);
    if ((align & 7) == 0)
        return launch_gather<u32x2, 4>(ids, n_tok, rows, n_rows, row_bytes, out, err, st);
    if ((align & 3) == 0)
        return launch_gather<uint32_t, 4>(ids, n_tok, rows, n_rows, row_bytes, out, err, st);
    if ((align & 1) == 0)
        return launch_gather<uint16_t, 4>(ids, n_tok, rows, n_rows, row_bytes, out, err, st);
    return launch_gather<uint8_t, 4>(ids, n_tok, rows, n_rows, row_bytes, out, err, st);
}

}  // namespace scone

extern "C" int scone_gather(const int32_t* fgram_ids, int64_t n_tok, const void* rows,
                            int64_t n_rows, int64_t row_bytes, void* out, int32_t placement,
                            void* stream) {
    using namespace scone;
    if (n_tok < 0 || n_rows < 0 || row_bytes <= 0) return SCONE_EINVAL;
    if (placement != SCONE_PLACE_HBM && placement != SCONE_PLACE_HOST) return SCONE_EINVAL;
    if (n_tok > ((int64_t)1 << 62) / row_bytes) return SCONE_EINVAL;
    if (n_tok == 0) return SCONE_OK;
    if (!fgram_ids || !out || (!rows && n_rows > 0)) return SCONE_EINVAL;
    // Rows are written while other wavefronts still read their ids and rows.
    const int64_t out_b = n_tok * row_bytes;
    if (overlaps(out, out_b, fgram_ids, span_bytes(n_tok, 4)) ||
        overlaps(out, out_b, rows, span_bytes(n_rows, row_bytes)))
        return SCONE_EINVAL;
    unsigned* err = device_error_word();
    if (!err) return SCONE_EHIP;
    const hipError_t e = launch_gather_any(fgram_ids, n_tok, rows, n_rows, row_bytes, out, err,
                                           static_cast<hipStream_t>(stream));
    return status_of(e);
}
