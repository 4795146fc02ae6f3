// Fused lookup + gather: Algorithm 1's inference branch in one pass.
//
// Each workgroup first resolves the longest match for its tile of positions
// (the same tile lookup as scone_lookup, ids kept in LDS), then copies the
// tile's rows into the contiguous output block that those positions own.
// Fusing removes the id round trip through HBM and the separate
// latency-bound lookup launch.  Tiles are small (16 to 32 KiB of rows) so the
// grid holds many generations of short-lived workgroups: some wait on hash
// probes while the others on the same compute unit keep HBM busy with row
// copies.  Measured on MI355X this matches, within a few percent, the two
// separate kernels back to back: the hash probes are random HBM reads that
// cost bandwidth the row stream would otherwise use, so overlapping them
// hides their latency but not their cost.
#include "tile_lookup.h"

namespace scone {
namespace {

// Row copy helpers for one batch of U units per thread (unit i of the tile's
// output block).  A bad id reads row 0 and the unit is zeroed afterwards, so
// the loads of a batch carry no branch and stay in flight together.
template <typename V, int U, bool kPow2>
struct TileCopy {
    const int32_t* s_id;
    const V* __restrict__ rows;
    V* __restrict__ dst;
    int64_t n_rows, upr;
    int shift;

    __device__ __forceinline__ void load(int64_t base, V (&v)[U], bool (&ok)[U]) const {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = base + (int64_t)u * kTileThreads;
            const int64_t r = kPow2 ? (i >> shift) : (i / upr);
            const int64_t c = i - r * upr;
            const int64_t id = s_id[r];
            ok[u] = (id >= 0) & (id < n_rows);
            const int64_t src = ok[u] ? id : 0;
            v[u] = rows[(kPow2 ? (src << shift) : src * upr) + c];
        }
    }
    __device__ __forceinline__ bool store(int64_t base, V (&v)[U], const bool (&ok)[U]) const {
        bool bad = false;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            __builtin_nontemporal_store(ok[u] ? v[u] : V{}, dst + base + (int64_t)u * kTileThreads);
            bad |= !ok[u];
        }
        return bad;
    }
};

template <int SB, int G, typename V, int U, bool kPow2>
__global__ __launch_bounds__(kTileThreads) void k_embed(
    const typename SlotOps<SB>::Slot* __restrict__ slots, uint64_t mask,
    const int32_t* __restrict__ X, int64_t T, int P, int max_n, int64_t tiles_per_row,
    const V* __restrict__ rows, int64_t n_rows, int64_t upr, int shift, V* __restrict__ out,
    int32_t* __restrict__ ids_out, int8_t* __restrict__ len_out, unsigned* __restrict__ err,
    int64_t block0) {
    __shared__ int32_t s_tok[TileShape<G>::kPositions + kMaxHalo];
    __shared__ int32_t s_id[TileShape<G>::kPositions];

    const int64_t blk = block_index(block0);
    const int64_t b = blk / tiles_per_row;
    const int64_t t0 = (blk - b * tiles_per_row) * (int64_t)P;
    stage_tokens(s_tok, X + b * T, T, t0, P, max_n - 1);
    __syncthreads();
    if (threadIdx.x < ((P * G + 63) & ~63)) {  // whole waves only
        int32_t id;
        int len;
        bool tok_ok;
        tile_lookup<SB, G>(slots, mask, s_tok, T, t0, P, max_n, id, len, tok_ok);
        const int p = threadIdx.x / G;
        const int64_t t = t0 + p;
        if (threadIdx.x % G == 0 && p < P) {
            s_id[p] = id;
            if (t < T) {
                if (!tok_ok) atomicOr(err, err_bit(SCONE_ETOKEN));
                if (ids_out) ids_out[b * T + t] = id;
                if (len_out) len_out[b * T + t] = (int8_t)len;
            }
        }
    }
    __syncthreads();

    // Copy the tile's rows: positions t0 .. t0+npos-1 own one contiguous
    // output block of npos * upr units.  Whole batches are software-pipelined
    // (the next batch's loads are issued before this batch's stores).
    const int64_t npos = (T - t0) < P ? (T - t0) : P;
    const int64_t total = npos * upr;
    const TileCopy<V, U, kPow2> cp{s_id, rows, out + (b * T + t0) * upr, n_rows, upr, shift};
    constexpr int64_t kStride = (int64_t)kTileThreads * U;
    const int64_t whole = total / kStride * kStride;
    bool bad = false;
    int64_t base = threadIdx.x;
    if (whole > 0) {
        V a[U];
        bool oka[U];
        cp.load(base, a, oka);
        for (; base + kStride < whole; base += kStride) {
            V nb[U];
            bool okb[U];
            cp.load(base + kStride, nb, okb);
            bad |= cp.store(base, a, oka);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                a[u] = nb[u];
                oka[u] = okb[u];
            }
        }
        bad |= cp.store(base, a, oka);
        base += kStride;
    }
    for (int64_t i = base; i < total; i += kTileThreads) {  // ragged remainder
        const int64_t r = kPow2 ? (i >> shift) : (i / upr);
        const int64_t c = i - r * upr;
        const int64_t id = s_id[r];
        const bool okk = (id >= 0) & (id < n_rows);
        __builtin_nontemporal_store(okk ? rows[id * upr + c] : V{}, cp.dst + i);
        bad |= !okk;
    }
    if (bad) atomicOr(err, err_bit(SCONE_EROW));
}

template <int SB, int G, typename V, bool kPow2>
hipError_t launch(const scone_table* tb, const int32_t* X, int64_t B, int64_t T, int max_n,
                  const void* rows, int64_t n_rows, int64_t upr, int shift, void* out,
                  int32_t* ids, int8_t* lens, unsigned* err, hipStream_t st) {
    using Slot = typename SlotOps<SB>::Slot;
    // Positions per workgroup: up to 16 positions and 32 KiB of rows, at
    // least 4 positions.  Short-lived workgroups let the probes of some
    // overlap the copies of others on the same compute unit (16 to 32 KiB
    // per workgroup measured best for 2 and 4 KiB rows).
    const int64_t row_bytes = upr * (int64_t)sizeof(V);
    int P = TileShape<G>::kPositions < 16 ? TileShape<G>::kPositions : 16;
    while (P > 4 && (int64_t)P * row_bytes > (32 << 10)) P >>= 1;
    const int64_t tiles = (T + P - 1) / P;
    return launch_blocks(B * tiles, kTileThreads, [&](int64_t b0, dim3 grid) {
        hipLaunchKernelGGL((k_embed<SB, G, V, 4, kPow2>), grid, dim3(kTileThreads), 0, st,
                           static_cast<const Slot*>(tb->slots), (uint64_t)tb->capacity - 1, X,
                           T, P, max_n, tiles, static_cast<const V*>(rows), n_rows, upr, shift,
                           static_cast<V*>(out), ids, lens, err, b0);
    });
}

template <int SB, typename V, bool kPow2>
hipError_t dispatch(const scone_table* tb, const int32_t* X, int64_t B, int64_t T, int max_n,
                    const void* rows, int64_t n_rows, int64_t upr, int shift, void* out,
                    int32_t* ids, int8_t* lens, unsigned* err, hipStream_t st) {
    if (tile_lanes_for(max_n) == 1)
        return launch<SB, 1, V, kPow2>(tb, X, B, T, max_n, rows, n_rows, upr, shift, out, ids,
                                       lens, err, st);
    return launch<SB, 2, V, kPow2>(tb, X, B, T, max_n, rows, n_rows, upr, shift, out, ids, lens,
                                   err, st);
}

template <typename V, bool kPow2>
hipError_t dispatch_slots(const scone_table* tb, const int32_t* X, int64_t B, int64_t T,
                          int max_n, const void* rows, int64_t n_rows, int64_t upr, int shift,
                          void* out, int32_t* ids, int8_t* lens, unsigned* err, hipStream_t st) {
    return tb->slot_bytes == 16
               ? dispatch<16, V, kPow2>(tb, X, B, T, max_n, rows, n_rows, upr, shift, out, ids,
                                        lens, err, st)
               : dispatch<32, V, kPow2>(tb, X, B, T, max_n, rows, n_rows, upr, shift, out, ids,
                                        lens, err, st);
}

}  // namespace
}  // namespace scone

extern "C" int scone_embed(const scone_table_t* table, const int32_t* token_ids, int64_t B,
                           int64_t T, int32_t max_n, const void* rows, int64_t n_rows,
                           int64_t row_bytes, int32_t placement, void* out, int32_t* fgram_ids,
                           int8_t* match_len, void* stream) {
    using namespace scone;
    if (!table || B < 0 || T < 0 || max_n < 1 || n_rows < 0 || row_bytes <= 0)
        return SCONE_EINVAL;
    if (placement != SCONE_PLACE_HBM && placement != SCONE_PLACE_HOST) return SCONE_EINVAL;
    if (B > 0 && T > ((int64_t)1 << 62) / B) return SCONE_EINVAL;
    if (B * T > ((int64_t)1 << 62) / row_bytes) return SCONE_EINVAL;
    if (B * T == 0) return SCONE_OK;
    if (!token_ids || !out || (!rows && n_rows > 0)) return SCONE_EINVAL;
    {
        const int64_t n = B * T, out_b = n * row_bytes;
        const void* outs[3] = {out, fgram_ids, match_len};
        const int64_t outs_b[3] = {out_b, span_bytes(n, 4), n};
        for (int i = 0; i < 3; ++i) {
            if (overlaps(outs[i], outs_b[i], token_ids, span_bytes(n, 4)) ||
                overlaps(outs[i], outs_b[i], rows, span_bytes(n_rows, row_bytes)))
                return SCONE_EINVAL;
            for (int j = i + 1; j < 3; ++j)
                if (overlaps(outs[i], outs_b[i], outs[j], outs_b[j])) return SCONE_EINVAL;
        }
    }
    int dev = 0;
    SCONE_HIP_TRY(hipGetDevice(&dev));
    if (dev != table->device) return SCONE_EINVAL;
    unsigned* err = device_error_word();
    if (!err) return SCONE_EHIP;
    const int eff = max_n < table->max_len ? max_n : table->max_len;
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (n_rows == 0) {
        // No row is valid: the ids are still produced, the output is zeroed.
        hipError_t e0 = hipSuccess;
        if (fgram_ids || match_len)
            e0 = launch_lookup(table, token_ids, B, T, eff, fgram_ids, match_len, err, st);
        if (e0 == hipSuccess) e0 = launch_zero_rows(out, B * T * row_bytes, err, st);
        return status_of(e0);
    }
    const uintptr_t align = (uintptr_t)rows | (uintptr_t)out | (uintptr_t)row_bytes;
    hipError_t e;
    if ((align & 15) == 0 && ((row_bytes / 16) & (row_bytes / 16 - 1)) == 0) {
        const int64_t upr = row_bytes / 16;
        int shift = 0;
        while (((int64_t)1 << shift) < upr) ++shift;
        e = dispatch_slots<u32x4, true>(table, token_ids, B, T, eff, rows, n_rows, upr, shift,
                                        out, fgram_ids, match_len, err, st);
    } else {
        e = dispatch_slots<uint8_t, false>(table, token_ids, B, T, eff, rows, n_rows, row_bytes,
                                           0, out, fgram_ids, match_len, err, st);
    }
    return status_of(e);
}
