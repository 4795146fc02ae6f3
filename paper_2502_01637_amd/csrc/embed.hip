// Fused lookup + gather: Algorithm 1's inference branch in one pass.
//
// Each workgroup first resolves the longest match for its tile of positions
// (the same tile lookup as scone_lookup, ids kept in LDS), then copies the
// tile's rows into the contiguous output block that those positions own.
// Fusing removes the id round trip through HBM and, more importantly, the
// separate latency-bound lookup launch: while some workgroups wait on hash
// probes, the others on the same compute unit keep HBM busy with row copies.
#include "tile_lookup.h"

namespace scone {
namespace {

template <int SB, int G, typename V, int U, bool kPow2>
__global__ __launch_bounds__(kTileThreads) void k_embed(
    const typename SlotOps<SB>::Slot* __restrict__ slots, uint64_t mask,
    const int32_t* __restrict__ X, int64_t T, int max_n, int64_t tiles_per_row,
    const V* __restrict__ rows, int64_t n_rows, int64_t upr, int shift, V* __restrict__ out,
    int32_t* __restrict__ ids_out, int8_t* __restrict__ len_out, unsigned* __restrict__ err) {
    constexpr int P = TileShape<G>::kPositions;
    __shared__ int32_t s_tok[P + kMaxHalo];
    __shared__ int32_t s_id[P];

    const int64_t b = blockIdx.x / tiles_per_row;
    const int64_t t0 = (blockIdx.x - b * tiles_per_row) * (int64_t)P;
    stage_tokens<G>(s_tok, X + b * T, T, t0, max_n - 1);
    __syncthreads();
    {
        int32_t id;
        int len;
        bool tok_ok;
        tile_lookup<SB, G>(slots, mask, s_tok, T, t0, max_n, id, len, tok_ok);
        const int p = threadIdx.x / G;
        const int64_t t = t0 + p;
        if (threadIdx.x % G == 0) {
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
    // output block of npos * upr units.
    const int64_t npos = (T - t0) < P ? (T - t0) : P;
    const int64_t total = npos * upr;
    V* __restrict__ dst = out + (b * T + t0) * upr;
    bool bad = false;
    for (int64_t base = threadIdx.x; base < total; base += (int64_t)kTileThreads * U) {
        V v[U];
        bool ok[U];
        if (base + (int64_t)(U - 1) * kTileThreads < total) {
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
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (!ok[u]) v[u] = V{};
                __builtin_nontemporal_store(v[u], dst + base + (int64_t)u * kTileThreads);
                bad |= !ok[u];
            }
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t i = base + (int64_t)u * kTileThreads;
                if (i < total) {
                    const int64_t r = kPow2 ? (i >> shift) : (i / upr);
                    const int64_t c = i - r * upr;
                    const int64_t id = s_id[r];
                    const bool okk = (id >= 0) & (id < n_rows);
                    const V val = okk ? rows[id * upr + c] : V{};
                    __builtin_nontemporal_store(val, dst + i);
                    bad |= !okk;
                }
            }
        }
    }
    if (bad) atomicOr(err, err_bit(SCONE_EROW));
}

template <int SB, int G, typename V, bool kPow2>
hipError_t launch(const scone_table* tb, const int32_t* X, int64_t B, int64_t T, int max_n,
                  const void* rows, int64_t n_rows, int64_t upr, int shift, void* out,
                  int32_t* ids, int8_t* lens, unsigned* err, hipStream_t st) {
    using Slot = typename SlotOps<SB>::Slot;
    constexpr int P = TileShape<G>::kPositions;
    const int64_t tiles = (T + P - 1) / P;
    const int64_t grid = B * tiles;
    if (grid > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((k_embed<SB, G, V, 4, kPow2>), dim3((unsigned)grid), dim3(kTileThreads),
                       0, st, static_cast<const Slot*>(tb->slots), (uint64_t)tb->capacity - 1, X,
                       T, max_n, tiles, static_cast<const V*>(rows), n_rows, upr, shift,
                       static_cast<V*>(out), ids, lens, err);
    return hipGetLastError();
}

template <int SB, typename V, bool kPow2>
hipError_t dispatch(const scone_table* tb, const int32_t* X, int64_t B, int64_t T, int max_n,
                    const void* rows, int64_t n_rows, int64_t upr, int shift, void* out,
                    int32_t* ids, int8_t* lens, unsigned* err, hipStream_t st) {
    switch (lanes_for(max_n)) {
        case 1:
            return launch<SB, 1, V, kPow2>(tb, X, B, T, max_n, rows, n_rows, upr, shift, out,
                                           ids, lens, err, st);
        case 2:
            return launch<SB, 2, V, kPow2>(tb, X, B, T, max_n, rows, n_rows, upr, shift, out,
                                           ids, lens, err, st);
        case 4:
            return launch<SB, 4, V, kPow2>(tb, X, B, T, max_n, rows, n_rows, upr, shift, out,
                                           ids, lens, err, st);
        default:
            return launch<SB, 8, V, kPow2>(tb, X, B, T, max_n, rows, n_rows, upr, shift, out,
                                           ids, lens, err, st);
    }
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
        if (e0 == hipErrorInvalidConfiguration) return SCONE_EINVAL;
        return e0 == hipSuccess ? SCONE_OK : SCONE_EHIP;
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
    if (e == hipErrorInvalidConfiguration) return SCONE_EINVAL;
    return e == hipSuccess ? SCONE_OK : SCONE_EHIP;
}
