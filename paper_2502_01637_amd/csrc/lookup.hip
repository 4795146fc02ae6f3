// Longest-suffix f-gram lookup (Algorithm 1's choice of j, inference branch).
//
// A workgroup owns a tile of consecutive positions of one row.  It stages the
// tile's tokens plus a halo of (max_n - 1) earlier tokens of the same row in
// LDS, clipped at t = 0 so no window reaches into another row.  Each position
// gets two lanes, which probe lengths 3 and 2, then 5 and 4 where the
// length-3 suffix's entry says a longer f-gram ends with it, then 7 and 6
// where the length-5 suffix's entry says so (tile_lookup).  Every length that
// can match is probed on its own (the f-gram set need not hold the suffixes
// of its members: the build adds flagged entries for them).  The pair's
// first lane keeps the longer hit and writes the result.
#include "tile_lookup.h"

namespace scone {
namespace {

template <int SB, int G, bool kCount>
__global__ __launch_bounds__(kTileThreads) void k_lookup(
    const typename SlotOps<SB>::Slot* __restrict__ slots, uint64_t mask,
    const int32_t* __restrict__ X, int64_t T, int max_n, int64_t tiles_per_row,
    int32_t* __restrict__ ids_out, int8_t* __restrict__ len_out,
    unsigned long long* __restrict__ hist, unsigned* __restrict__ err, int64_t block0,
    unsigned long long* __restrict__ probes) {
    constexpr int P = TileShape<G>::kPositions;
    __shared__ int32_t s_tok[P + kMaxHalo];
    __shared__ unsigned s_hist[SCONE_MAX_FGRAM_LEN + 1];
    if (hist && threadIdx.x <= SCONE_MAX_FGRAM_LEN) s_hist[threadIdx.x] = 0;
    const int len = lookup_block<SB, G, kCount>(slots, mask, X, T, max_n, tiles_per_row,
                                                block_index(block0), s_tok, ids_out, len_out,
                                                err, probes);
    if (hist && len) atomicAdd(&s_hist[len], 1u);
    if (hist) {  // uniform: the whole workgroup takes this branch or none does
        __syncthreads();
        if (threadIdx.x <= SCONE_MAX_FGRAM_LEN && s_hist[threadIdx.x])
            atomicAdd(hist + threadIdx.x, (unsigned long long)s_hist[threadIdx.x]);
    }
}

template <int SB, int G, bool kCount>
hipError_t launch(const scone_table* tb, const int32_t* X, int64_t B, int64_t T, int max_n,
                  int32_t* ids, int8_t* lens, unsigned long long* hist, unsigned* err,
                  hipStream_t st, unsigned long long* probes) {
    using Slot = typename SlotOps<SB>::Slot;
    constexpr int P = TileShape<G>::kPositions;
    const int64_t tiles = (T + P - 1) / P;
    return launch_blocks(B * tiles, kTileThreads, [&](int64_t b0, dim3 grid) {
        hipLaunchKernelGGL((k_lookup<SB, G, kCount>), grid, dim3(kTileThreads), 0, st,
                           static_cast<const Slot*>(tb->slots), (uint64_t)tb->capacity - 1, X, T,
                           max_n, tiles, ids, lens, hist, err, b0, probes);
    });
}

template <int SB, bool kCount>
hipError_t dispatch_groups(const scone_table* tb, const int32_t* X, int64_t B, int64_t T,
                           int max_n, int32_t* ids, int8_t* lens, unsigned long long* hist,
                           unsigned* err, hipStream_t st, unsigned long long* probes) {
    return tile_lanes_for(max_n) == 1
               ? launch<SB, 1, kCount>(tb, X, B, T, max_n, ids, lens, hist, err, st, probes)
               : launch<SB, 2, kCount>(tb, X, B, T, max_n, ids, lens, hist, err, st, probes);
}

template <bool kCount>
hipError_t by_slot(const scone_table* tb, const int32_t* X, int64_t B, int64_t T, int max_n,
                   int32_t* ids, int8_t* lens, unsigned* err, hipStream_t st,
                   unsigned long long* hist, unsigned long long* probes) {
    return tb->slot_bytes == 16
               ? dispatch_groups<16, kCount>(tb, X, B, T, max_n, ids, lens, hist, err, st, probes)
               : dispatch_groups<32, kCount>(tb, X, B, T, max_n, ids, lens, hist, err, st, probes);
}

}  // namespace

hipError_t launch_lookup(const scone_table* tb, const int32_t* X, int64_t B, int64_t T,
                         int max_n, int32_t* ids, int8_t* lens, unsigned* err, hipStream_t st,
                         unsigned long long* hist) {
    return by_slot<false>(tb, X, B, T, max_n, ids, lens, err, st, hist, nullptr);
}

}  // namespace scone

extern "C" int scone_lookup(const scone_table_t* table, const int32_t* token_ids, int64_t B,
                            int64_t T, int32_t max_n, int32_t* fgram_ids, int8_t* match_len,
                            void* stream) {
    using namespace scone;
    if (!table || B < 0 || T < 0 || max_n < 1) return SCONE_EINVAL;
    if (B > 0 && T > ((int64_t)1 << 62) / B) return SCONE_EINVAL;
    if (B * T == 0) return SCONE_OK;
    if (!token_ids || !fgram_ids) return SCONE_EINVAL;
    // Workgroups read their tile's tokens plus a halo that other workgroups'
    // positions own, so the outputs must not alias the tokens.
    if (overlaps(fgram_ids, span_bytes(B * T, 4), token_ids, span_bytes(B * T, 4)) ||
        overlaps(match_len, B * T, token_ids, span_bytes(B * T, 4)) ||
        overlaps(match_len, B * T, fgram_ids, span_bytes(B * T, 4)))
        return SCONE_EINVAL;
    int dev = 0;
    SCONE_HIP_TRY(hipGetDevice(&dev));
    if (dev != table->device) return SCONE_EINVAL;
    unsigned* err = device_error_word();
    if (!err) return SCONE_EHIP;
    const int eff = max_n < table->max_len ? max_n : table->max_len;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const hipError_t e = launch_lookup(table, token_ids, B, T, eff, fgram_ids, match_len, err, st);
    return status_of(e);
}

// scone_lookup that also adds the number of keys it probed to *probes.
extern "C" int scone_lookup_counted(const scone_table_t* table, const int32_t* token_ids,
                                    int64_t B, int64_t T, int32_t max_n, int32_t* fgram_ids,
                                    int8_t* match_len, uint64_t* probes, void* stream) {
    using namespace scone;
    if (!probes) return SCONE_EINVAL;
    if (!table || B < 0 || T < 0 || max_n < 1) return SCONE_EINVAL;
    if (B > 0 && T > ((int64_t)1 << 62) / B) return SCONE_EINVAL;
    if (B * T == 0) return SCONE_OK;
    if (!token_ids || !fgram_ids) return SCONE_EINVAL;
    const int64_t tb = span_bytes(B * T, 4);
    if (overlaps(fgram_ids, tb, token_ids, tb) || overlaps(match_len, B * T, token_ids, tb) ||
        overlaps(match_len, B * T, fgram_ids, tb) || overlaps(probes, 8, token_ids, tb) ||
        overlaps(probes, 8, fgram_ids, tb) || overlaps(probes, 8, match_len, B * T))
        return SCONE_EINVAL;
    int dev = 0;
    SCONE_HIP_TRY(hipGetDevice(&dev));
    if (dev != table->device) return SCONE_EINVAL;
    unsigned* err = device_error_word();
    if (!err) return SCONE_EHIP;
    const int eff = max_n < table->max_len ? max_n : table->max_len;
    const hipError_t e =
        by_slot<true>(table, token_ids, B, T, eff, fgram_ids, match_len, err,
                      static_cast<hipStream_t>(stream), nullptr,
                      reinterpret_cast<unsigned long long*>(probes));
    return status_of(e);
}

// Pre-scan tagging: the lookup's match lengths and their histogram, without ids.
extern "C" int scone_tag(const scone_table_t* table, const int32_t* token_ids, int64_t B,
                         int64_t T, int32_t max_n, int8_t* match_len, uint64_t* hist,
                         void* stream) {
    using namespace scone;
    if (!table || B < 0 || T < 0 || max_n < 1) return SCONE_EINVAL;
    if (B > 0 && T > ((int64_t)1 << 62) / B) return SCONE_EINVAL;
    if (B * T == 0) return SCONE_OK;
    if (!token_ids || (!match_len && !hist)) return SCONE_EINVAL;
    if (overlaps(match_len, B * T, token_ids, span_bytes(B * T, 4)) ||
        overlaps(hist, 8 * (SCONE_MAX_FGRAM_LEN + 1), token_ids, span_bytes(B * T, 4)) ||
        overlaps(hist, 8 * (SCONE_MAX_FGRAM_LEN + 1), match_len, B * T))
        return SCONE_EINVAL;
    int dev = 0;
    SCONE_HIP_TRY(hipGetDevice(&dev));
    if (dev != table->device) return SCONE_EINVAL;
    unsigned* err = device_error_word();
    if (!err) return SCONE_EHIP;
    const int eff = max_n < table->max_len ? max_n : table->max_len;
    const hipError_t e = launch_lookup(table, token_ids, B, T, eff, nullptr, match_len, err,
                                       static_cast<hipStream_t>(stream),
                                       reinterpret_cast<unsigned long long*>(hist));
    return status_of(e);
}
