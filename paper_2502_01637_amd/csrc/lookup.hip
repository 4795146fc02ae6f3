// Longest-suffix f-gram lookup (Algorithm 1's choice of j, inference branch).
//
// A workgroup owns a tile of consecutive positions of one row.  It stages the
// tile's tokens plus a halo of (max_n - 1) earlier tokens of the same row in
// LDS, clipped at t = 0 so no window reaches into another row.  Each position
// gets a group of G lanes (G a power of two >= max_n - 1); lane j of the group
// probes the suffix of length n = max_n - j, so all lengths are probed at once
// and independently (the f-gram set need not hold the suffixes of its
// members).  A wave-wide ballot of the hit flags then gives, per group, the
// lowest hitting lane, i.e. the longest matching f-gram, and a lane shuffle
// moves its id to the group's first lane, which writes the result.
#include "tile_lookup.h"

namespace scone {
namespace {

template <int SB, int G, bool kPrune>
__global__ __launch_bounds__(kTileThreads) void k_lookup(
    const typename SlotOps<SB>::Slot* __restrict__ slots, uint64_t mask,
    const int32_t* __restrict__ X, int64_t T, int max_n, int64_t tiles_per_row,
    int32_t* __restrict__ ids_out, int8_t* __restrict__ len_out,
    unsigned long long* __restrict__ hist, unsigned* __restrict__ err, int64_t block0) {
    constexpr int P = TileShape<G>::kPositions;
    __shared__ int32_t s_tok[P + kMaxHalo];
    __shared__ unsigned s_hist[SCONE_MAX_FGRAM_LEN + 1];
    if (hist && threadIdx.x <= SCONE_MAX_FGRAM_LEN) s_hist[threadIdx.x] = 0;
    const int len = lookup_block<SB, G, kPrune>(slots, mask, X, T, max_n, tiles_per_row,
                                        block_index(block0), s_tok, ids_out, len_out, err);
    if (hist && len) atomicAdd(&s_hist[len], 1u);
    if (hist) {  // uniform: the whole workgroup takes this branch or none does
        __syncthreads();
        if (threadIdx.x <= SCONE_MAX_FGRAM_LEN && s_hist[threadIdx.x])
            atomicAdd(hist + threadIdx.x, (unsigned long long)s_hist[threadIdx.x]);
    }
}

template <int SB, int G, bool kPrune>
hipError_t launch(const scone_table* tb, const int32_t* X, int64_t B, int64_t T, int max_n,
                  int32_t* ids, int8_t* lens, unsigned long long* hist, unsigned* err,
                  hipStream_t st) {
    using Slot = typename SlotOps<SB>::Slot;
    constexpr int P = TileShape<G>::kPositions;
    const int64_t tiles = (T + P - 1) / P;
    return launch_blocks(B * tiles, kTileThreads, [&](int64_t b0, dim3 grid) {
        hipLaunchKernelGGL((k_lookup<SB, G, kPrune>), grid, dim3(kTileThreads), 0, st,
                           static_cast<const Slot*>(tb->slots), (uint64_t)tb->capacity - 1, X, T,
                           max_n, tiles, ids, lens, hist, err, b0);
    });
}

template <int SB, bool kPrune>
hipError_t dispatch_groups(const scone_table* tb, const int32_t* X, int64_t B, int64_t T,
                           int max_n, int32_t* ids, int8_t* lens, unsigned long long* hist,
                           unsigned* err, hipStream_t st) {
    switch (lanes_for(max_n)) {
        case 1: return launch<SB, 1, false>(tb, X, B, T, max_n, ids, lens, hist, err, st);
        case 2: return launch<SB, 2, false>(tb, X, B, T, max_n, ids, lens, hist, err, st);
        case 4: return launch<SB, 4, kPrune>(tb, X, B, T, max_n, ids, lens, hist, err, st);
        default: return launch<SB, 8, kPrune>(tb, X, B, T, max_n, ids, lens, hist, err, st);
    }
}

}  // namespace

hipError_t launch_lookup(const scone_table* tb, const int32_t* X, int64_t B, int64_t T,
                         int max_n, int32_t* ids, int8_t* lens, unsigned* err, hipStream_t st,
                         unsigned long long* hist, bool prune) {
    if (prune)
        return tb->slot_bytes == 16
                   ? dispatch_groups<16, true>(tb, X, B, T, max_n, ids, lens, hist, err, st)
                   : dispatch_groups<32, true>(tb, X, B, T, max_n, ids, lens, hist, err, st);
    return tb->slot_bytes == 16
               ? dispatch_groups<16, false>(tb, X, B, T, max_n, ids, lens, hist, err, st)
               : dispatch_groups<32, false>(tb, X, B, T, max_n, ids, lens, hist, err, st);
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
    int dev = 0;
    SCONE_HIP_TRY(hipGetDevice(&dev));
    if (dev != table->device) return SCONE_EINVAL;
    unsigned* err = device_error_word();
    if (!err) return SCONE_EHIP;
    const int eff = max_n < table->max_len ? max_n : table->max_len;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const hipError_t e = launch_lookup(table, token_ids, B, T, eff, fgram_ids, match_len, err, st);
    if (e == hipErrorInvalidConfiguration) return SCONE_EINVAL;
    return e == hipSuccess ? SCONE_OK : SCONE_EHIP;
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
    int dev = 0;
    SCONE_HIP_TRY(hipGetDevice(&dev));
    if (dev != table->device) return SCONE_EINVAL;
    unsigned* err = device_error_word();
    if (!err) return SCONE_EHIP;
    const int eff = max_n < table->max_len ? max_n : table->max_len;
    // a corpus-sized pass: probe pruning trades latency for memory traffic
    const hipError_t e = launch_lookup(table, token_ids, B, T, eff, nullptr, match_len, err,
                                       static_cast<hipStream_t>(stream),
                                       reinterpret_cast<unsigned long long*>(hist), true);
    if (e == hipErrorInvalidConfiguration) return SCONE_EINVAL;
    return e == hipSuccess ? SCONE_OK : SCONE_EHIP;
}
