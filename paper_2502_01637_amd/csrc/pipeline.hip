// Pipelined inference step: the lookup of batch k+1 and the row gather of
// batch k in one launch (Algorithm 1's inference branch, software-pipelined
// across batches).
//
// The lookup is latency-bound (dependent hash probes, a few KiB per tile) and
// the gather is HBM-bound (streaming rows).  Run back to back, the lookup
// launch leaves the memory system idle while its probes wait and the gather
// launch pays its ramp-up and tail on its own.  Here the first workgroups of
// the grid run tile lookups of the next batch and the rest copy rows of the
// current one, so the probes of the lookup workgroups overlap the row stream
// of the gather workgroups on every compute unit.  The ids of step k were
// written by step k-1, so the two halves share no data within a launch.
// Lookup workgroups come first in the grid: they are dispatched before the
// gather workgroups and their long probe chains start early.
#include "row_copy.h"
#include "tile_lookup.h"

namespace scone {
namespace {

template <int SB, int G, int U>
__global__ __launch_bounds__(kTileThreads) void k_pipelined(
    const typename SlotOps<SB>::Slot* __restrict__ slots, uint64_t mask,
    const int32_t* __restrict__ X, int64_t T, int max_n, int64_t tiles_per_row,
    int64_t n_lookup_blocks, int32_t* __restrict__ next_ids, int8_t* __restrict__ next_len,
    const int32_t* __restrict__ cur_ids, int64_t n_cur, const u32x4* __restrict__ rows,
    int64_t n_rows, u32x4* __restrict__ out, unsigned* __restrict__ err, int64_t block0) {
    __shared__ int32_t s_tok[TileShape<G>::kPositions + kMaxHalo];
    const int64_t blk = block_index(block0);
    if (blk < n_lookup_blocks) {  // workgroup-uniform
        lookup_block<SB, G>(slots, mask, X, T, max_n, tiles_per_row, blk, s_tok, next_ids,
                            next_len, err);
        return;
    }
    constexpr int W = pipelined_row_waves(U);
    const int64_t w = (blk - n_lookup_blocks) * (kTileThreads / 64) +
                      __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t r = w / W;
    if (r >= n_cur) return;  // wave-uniform
    copy_row_part<U, W>(cur_ids, r, (int)(w - r * W), rows, n_rows, out, err);
}

struct Step {
    const scone_table* tb;
    const int32_t* X;
    int64_t B, T;
    int max_n;
    int32_t* next_ids;
    int8_t* next_len;
    const int32_t* cur_ids;
    int64_t n_cur;
    const void* rows;
    int64_t n_rows;
    void* out;
    unsigned* err;
    hipStream_t st;
};

template <int SB, int G, int U>
hipError_t launch(const Step& s) {
    using Slot = typename SlotOps<SB>::Slot;
    constexpr int P = TileShape<G>::kPositions;
    const int64_t tiles = (s.T + P - 1) / P;
    const int64_t n_lookup = s.B * tiles;
    const int64_t n_waves = s.n_cur * pipelined_row_waves(U);
    const int64_t n_gather = (n_waves + kTileThreads / 64 - 1) / (kTileThreads / 64);
    return launch_blocks(n_lookup + n_gather, kTileThreads, [&](int64_t b0, dim3 grid) {
        hipLaunchKernelGGL((k_pipelined<SB, G, U>), grid, dim3(kTileThreads), 0, s.st,
                           static_cast<const Slot*>(s.tb->slots), (uint64_t)s.tb->capacity - 1,
                           s.X, s.T, s.max_n, tiles, n_lookup, s.next_ids, s.next_len,
                           s.cur_ids, s.n_cur, static_cast<const u32x4*>(s.rows), s.n_rows,
                           static_cast<u32x4*>(s.out), s.err, b0);
    });
}

template <int SB, int G>
hipError_t by_units(const Step& s, int units) {
    switch (units) {
        case 1: return launch<SB, G, 1>(s);
        case 2: return launch<SB, G, 2>(s);
        case 4: return launch<SB, G, 4>(s);
        default: return launch<SB, G, 8>(s);
    }
}

template <int SB>
hipError_t by_lanes(const Step& s, int units) {
    return tile_lanes_for(s.max_n) == 1 ? by_units<SB, 1>(s, units)
                                        : by_units<SB, 2>(s, units);
}

}  // namespace
}  // namespace scone

extern "C" int scone_embed_pipelined(const scone_table_t* table, const int32_t* next_tokens,
                                     int64_t B, int64_t T, int32_t max_n, int32_t* next_ids,
                                     int8_t* next_len, const int32_t* cur_ids, int64_t n_cur,
                                     const void* rows, int64_t n_rows, int64_t row_bytes,
                                     int32_t placement, void* out, void* stream) {
    using namespace scone;
    if (!table || B < 0 || T < 0 || max_n < 1 || n_cur < 0 || n_rows < 0 || row_bytes <= 0)
        return SCONE_EINVAL;
    if (placement != SCONE_PLACE_HBM && placement != SCONE_PLACE_HOST) return SCONE_EINVAL;
    if (B > 0 && T > ((int64_t)1 << 62) / B) return SCONE_EINVAL;
    if (n_cur > ((int64_t)1 << 62) / row_bytes) return SCONE_EINVAL;
    const int64_t n_next = B * T;
    if (n_next > 0 && (!next_tokens || !next_ids)) return SCONE_EINVAL;
    if (n_cur > 0 && (!cur_ids || !out || (!rows && n_rows > 0))) return SCONE_EINVAL;
    // One launch writes next_ids, next_len and out while other workgroups of it
    // read next_tokens (each tile with its halo) and cur_ids: no output may
    // share memory with an input or with another output.
    {
        const int64_t tok_b = span_bytes(n_next, 4), len_b = n_next > 0 ? n_next : 0;
        const int64_t cur_b = span_bytes(n_cur, 4), out_b = span_bytes(n_cur, row_bytes);
        const void* outs[3] = {next_ids, next_len, n_cur > 0 ? out : nullptr};
        const int64_t outs_b[3] = {tok_b, next_len ? len_b : 0, out_b};
        for (int i = 0; i < 3; ++i) {
            if (overlaps(outs[i], outs_b[i], next_tokens, tok_b) ||
                overlaps(outs[i], outs_b[i], cur_ids, cur_b))
                return SCONE_EINVAL;
            for (int j = i + 1; j < 3; ++j)
                if (overlaps(outs[i], outs_b[i], outs[j], outs_b[j])) return SCONE_EINVAL;
        }
    }
    int dev = 0;
    SCONE_HIP_TRY(hipGetDevice(&dev));
    if (dev != table->device) return SCONE_EINVAL;
    if (n_next == 0 && n_cur == 0) return SCONE_OK;
    unsigned* err = device_error_word();
    if (!err) return SCONE_EHIP;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int eff = max_n < table->max_len ? max_n : table->max_len;
    const int units = wave_row_units(row_bytes);
    const bool aligned = (((uintptr_t)rows | (uintptr_t)out) & 15) == 0;
    hipError_t e = hipSuccess;
    if (n_next > 0 && n_cur > 0 && units > 0 && aligned && n_rows > 0) {
        const Step s{table, next_tokens, B, T, eff, next_ids, next_len, cur_ids, n_cur,
                     rows, n_rows, out, err, st};
        e = table->slot_bytes == 16 ? by_lanes<16>(s, units) : by_lanes<32>(s, units);
    } else {
        // One half empty, or rows the one-wavefront copy does not cover: the
        // two kernels of scone_lookup and scone_gather, back to back.
        if (n_next > 0)
            e = launch_lookup(table, next_tokens, B, T, eff, next_ids, next_len, err, st);
        if (e == hipSuccess && n_cur > 0)
            e = launch_gather_any(cur_ids, n_cur, rows, n_rows, row_bytes, out, err, st);
    }
    return status_of(e);
}
