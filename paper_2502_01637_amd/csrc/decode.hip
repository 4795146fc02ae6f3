// One decoding step for many sequences: shift the new token into each
// sequence's rolling context, find the longest f-gram ending at it, and copy
// its row (Algorithm 1 applied to the newest position only; decoding emits one
// token per step, Section 4.3 and the resource summary in the appendix).
//
// One wavefront owns one sequence.  Lanes 0..G-1 probe the suffix lengths
// max_n .. 2 of (context + new token) in parallel and a ballot picks the
// longest hit; the wave then rewrites the context (the last ctx_cap tokens)
// and copies the chosen row with 16-byte vectors.  Because the context keeps
// the last max_n - 1 tokens, the step's result equals the prefill lookup at
// the same position of the whole sequence.
#include "tile_lookup.h"

namespace scone {
namespace {

constexpr int kDecodeThreads = 64;  // one wavefront, one sequence

template <int SB, int G, typename V, int U, bool kPow2>
__global__ __launch_bounds__(kDecodeThreads) void k_decode(
    const typename SlotOps<SB>::Slot* __restrict__ slots, uint64_t mask, int32_t* __restrict__ ctx,
    int32_t* __restrict__ ctx_len, int ctx_cap, const int32_t* __restrict__ new_tok, int max_n,
    const V* __restrict__ rows, int64_t n_rows, int64_t upr, int shift, V* __restrict__ out,
    int32_t* __restrict__ ids_out, int8_t* __restrict__ len_out, unsigned* __restrict__ err,
    int64_t block0) {
    const int64_t s = block_index(block0);
    const int lane = threadIdx.x;
    int32_t* my_ctx = ctx + s * ctx_cap;
    // The length, the new token and the whole context are loaded at once (the
    // context without waiting for its length); probe windows then come from
    // the lanes holding the context, so a step has three dependent memory
    // round trips: inputs, one hash bucket, the row.
    int L = ctx_len[s];
    const int32_t nt = new_tok[s];
    const int32_t cv_raw = lane < ctx_cap ? my_ctx[lane] : 0;
    L = L < 0 ? 0 : (L > ctx_cap ? ctx_cap : L);
    // seq[0..L] = context (oldest first) followed by the new token
    const int32_t cv = lane < L ? cv_raw : 0;

    bool hit = false;
    int32_t id = 0;
    const int n = max_n - lane;
    int32_t win[SCONE_MAX_FGRAM_LEN];
#pragma unroll
    for (int i = 0; i < SCONE_MAX_FGRAM_LEN; ++i) {
        const int k = L + 1 - n + i;  // position of window token i in seq
        const int32_t c = __shfl(cv, k & 63);
        win[i] = k < L ? c : nt;
    }
    if (lane < G && n >= 2 && n <= L + 1) {
        bool ok = true;
#pragma unroll
        for (int i = 0; i < SCONE_MAX_FGRAM_LEN; ++i)
            if (i < n) ok &= (win[i] >= 0) & (win[i] < SCONE_TOKEN_LIMIT);
        if (ok) hit = probe<SB>(slots, mask, pack_key(win, n), id);
    }
    const unsigned long long m = __ballot(hit);
    const unsigned gm = (unsigned)m & ((1u << G) - 1u);
    const int jb = gm ? __ffs(gm) - 1 : 0;
    const int32_t best = __shfl(id, jb);
    const int32_t rid = gm ? best : nt;

    // New context: the last min(ctx_cap, L + 1) tokens of seq.
    const int Lp = L + 1 < ctx_cap ? L + 1 : ctx_cap;
    const int d = L + 1 - Lp;
    const int32_t moved = __shfl(cv, (lane + d) & 63);
    if (lane < Lp) my_ctx[lane] = (lane + d < L) ? moved : nt;
    if (lane == 0) {
        ctx_len[s] = Lp;
        if (nt < 0 || nt >= SCONE_TOKEN_LIMIT) atomicOr(err, err_bit(SCONE_ETOKEN));
        if (ids_out) ids_out[s] = rid;
        if (len_out) len_out[s] = (int8_t)(gm ? max_n - jb : 1);
    }

    // Copy the row.
    const bool ok = (rid >= 0) & ((int64_t)rid < n_rows);
    if (!ok && lane == 0) atomicOr(err, err_bit(SCONE_EROW));
    V* __restrict__ dst = out + s * upr;
    const V* __restrict__ src = rows + (kPow2 ? ((int64_t)rid << shift) : (int64_t)rid * upr);
    for (int64_t c0 = lane; c0 < upr; c0 += (int64_t)kDecodeThreads * U) {
        V v[U];
        if (ok) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t c = c0 + (int64_t)u * kDecodeThreads;
                if (c < upr) v[u] = src[c];
            }
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) v[u] = V{};
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t c = c0 + (int64_t)u * kDecodeThreads;
            if (c < upr) __builtin_nontemporal_store(v[u], dst + c);
        }
    }
}

template <int SB, int G, typename V, bool kPow2>
hipError_t launch(const scone_table* tb, int32_t* ctx, int32_t* ctx_len, int ctx_cap,
                  const int32_t* new_tok, int64_t S, int max_n, const void* rows,
                  int64_t n_rows, int64_t upr, int shift, void* out, int32_t* ids, int8_t* lens,
                  unsigned* err, hipStream_t st) {
    using Slot = typename SlotOps<SB>::Slot;
    return launch_blocks(S, kDecodeThreads, [&](int64_t b0, dim3 grid) {
        hipLaunchKernelGGL((k_decode<SB, G, V, 4, kPow2>), grid, dim3(kDecodeThreads), 0, st,
                           static_cast<const Slot*>(tb->slots), (uint64_t)tb->capacity - 1, ctx,
                           ctx_len, ctx_cap, new_tok, max_n, static_cast<const V*>(rows), n_rows,
                           upr, shift, static_cast<V*>(out), ids, lens, err, b0);
    });
}

template <int SB, typename V, bool kPow2>
hipError_t dispatch(const scone_table* tb, int32_t* ctx, int32_t* ctx_len, int ctx_cap,
                    const int32_t* new_tok, int64_t S, int max_n, const void* rows,
                    int64_t n_rows, int64_t upr, int shift, void* out, int32_t* ids,
                    int8_t* lens, unsigned* err, hipStream_t st) {
    switch (lanes_for(max_n)) {
        case 1:
            return launch<SB, 1, V, kPow2>(tb, ctx, ctx_len, ctx_cap, new_tok, S, max_n, rows,
                                           n_rows, upr, shift, out, ids, lens, err, st);
        case 2:
            return launch<SB, 2, V, kPow2>(tb, ctx, ctx_len, ctx_cap, new_tok, S, max_n, rows,
                                           n_rows, upr, shift, out, ids, lens, err, st);
        case 4:
            return launch<SB, 4, V, kPow2>(tb, ctx, ctx_len, ctx_cap, new_tok, S, max_n, rows,
                                           n_rows, upr, shift, out, ids, lens, err, st);
        default:
            return launch<SB, 8, V, kPow2>(tb, ctx, ctx_len, ctx_cap, new_tok, S, max_n, rows,
                                           n_rows, upr, shift, out, ids, lens, err, st);
    }
}

template <typename V, bool kPow2>
hipError_t dispatch_slots(const scone_table* tb, int32_t* ctx, int32_t* ctx_len, int ctx_cap,
                          const int32_t* new_tok, int64_t S, int max_n, const void* rows,
                          int64_t n_rows, int64_t upr, int shift, void* out, int32_t* ids,
                          int8_t* lens, unsigned* err, hipStream_t st) {
    return tb->slot_bytes == 16
               ? dispatch<16, V, kPow2>(tb, ctx, ctx_len, ctx_cap, new_tok, S, max_n, rows,
                                        n_rows, upr, shift, out, ids, lens, err, st)
               : dispatch<32, V, kPow2>(tb, ctx, ctx_len, ctx_cap, new_tok, S, max_n, rows,
                                        n_rows, upr, shift, out, ids, lens, err, st);
}

}  // namespace
}  // namespace scone

extern "C" int scone_decode_step(const scone_table_t* table, int32_t* ctx, int32_t* ctx_len,
                                 int32_t ctx_cap, const int32_t* new_tok, int64_t S,
                                 int32_t max_n, const void* rows, int64_t n_rows,
                                 int64_t row_bytes, int32_t placement, void* out,
                                 int32_t* fgram_ids, int8_t* match_len, void* stream) {
    using namespace scone;
    if (!table || S < 0 || max_n < 1 || n_rows < 0 || row_bytes <= 0) return SCONE_EINVAL;
    if (placement != SCONE_PLACE_HBM && placement != SCONE_PLACE_HOST) return SCONE_EINVAL;
    const int eff = max_n < table->max_len ? max_n : table->max_len;
    if (ctx_cap < eff - 1 || ctx_cap > 63 || ctx_cap < 0) return SCONE_EINVAL;
    if (S > ((int64_t)1 << 62) / row_bytes) return SCONE_EINVAL;
    if (S == 0) return SCONE_OK;
    if (!ctx_len || !new_tok || !out || (!ctx && ctx_cap > 0) || (!rows && n_rows > 0))
        return SCONE_EINVAL;
    // Each wavefront rewrites its own sequence's context in place; the other
    // outputs must not alias any input or each other.
    {
        const void* outs[3] = {out, fgram_ids, match_len};
        const int64_t outs_b[3] = {S * row_bytes, span_bytes(S, 4), S};
        const void* ins[4] = {ctx, ctx_len, new_tok, rows};
        const int64_t ins_b[4] = {span_bytes(S, 4 * (int64_t)ctx_cap), span_bytes(S, 4),
                                  span_bytes(S, 4), span_bytes(n_rows, row_bytes)};
        for (int i = 0; i < 3; ++i) {
            for (int j = 0; j < 4; ++j)
                if (overlaps(outs[i], outs_b[i], ins[j], ins_b[j])) return SCONE_EINVAL;
            for (int j = i + 1; j < 3; ++j)
                if (overlaps(outs[i], outs_b[i], outs[j], outs_b[j])) return SCONE_EINVAL;
        }
        if (overlaps(ctx, ins_b[0], ctx_len, ins_b[1]) || overlaps(ctx, ins_b[0], new_tok, ins_b[2]) ||
            overlaps(ctx_len, ins_b[1], new_tok, ins_b[2]))
            return SCONE_EINVAL;
    }
    int dev = 0;
    SCONE_HIP_TRY(hipGetDevice(&dev));
    if (dev != table->device) return SCONE_EINVAL;
    unsigned* err = device_error_word();
    if (!err) return SCONE_EHIP;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const uintptr_t align = (uintptr_t)rows | (uintptr_t)out | (uintptr_t)row_bytes;
    hipError_t e;
    if ((align & 15) == 0 && ((row_bytes / 16) & (row_bytes / 16 - 1)) == 0) {
        const int64_t upr = row_bytes / 16;
        int shift = 0;
        while (((int64_t)1 << shift) < upr) ++shift;
        e = dispatch_slots<u32x4, true>(table, ctx, ctx_len, ctx_cap, new_tok, S, eff, rows,
                                        n_rows, upr, shift, out, fgram_ids, match_len, err, st);
    } else {
        e = dispatch_slots<uint8_t, false>(table, ctx, ctx_len, ctx_cap, new_tok, S, eff, rows,
                                           n_rows, row_bytes, 0, out, fgram_ids, match_len, err,
                                           st);
    }
    return status_of(e);
}
