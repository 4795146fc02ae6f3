// Tile-level longest-suffix lookup shared by the lookup, embed and decode kernels.
#pragma once

#include "scone_internal.h"

namespace scone {

constexpr int kTileThreads = 256;
constexpr int kMaxHalo = SCONE_MAX_FGRAM_LEN - 1;

template <int G>
struct TileShape {
    static constexpr int kPositions = kTileThreads / G;  // most positions a workgroup can probe
};

// Lanes per position when every length is probed at once (the decode
// kernel): a power of two >= max_n - 1.
__host__ __device__ constexpr int lanes_for(int max_n) {
    return max_n - 1 <= 1 ? 1 : max_n - 1 <= 2 ? 2 : max_n - 1 <= 4 ? 4 : 8;
}

// Lanes per position of tile_lookup: one for windows up to 2, else two.
__host__ __device__ constexpr int tile_lanes_for(int max_n) { return max_n <= 2 ? 1 : 2; }

// Stage X[b, t0 - halo .. t0 + P) of one row into LDS (zero outside [0, T));
// called by the whole workgroup, which then synchronises.
__device__ __forceinline__ void stage_tokens(int32_t* s_tok, const int32_t* __restrict__ row,
                                             int64_t T, int64_t t0, int P, int halo) {
    for (int i = threadIdx.x; i < P + halo; i += kTileThreads) {
        const int64_t t = t0 - halo + i;
        s_tok[i] = (t >= 0 && t < T) ? row[t] : 0;
    }
}

// After stage_tokens and a barrier: position p = threadIdx.x / G (p < P) of
// the tile gets its longest match, G = tile_lanes_for(max_n).  Lane j of the
// position's pair probes length 3 - j, then 5 - j, then 7 - j (with G = 1
// the single lane probes length 2).  A round runs only when the previous
// round's length-3 (length-5) suffix has an entry with kExtBit, i.e. some
// longer f-gram ends with it, so a position stops as soon as no longer
// f-gram can end there; the two lanes then compare their longest hits.  On
// a workload of 10M f-grams of length 2..5 this takes 2.75 probes per
// position instead of 4.  Two lanes per position, each probing once per
// round, keep every lane busy: measured against one lane per length (four
// for max_n = 5, pruned or not), it halved the tagging time and cut the
// standalone lookup by about a fifth.  Returns, on lane j = 0 of a valid
// position (p < P, t0 + p < T), the id (or the token itself) and the matched
// length (1 when nothing matched); `tok_ok` reports whether the position's
// own token is in range.  All lanes of the wave must call it.  With kCount,
// the wave also adds the number of keys it probed to *probes (a diagnostic
// instantiation; the lookup itself is the same).
template <int SB, int G, bool kCount = false>
__device__ __forceinline__ void tile_lookup(const typename SlotOps<SB>::Slot* __restrict__ slots,
                                            uint64_t mask, const int32_t* s_tok, int64_t T,
                                            int64_t t0, int P, int max_n, int32_t& id_out,
                                            int& len_out, bool& tok_ok,
                                            unsigned long long* probes = nullptr) {
    static_assert(G == 1 || G == 2, "one or two lanes per position");
    const int halo = max_n - 1;
    const int p = threadIdx.x / G;
    const int j = threadIdx.x % G;
    const int64_t t = t0 + p;
    const bool valid = p < P && t < T;
    const int base = (threadIdx.x & 63) & ~(G - 1);
    const int32_t tok = valid ? s_tok[p + halo] : 0;
    tok_ok = (tok >= 0) & (tok < SCONE_TOKEN_LIMIT);
    int best = 0;  // longest f-gram length this lane found
    int32_t best_id = 0;
    bool ext = false;  // the last probed key has an entry with kExtBit
    int n_probes = 0;  // keys this lane probed (kCount)
    auto step = [&](int n) {
        ext = false;
        if (!(valid && n >= 2 && n <= max_n && (int64_t)n <= t + 1)) return;
        const int32_t* win = s_tok + p + halo - n + 1;  // X[b, t-n+1 .. t]
        bool ok = true;
#pragma unroll
        for (int i = 0; i < SCONE_MAX_FGRAM_LEN; ++i)
            if (i < n) ok &= (win[i] >= 0) & (win[i] < SCONE_TOKEN_LIMIT);
        int32_t raw = 0;
        if constexpr (kCount) n_probes += ok ? 1 : 0;
        if (ok && probe_raw<SB>(slots, mask, pack_key(win, n), raw)) {
            if (entry_is_fgram(raw)) {
                best = n;
                best_id = raw & kIdMask;
            }
            ext = entry_extends(raw);
        }
    };
    step(G == 2 ? 3 - j : 2);
    if (max_n >= 4) {  // the same for every lane of the launch
        const bool go4 = __shfl((int)ext, base) != 0;  // lane j = 0 probed length 3
        if (go4) step(5 - j);
        else ext = false;
        if (max_n >= 6) {
            const bool go6 = __shfl((int)ext, base) != 0;  // and then length 5
            if (go6) step(7 - j);
        }
    }
    if (G == 2) {
        const int ob = __shfl_xor(best, 1);
        const int32_t oid = __shfl_xor(best_id, 1);
        if (ob > best) {
            best = ob;
            best_id = oid;
        }
    }
    id_out = best ? best_id : tok;
    len_out = best ? best : 1;
    if constexpr (kCount) {
#pragma unroll
        for (int w = 32; w >= 1; w >>= 1) n_probes += __shfl_xor(n_probes, w);
        if ((threadIdx.x & 63) == 0 && n_probes)
            atomicAdd(probes, (unsigned long long)n_probes);
    }
}

// One workgroup's share of a lookup over X [B, T]: tile `tile` of the row-major
// tile grid (tiles_per_row tiles of P positions per row).  Stages the tile's
// tokens in s_tok, finds each position's longest match and writes the id and
// length (either output may be null); a bad token raises SCONE_ETOKEN.
// Returns the matched length on the lane that wrote a position, else 0.
// Called by the whole workgroup (it synchronises once).
template <int SB, int G, bool kCount = false>
__device__ __forceinline__ int lookup_block(const typename SlotOps<SB>::Slot* __restrict__ slots,
                                            uint64_t mask, const int32_t* __restrict__ X,
                                            int64_t T, int max_n, int64_t tiles_per_row,
                                            int64_t tile, int32_t* s_tok,
                                            int32_t* __restrict__ ids_out,
                                            int8_t* __restrict__ len_out,
                                            unsigned* __restrict__ err,
                                            unsigned long long* probes = nullptr) {
    constexpr int P = TileShape<G>::kPositions;
    const int64_t b = tile / tiles_per_row;
    const int64_t t0 = (tile - b * tiles_per_row) * (int64_t)P;
    stage_tokens(s_tok, X + b * T, T, t0, P, max_n - 1);
    __syncthreads();
    int32_t id;
    int len;
    bool tok_ok;
    tile_lookup<SB, G, kCount>(slots, mask, s_tok, T, t0, P, max_n, id, len, tok_ok, probes);
    const int64_t t = t0 + threadIdx.x / G;
    if (threadIdx.x % G == 0 && t < T) {
        if (!tok_ok) atomicOr(err, err_bit(SCONE_ETOKEN));
        if (ids_out) ids_out[b * T + t] = id;
        if (len_out) len_out[b * T + t] = (int8_t)len;
        return len;
    }
    return 0;
}

}  // namespace scone
