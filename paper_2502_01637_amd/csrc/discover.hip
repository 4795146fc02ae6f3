// F-gram discovery on the device: Algorithm 3 with the K-1 linear scans of
// Section 3.1.
//
// Scan n counts the n-grams of every sequence in an open-addressing table
// keyed by an exact 64-bit code.  For n = 2 the code is (t0 << 16) | t1.
// From n = 3 on, an n-gram is counted only when both its (n-1)-prefix and its
// (n-1)-suffix survived scan n-1 (count >= the minimum count): an n-gram that
// reaches the minimum appears inside both of them at least as often, so
// nothing that could survive is skipped.  Every survivor of scan n-1 has a
// dense id, and an n-gram is coded as (dense id of its prefix << 16) | last
// token, which is exact and fits 64 bits at any length, so the counting
// tables need only a 64-bit compare-and-swap.  After each scan the survivors
// get dense ids and every position learns the id of the survivor ending there
// (or -1), which is all the next scan reads.
//
// The candidates are all 2-grams and the survivors of scans 3..K; the top S by
// count are found with a threshold search (equal counts at the threshold are
// taken in an unspecified order, as Algorithm 3 allows) and their tokens are
// rebuilt by walking the prefix ids back to scan 2.
#include <vector>

#include "scone_internal.h"

namespace scone {
namespace {

constexpr int kThreads = 256;
constexpr uint64_t kEmptyKey = ~0ull;

struct alignas(16) CountSlot {
    uint64_t key;
    uint32_t count;
    int32_t dense;
};

__device__ __forceinline__ uint64_t count_hash(uint64_t key) {
    return fmix64(key ^ 0x9E3779B97F4A7C15ULL);
}

// Candidate and survivor slots are claimed in chunks: a wavefront owns
// kChunk consecutive entries, counts them in a first pass, reserves its whole
// range with one atomic per counter, and fills it in a second pass.  (One
// atomic per wavefront on a shared counter still serialises half a million
// times per scan at these sizes.)
constexpr int kChunk = 4096;

__global__ __launch_bounds__(kThreads) void k_table_clear(CountSlot* __restrict__ t,
                                                          uint64_t cap, int64_t block0) {
    const uint64_t i = (uint64_t)block_index(block0) * kThreads + threadIdx.x;
    if (i < cap) {
        t[i].key = kEmptyKey;
        t[i].count = 0;
        t[i].dense = -1;
    }
}

// Code of the n-gram ending at flat position i (row position tt), or kEmptyKey
// when it is not a candidate of scan n.
__device__ __forceinline__ uint64_t ngram_code(const int32_t* __restrict__ X,
                                               const int32_t* __restrict__ ids_prev, int64_t i,
                                               int64_t tt, int n) {
    if (tt < n - 1) return kEmptyKey;
    const uint32_t tok = (uint32_t)X[i];
    if (n == 2) return ((uint64_t)(uint32_t)X[i - 1] << 16) | tok;
    const int32_t p = ids_prev[i - 1];  // (n-1)-gram ending one earlier: the prefix
    const int32_t s = ids_prev[i];      // (n-1)-gram ending here: the suffix
    if (p < 0 || s < 0) return kEmptyKey;
    return ((uint64_t)p << 16) | tok;
}

// Add c to key's count in the global table; false if the table is full.
__device__ __forceinline__ bool global_add(CountSlot* __restrict__ t, uint64_t mask,
                                           uint64_t key, uint32_t c) {
    uint64_t s = count_hash(key) & mask;
    for (uint64_t step = 0; step <= mask; ++step) {
        const unsigned long long old = atomicCAS(reinterpret_cast<unsigned long long*>(&t[s].key),
                                                 (unsigned long long)kEmptyKey,
                                                 (unsigned long long)key);
        if (old == kEmptyKey || old == key) {
            atomicAdd(&t[s].count, c);
            return true;
        }
        s = (s + 1) & mask;
    }
    return false;
}

// Counting is aggregated per workgroup first: a workgroup counts
// kCountPerBlock consecutive positions in an LDS table, then adds each
// distinct key to the global table once.  Frequent n-grams (a Zipf stream's
// top bigram is about 1% of all positions) would otherwise serialise hundreds
// of thousands of increments on one global slot.  Keys that find no LDS slot
// within kLdsProbe probes go straight to the global table.
constexpr int kCountPerBlock = 4096;
constexpr int kLdsSlots = 4096;
constexpr int kLdsProbe = 32;

__global__ __launch_bounds__(kThreads) void k_count(const int32_t* __restrict__ X, int64_t BT,
                                                    int64_t T, int n,
                                                    const int32_t* __restrict__ ids_prev,
                                                    CountSlot* __restrict__ t, uint64_t mask,
                                                    unsigned* __restrict__ status) {
    __shared__ unsigned long long s_key[kLdsSlots];
    __shared__ unsigned s_cnt[kLdsSlots];
    for (int j = threadIdx.x; j < kLdsSlots; j += kThreads) {
        s_key[j] = (unsigned long long)kEmptyKey;
        s_cnt[j] = 0;
    }
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kCountPerBlock;
    bool full = false, bad_token = false;
    for (int r = 0; r < kCountPerBlock / kThreads; ++r) {
        const int64_t i = base + r * kThreads + threadIdx.x;
        if (i >= BT) break;
        if (n == 2) {
            const int32_t tok = X[i];
            if (tok < 0 || tok >= SCONE_TOKEN_LIMIT) {
                bad_token = true;
                continue;
            }
        }
        const uint64_t key = ngram_code(X, ids_prev, i, i % T, n);
        if (key == kEmptyKey) continue;
        if (n == 2 && (X[i - 1] < 0 || X[i - 1] >= SCONE_TOKEN_LIMIT)) continue;  // reported there
        uint32_t h = (uint32_t)count_hash(key) & (kLdsSlots - 1);
        bool done = false;
        for (int q = 0; q < kLdsProbe; ++q) {
            const unsigned long long old =
                atomicCAS(&s_key[h], (unsigned long long)kEmptyKey, (unsigned long long)key);
            if (old == kEmptyKey || old == key) {
                atomicAdd(&s_cnt[h], 1u);
                done = true;
                break;
            }
            h = (h + 1) & (kLdsSlots - 1);
        }
        if (!done && !global_add(t, mask, key, 1u)) full = true;
    }
    __syncthreads();
    for (int j = threadIdx.x; j < kLdsSlots; j += kThreads) {
        const unsigned long long key = s_key[j];
        if (key != kEmptyKey && !global_add(t, mask, key, s_cnt[j])) full = true;
    }
    if (bad_token) atomicOr(status, err_bit(SCONE_ETOKEN));
    if (full) atomicOr(status, err_bit(SCONE_EFULL));
}

// Dense ids for the survivors (count >= min_count) and, for scan 2, every
// entry as a candidate; for later scans the survivors are the candidates.
__global__ __launch_bounds__(kThreads) void k_survivors(
    CountSlot* __restrict__ t, uint64_t cap, uint32_t min_count, int level, int keep_all,
    unsigned* __restrict__ n_surv, uint64_t* __restrict__ skey, unsigned* __restrict__ n_cand,
    uint64_t* __restrict__ cand_key, uint32_t* __restrict__ cand_count,
    int8_t* __restrict__ cand_level, unsigned* __restrict__ max_count) {
    const uint64_t s0 = ((uint64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6)) * kChunk;
    if (s0 >= cap) return;  // wave-uniform
    const uint64_t s1 = s0 + kChunk < cap ? s0 + kChunk : cap;
    const int lane = threadIdx.x & 63;
    const unsigned long long below = (1ull << lane) - 1ull;
    unsigned ns = 0, nc = 0;
    uint32_t mx = 0;
    for (uint64_t b = s0; b < s1; b += 64) {
        const uint64_t s = b + lane;
        const uint64_t key = s < s1 ? t[s].key : kEmptyKey;
        const bool occupied = key != kEmptyKey;
        const uint32_t c = occupied ? t[s].count : 0;
        const bool survive = occupied && c >= min_count;
        const bool cand = occupied && (survive || keep_all);
        ns += (unsigned)__popcll(__ballot(survive));
        nc += (unsigned)__popcll(__ballot(cand));
        if (cand) mx = c > mx ? c : mx;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const uint32_t y = (uint32_t)__shfl_xor((int)mx, o);
        mx = y > mx ? y : mx;
    }
    unsigned bs = 0, bc = 0;
    if (lane == 0) {
        if (ns) bs = atomicAdd(n_surv, ns);
        if (nc) bc = atomicAdd(n_cand, nc);
        if (mx) atomicMax(max_count, mx);
    }
    bs = (unsigned)__shfl((int)bs, 0);
    bc = (unsigned)__shfl((int)bc, 0);
    for (uint64_t b = s0; b < s1; b += 64) {
        const uint64_t s = b + lane;
        const uint64_t key = s < s1 ? t[s].key : kEmptyKey;
        const bool occupied = key != kEmptyKey;
        const uint32_t c = occupied ? t[s].count : 0;
        const bool survive = occupied && c >= min_count;
        const bool cand = occupied && (survive || keep_all);
        const unsigned long long ms = __ballot(survive), mc = __ballot(cand);
        if (survive) {
            const unsigned id = bs + (unsigned)__popcll(ms & below);
            t[s].dense = (int32_t)id;
            if (skey) skey[id] = key;
        }
        if (cand) {
            const unsigned k = bc + (unsigned)__popcll(mc & below);
            cand_key[k] = key;
            cand_count[k] = c;
            cand_level[k] = (int8_t)level;
        }
        bs += (unsigned)__popcll(ms);
        bc += (unsigned)__popcll(mc);
    }
}

// Dense id of the survivor of scan n ending at every position, or -1.
__global__ __launch_bounds__(kThreads) void k_ids(const int32_t* __restrict__ X, int64_t BT,
                                                  int64_t T, int n,
                                                  const int32_t* __restrict__ ids_prev,
                                                  const CountSlot* __restrict__ t, uint64_t mask,
                                                  int32_t* __restrict__ ids_cur,
                                                  int64_t block0) {
    const int64_t i = block_index(block0) * kThreads + threadIdx.x;
    if (i >= BT) return;
    const uint64_t key = ngram_code(X, ids_prev, i, i % T, n);
    int32_t d = -1;
    if (key != kEmptyKey) {
        uint64_t s = count_hash(key) & mask;
        for (uint64_t step = 0; step <= mask; ++step) {
            const uint64_t k = t[s].key;
            if (k == key) {
                d = t[s].dense;
                break;
            }
            if (k == kEmptyKey) break;
            s = (s + 1) & mask;
        }
    }
    ids_cur[i] = d;
}

__global__ __launch_bounds__(kThreads) void k_count_at_least(const uint32_t* __restrict__ cnt,
                                                             int64_t n, uint32_t c,
                                                             unsigned long long* __restrict__ out,
                                                             int64_t block0) {
    const int64_t i = block_index(block0) * kThreads + threadIdx.x;
    const bool hit = i < n && cnt[i] >= c;
    const unsigned long long m = __ballot(hit);
    if ((threadIdx.x & 63) == 0 && m) atomicAdd(out, (unsigned long long)__popcll(m));
}

// Histogram of candidate counts, exact below kHistBins - 1 and pooled above:
// a workgroup counts a run of candidates in LDS and adds its non-zero bins.
constexpr int kHistBins = 4096;

__global__ __launch_bounds__(kThreads) void k_count_hist(const uint32_t* __restrict__ cnt,
                                                         int64_t n, int64_t per_block,
                                                         unsigned long long* __restrict__ hist) {
    __shared__ unsigned h[kHistBins];
    for (int i = threadIdx.x; i < kHistBins; i += kThreads) h[i] = 0;
    __syncthreads();
    const int64_t i0 = (int64_t)blockIdx.x * per_block;
    const int64_t i1 = i0 + per_block < n ? i0 + per_block : n;
    for (int64_t i = i0 + threadIdx.x; i < i1; i += kThreads) {
        const uint32_t c = cnt[i];
        atomicAdd(&h[c < kHistBins - 1 ? c : kHistBins - 1], 1u);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < kHistBins; i += kThreads)
        if (h[i]) atomicAdd(hist + i, (unsigned long long)h[i]);
}

struct LevelKeys {
    const uint64_t* skey[SCONE_MAX_FGRAM_LEN + 1];  // survivors' codes by scan
};

// Emit the selected candidates with their tokens.
__global__ __launch_bounds__(kThreads) void k_select(
    const uint64_t* __restrict__ cand_key, const uint32_t* __restrict__ cand_count,
    const int8_t* __restrict__ cand_level, int64_t n_cand, uint32_t thresh, int64_t n_above,
    int64_t S, LevelKeys lk, int max_len, unsigned* __restrict__ n_gt,
    unsigned* __restrict__ n_eq, int32_t* __restrict__ fgrams, int32_t* __restrict__ lengths,
    int32_t* __restrict__ counts) {
    const int64_t i0 = ((int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6)) * kChunk;
    if (i0 >= n_cand) return;  // wave-uniform
    const int64_t i1 = i0 + kChunk < n_cand ? i0 + kChunk : n_cand;
    const int lane = threadIdx.x & 63;
    const unsigned long long below = (1ull << lane) - 1ull;
    unsigned ng = 0, ne = 0;
    for (int64_t b = i0; b < i1; b += 64) {
        const int64_t i = b + lane;
        const uint32_t c = i < i1 ? cand_count[i] : 0;
        ng += (unsigned)__popcll(__ballot(i < i1 && c > thresh));
        ne += (unsigned)__popcll(__ballot(i < i1 && c == thresh));
    }
    unsigned bg = 0, be = 0;
    if (lane == 0) {
        if (ng) bg = atomicAdd(n_gt, ng);
        if (ne) be = atomicAdd(n_eq, ne);
    }
    bg = (unsigned)__shfl((int)bg, 0);
    be = (unsigned)__shfl((int)be, 0);
    for (int64_t b = i0; b < i1; b += 64) {
        const int64_t i = b + lane;
        const bool valid = i < i1;
        const uint32_t c = valid ? cand_count[i] : 0;
        const bool gt = valid && c > thresh, eq = valid && c == thresh;
        const unsigned long long mg = __ballot(gt), me = __ballot(eq);
        int64_t pos = -1;
        if (gt) {
            pos = bg + (unsigned)__popcll(mg & below);
        } else if (eq) {
            const int64_t e = be + (unsigned)__popcll(me & below);
            if (n_above + e < S) pos = n_above + e;
        }
        bg += (unsigned)__popcll(mg);
        be += (unsigned)__popcll(me);
        if (pos < 0 || pos >= S) continue;
        const int level = cand_level[i];
        int32_t tok[SCONE_MAX_FGRAM_LEN];
        uint64_t key = cand_key[i];
        for (int L = level; L >= 3; --L) {
            tok[L - 1] = (int32_t)(key & 0xFFFF);
            key = lk.skey[L - 1][key >> 16];
        }
        tok[1] = (int32_t)(key & 0xFFFF);
        tok[0] = (int32_t)(key >> 16);
        int32_t* row = fgrams + pos * (int64_t)max_len;
        for (int j = 0; j < max_len; ++j) row[j] = j < level ? tok[j] : -1;
        lengths[pos] = level;
        counts[pos] = (int32_t)c;
    }
}

}  // namespace
}  // namespace scone

namespace scone {
namespace {

// Scratch of one call, carved from one workspace: the counting table, the
// dense ids of two consecutive scans, the candidates, the counters and
// histogram, and the survivors' codes of every scan but the last.
struct DiscLayout {
    uint64_t cap;
    int64_t cand_cap;
    size_t table, ids_a, ids_b, cand_key, cand_count, cand_level, ctr, acc, hist;
    size_t skey[SCONE_MAX_FGRAM_LEN + 1];
    size_t total;
};

DiscLayout disc_layout(int64_t BT, int max_len) {
    DiscLayout l{};
    l.cap = 64;
    while ((int64_t)l.cap < 2 * BT) l.cap <<= 1;
    l.cand_cap = BT * (int64_t)(max_len - 1);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off = (off + bytes + 255) & ~(size_t)255;
        return at;
    };
    l.table = take(l.cap * sizeof(CountSlot));
    l.ids_a = take(BT * sizeof(int32_t));
    l.ids_b = take(BT * sizeof(int32_t));
    l.cand_key = take(l.cand_cap * sizeof(uint64_t));
    l.cand_count = take(l.cand_cap * sizeof(uint32_t));
    l.cand_level = take(l.cand_cap);
    l.ctr = take(16 * sizeof(unsigned));
    l.acc = take(sizeof(unsigned long long));
    l.hist = take(kHistBins * sizeof(unsigned long long));
    for (int L = 2; L < max_len; ++L) l.skey[L] = take(BT * sizeof(uint64_t));
    l.total = off;
    return l;
}

// SCONE_OK when (B, T, max_len) are sizes the call handles.
int disc_sizes_ok(int64_t B, int64_t T, int32_t max_len) {
    if (B < 0 || T < 0) return SCONE_EINVAL;
    if (max_len < 2 || max_len > SCONE_MAX_FGRAM_LEN) return SCONE_EINVAL;
    if (B > 0 && T > ((int64_t)1 << 40) / B) return SCONE_EINVAL;
    const int64_t BT = B * T;
    if (BT >= ((int64_t)1 << 31)) return SCONE_EINVAL;  // dense ids and counters are 32-bit
    // every candidate of every scan is counted in one 32-bit counter
    if (BT * (int64_t)(max_len - 1) >= ((int64_t)1 << 32)) return SCONE_EINVAL;
    return SCONE_OK;
}

}  // namespace
}  // namespace scone

extern "C" int64_t scone_discover_workspace(int64_t B, int64_t T, int32_t max_len) {
    using namespace scone;
    if (disc_sizes_ok(B, T, max_len) != SCONE_OK) return -1;
    return (int64_t)disc_layout(B * T, max_len).total;
}

extern "C" int scone_discover_fgrams(const int32_t* token_ids, int64_t B, int64_t T,
                                     int32_t max_len, int32_t min_count, int64_t S,
                                     int32_t* fgrams, int32_t* lengths, int32_t* counts,
                                     int64_t* n_found, void* workspace, int64_t workspace_bytes,
                                     void* stream) {
    using namespace scone;
    if (!n_found) return SCONE_EINVAL;
    *n_found = 0;
    if (S < 0 || min_count < 1) return SCONE_EINVAL;
    if (disc_sizes_ok(B, T, max_len) != SCONE_OK) return SCONE_EINVAL;
    const int64_t BT = B * T;
    if (BT == 0 || S == 0) return SCONE_OK;
    if (!token_ids || !fgrams || !lengths || !counts) return SCONE_EINVAL;
    const DiscLayout lay = disc_layout(BT, max_len);
    if (workspace && (workspace_bytes < 0 || (uint64_t)workspace_bytes < lay.total))
        return SCONE_EINVAL;
    if ((uintptr_t)workspace % 256 != 0) return SCONE_EINVAL;
    // The selection writes the outputs while it reads candidates from the
    // workspace, and the scans read the corpus while they write the
    // workspace: no two of these buffers may share memory.
    {
        const void* buf[5] = {token_ids, fgrams, lengths, counts, workspace};
        const int64_t len[5] = {span_bytes(BT, 4), span_bytes(S, 4 * (int64_t)max_len),
                                span_bytes(S, 4), span_bytes(S, 4),
                                workspace ? (int64_t)lay.total : 0};
        for (int i = 0; i < 5; ++i)
            for (int j = i + 1; j < 5; ++j)
                if (overlaps(buf[i], len[i], buf[j], len[j])) return SCONE_EINVAL;
    }
    hipStream_t st = static_cast<hipStream_t>(stream);

    const uint64_t cap = lay.cap;
    const uint64_t mask = cap - 1;

    // Without a workspace the call takes its scratch in one allocation and
    // frees it before returning (the call is synchronous).
    void* own = nullptr;
    if (!workspace) {
        if (hipMalloc(&own, lay.total) != hipSuccess) {
            (void)hipGetLastError();
            return SCONE_ENOMEM;
        }
        workspace = own;
    }
    auto release = [&]() {
        (void)hipStreamSynchronize(st);
        if (own) (void)hipFree(own);
    };
    uint8_t* ws = static_cast<uint8_t*>(workspace);
    CountSlot* table = reinterpret_cast<CountSlot*>(ws + lay.table);
    int32_t* ids_a = reinterpret_cast<int32_t*>(ws + lay.ids_a);
    int32_t* ids_b = reinterpret_cast<int32_t*>(ws + lay.ids_b);
    uint64_t* cand_key = reinterpret_cast<uint64_t*>(ws + lay.cand_key);
    uint32_t* cand_count = reinterpret_cast<uint32_t*>(ws + lay.cand_count);
    int8_t* cand_level = reinterpret_cast<int8_t*>(ws + lay.cand_level);
    unsigned* ctr = reinterpret_cast<unsigned*>(ws + lay.ctr);
    unsigned long long* acc = reinterpret_cast<unsigned long long*>(ws + lay.acc);
    unsigned long long* hist = reinterpret_cast<unsigned long long*>(ws + lay.hist);
    LevelKeys lk{};
    uint64_t* skeys[SCONE_MAX_FGRAM_LEN + 1] = {};
    for (int L = 2; L < max_len; ++L) {
        skeys[L] = reinterpret_cast<uint64_t*>(ws + lay.skey[L]);
        lk.skey[L] = skeys[L];
    }
    // ctr: [0] status, [1] survivors, [2] candidates, [3] max count, [4] n_gt, [5] n_eq
    int rc = SCONE_OK;
    // (The table clear covers up to 2^32 slots, more work-items than one
    // launch holds; the other grids stay far below that at BT < 2^31.)
    const int64_t g_cap = (int64_t)((cap + kThreads - 1) / kThreads);
    const int64_t g_bt = (BT + kThreads - 1) / kThreads;
    const dim3 block(kThreads);
    const int64_t waves_per_block = kThreads / 64;
    auto chunk_grid = [&](int64_t n) {
        const int64_t waves = (n + kChunk - 1) / kChunk;
        return (unsigned)((waves + waves_per_block - 1) / waves_per_block);
    };
    if (hipMemsetAsync(ctr, 0, 16 * sizeof(unsigned), st) != hipSuccess) rc = SCONE_EHIP;
    int32_t* ids_prev = ids_a;
    int32_t* ids_cur = ids_b;
    for (int n = 2; n <= max_len && rc == SCONE_OK; ++n) {
        if (launch_blocks(g_cap, kThreads, [&](int64_t b0, dim3 grid) {
                hipLaunchKernelGGL(k_table_clear, grid, block, 0, st, table, cap, b0);
            }) != hipSuccess)
            rc = SCONE_EHIP;
        hipLaunchKernelGGL(k_count, dim3((unsigned)((BT + kCountPerBlock - 1) / kCountPerBlock)),
                           dim3(kThreads), 0, st, token_ids, BT, T, n,
                           ids_prev, table, mask, ctr + 0);
        if (hipMemsetAsync(ctr + 1, 0, sizeof(unsigned), st) != hipSuccess) rc = SCONE_EHIP;
        hipLaunchKernelGGL(k_survivors, dim3(chunk_grid((int64_t)cap)), dim3(kThreads), 0, st,
                           table, cap,
                           (uint32_t)min_count, n, n == 2 ? 1 : 0, ctr + 1,
                           n < max_len ? skeys[n] : nullptr, ctr + 2, cand_key, cand_count,
                           cand_level, ctr + 3);
        if (n < max_len) {
            if (launch_blocks(g_bt, kThreads, [&](int64_t b0, dim3 grid) {
                    hipLaunchKernelGGL(k_ids, grid, block, 0, st, token_ids, BT, T, n, ids_prev,
                                       table, mask, ids_cur, b0);
                }) != hipSuccess)
                rc = SCONE_EHIP;
            int32_t* tmp = ids_prev;
            ids_prev = ids_cur;
            ids_cur = tmp;
        }
        if (hipGetLastError() != hipSuccess) rc = SCONE_EHIP;
    }
    unsigned h[4] = {0, 0, 0, 0};
    if (rc == SCONE_OK &&
        (hipMemcpyAsync(h, ctr, sizeof(h), hipMemcpyDeviceToHost, st) != hipSuccess ||
         hipStreamSynchronize(st) != hipSuccess))
        rc = SCONE_EHIP;
    if (rc == SCONE_OK && h[0]) rc = (h[0] & err_bit(SCONE_ETOKEN)) ? SCONE_ETOKEN : SCONE_EFULL;
    const int64_t n_cand = h[2];
    const uint32_t max_c = h[3];
    // Threshold: the largest count c with at least S candidates counting >= c.
    auto at_least = [&](uint32_t c, int64_t& out) -> bool {
        unsigned long long v = 0;
        if (hipMemsetAsync(acc, 0, sizeof(v), st) != hipSuccess) return false;
        if (launch_blocks((n_cand + kThreads - 1) / kThreads, kThreads,
                          [&](int64_t b0, dim3 grid) {
                              hipLaunchKernelGGL(k_count_at_least, grid, dim3(kThreads), 0, st,
                                                 cand_count, n_cand, c, acc, b0);
                          }) != hipSuccess ||
            hipMemcpyAsync(&v, acc, sizeof(v), hipMemcpyDeviceToHost, st) != hipSuccess ||
            hipStreamSynchronize(st) != hipSuccess)
            return false;
        out = (int64_t)v;
        return true;
    };
    uint32_t thresh = 0;   // every candidate counts >= 1 > 0
    int64_t n_above = 0;   // candidates counting > thresh
    if (rc == SCONE_OK && n_cand > S) {
        // One pass: a histogram of the counts, exact below kHistBins - 1.
        std::vector<unsigned long long> hh(kHistBins, 0);
        const int64_t per_block = 65536;
        if (hipMemsetAsync(hist, 0, kHistBins * sizeof(unsigned long long), st) != hipSuccess)
            rc = SCONE_EHIP;
        if (rc == SCONE_OK) {
            hipLaunchKernelGGL(k_count_hist, dim3((unsigned)((n_cand + per_block - 1) / per_block)),
                               dim3(kThreads), 0, st, cand_count, n_cand, per_block, hist);
            if (hipGetLastError() != hipSuccess ||
                hipMemcpyAsync(hh.data(), hist, kHistBins * sizeof(unsigned long long),
                               hipMemcpyDeviceToHost, st) != hipSuccess ||
                hipStreamSynchronize(st) != hipSuccess)
                rc = SCONE_EHIP;
        }
        if (rc == SCONE_OK && (int64_t)hh[kHistBins - 1] < S) {
            // the threshold is below the pooled bin: read it off the histogram
            int64_t ge = (int64_t)hh[kHistBins - 1];  // candidates counting >= c + 1
            for (uint32_t c = kHistBins - 2; c >= 1; --c) {
                const int64_t ge_c = ge + (int64_t)hh[c];
                if (ge_c >= S) {
                    thresh = c;
                    n_above = ge;
                    break;
                }
                ge = ge_c;
            }
        } else if (rc == SCONE_OK) {
            // at least S candidates count >= kHistBins - 1: search the rest
            uint32_t lo = kHistBins - 1, hi = max_c;  // at_least(lo) >= S
            while (lo < hi && rc == SCONE_OK) {
                const uint32_t mid = lo + (hi - lo + 1) / 2;
                int64_t k = 0;
                if (!at_least(mid, k)) rc = SCONE_EHIP;
                else if (k >= S) lo = mid;
                else hi = mid - 1;
            }
            thresh = lo;
            if (rc == SCONE_OK && thresh < max_c && !at_least(thresh + 1, n_above))
                rc = SCONE_EHIP;
        }
    }
    if (rc == SCONE_OK && n_cand > 0) {
        hipLaunchKernelGGL(k_select, dim3(chunk_grid(n_cand)), dim3(kThreads), 0, st, cand_key, cand_count, cand_level, n_cand, thresh,
                           n_above, S, lk, max_len, ctr + 4, ctr + 5, fgrams, lengths, counts);
        if (hipGetLastError() != hipSuccess) rc = SCONE_EHIP;
    }
    release();
    if (rc == SCONE_OK) *n_found = n_cand < S ? n_cand : S;
    return rc;
}
