// Building the f-gram dictionary: an open-addressing hash table in HBM.
//
// The paper stores the f-gram layer as a dense row matrix plus a hash
// dictionary from f-grams to row indices (Section 2), built before serving
// (Section 3.2).  Here the dictionary is a power-of-two array of slots with
// linear probing from the start of the key's 64-byte bucket.  Insertion
// claims the first empty slot on the key's probe path with a 64-bit
// compare-and-swap on the slot's first key word, then
// writes the rest of the key and the id; it never compares keys, so slot
// placement under concurrency does not matter.  A second pass re-probes every
// input key: the first slot holding that key must be the one its own thread
// claimed, otherwise the key was inserted twice (a duplicate f-gram).
//
// A third pass adds the suffix entries that let lookups skip probes: for
// every f-gram of length 4 or more, the entry of its last three tokens gets
// kExtBit, and for every f-gram of length 6 or more, so does the entry of its
// last five; where that suffix is not itself an f-gram, a marker entry
// (id kMarkerId) is inserted for it.  Two threads may insert the same marker
// at once, leaving two identical copies; lookups read whichever comes first
// on the probe path, so that costs a slot and nothing else.  The slot count
// allows for one marker per such suffix.
#include <algorithm>
#include <cmath>

#include "scone_internal.h"

namespace scone {
namespace {

constexpr int kBuildThreads = 256;

template <typename Tok>
__device__ __forceinline__ bool tokens_in_range(const Tok* tok, int n) {
    bool ok = true;
    for (int i = 0; i < n; ++i) ok &= (tok[i] >= 0) & (tok[i] < SCONE_TOKEN_LIMIT);
    return ok;
}

template <int SB>
__global__ __launch_bounds__(kBuildThreads) void k_insert(
    const int32_t* __restrict__ fgrams, const int32_t* __restrict__ lengths,
    const int32_t* __restrict__ ids, int64_t n, int max_len,
    typename SlotOps<SB>::Slot* __restrict__ slots, uint64_t mask,
    int64_t* __restrict__ slot_of, unsigned* __restrict__ status, int64_t block0) {
    const int64_t k = block_index(block0) * kBuildThreads + threadIdx.x;
    if (k >= n) return;
    slot_of[k] = -1;
    const int len = lengths[k];
    const int32_t id = ids[k];
    if (len < 2 || len > max_len) {
        atomicOr(status, err_bit(SCONE_ELEN));
        return;
    }
    if (id < 0 || id == kMarkerId) {
        atomicOr(status, err_bit(SCONE_EID));
        return;
    }
    const int32_t* tok = fgrams + k * (int64_t)max_len;
    if (!tokens_in_range(tok, len)) {
        atomicOr(status, err_bit(SCONE_ETOKEN));
        return;
    }
    const Key key = pack_key(tok, len);
    uint64_t s = home_slot(key, mask, Bucket<SB>::kSlots);
    for (uint64_t step = 0; step <= mask; ++step) {
        unsigned long long* w0 = reinterpret_cast<unsigned long long*>(&slots[s].w0);
        if (atomicCAS(w0, 0ull, (unsigned long long)key.w0) == 0ull) {
            SlotOps<SB>::write_rest(slots, s, key, id);
            slot_of[k] = (int64_t)s;
            return;
        }
        s = (s + 1) & mask;
    }
    atomicOr(status, err_bit(SCONE_EFULL));
}

template <int SB>
__global__ __launch_bounds__(kBuildThreads) void k_verify(
    const int32_t* __restrict__ fgrams, const int32_t* __restrict__ lengths, int64_t n,
    int max_len, const typename SlotOps<SB>::Slot* __restrict__ slots, uint64_t mask,
    const int64_t* __restrict__ slot_of, unsigned* __restrict__ status, int64_t block0) {
    const int64_t k = block_index(block0) * kBuildThreads + threadIdx.x;
    if (k >= n) return;
    const int64_t mine = slot_of[k];
    if (mine < 0) return;  // rejected or not placed: already reported
    const Key key = pack_key(fgrams + k * (int64_t)max_len, lengths[k]);
    uint64_t s = home_slot(key, mask, Bucket<SB>::kSlots);
    for (uint64_t step = 0; step <= mask; ++step) {
        uint64_t w0, w1;
        int32_t id;
        SlotOps<SB>::read(slots, s, w0, w1, id);
        if (w0 == key.w0 && w1 == key.w1) {
            if ((int64_t)s != mine) atomicOr(status, err_bit(SCONE_EDUP));
            return;
        }
        if (w0 == 0) break;
        s = (s + 1) & mask;
    }
    // Its own slot lies on its probe path, so reaching here is a broken table.
    atomicOr(status, err_bit(SCONE_EFULL));
}

// Counts the f-grams of length 4..max_len and 6..max_len (the suffix
// entries the third pass may add).
__global__ __launch_bounds__(kBuildThreads) void k_count_long(
    const int32_t* __restrict__ lengths, int64_t n, int max_len,
    unsigned long long* __restrict__ counts, int64_t block0) {
    __shared__ unsigned s_c[2];
    if (threadIdx.x < 2) s_c[threadIdx.x] = 0;
    __syncthreads();
    const int64_t k = block_index(block0) * kBuildThreads + threadIdx.x;
    const int len = k < n ? lengths[k] : 0;
    const unsigned c4 = (unsigned)__popcll(__ballot(len >= 4 && len <= max_len));
    const unsigned c6 = (unsigned)__popcll(__ballot(len >= 6 && len <= max_len));
    if ((threadIdx.x & 63) == 0) {
        if (c4) atomicAdd(&s_c[0], c4);
        if (c6) atomicAdd(&s_c[1], c6);
    }
    __syncthreads();
    // one global add per workgroup and counter (same-address atomics serialise)
    if (threadIdx.x < 2 && s_c[threadIdx.x])
        atomicAdd(counts + threadIdx.x, (unsigned long long)s_c[threadIdx.x]);
}

// Counts the slots in use (f-grams and suffix markers, non-zero first key
// word) after a build: kUsedPer slots per thread, one global add per workgroup.
constexpr int kUsedPer = 16;

template <int SB>
__global__ __launch_bounds__(kBuildThreads) void k_count_used(
    const typename SlotOps<SB>::Slot* __restrict__ slots, int64_t cap,
    unsigned long long* __restrict__ used, int64_t block0) {
    __shared__ unsigned s_c;
    if (threadIdx.x == 0) s_c = 0;
    __syncthreads();
    const int64_t base = block_index(block0) * (kBuildThreads * kUsedPer) + threadIdx.x;
    unsigned c = 0;
#pragma unroll
    for (int i = 0; i < kUsedPer; ++i) {
        const int64_t k = base + (int64_t)i * kBuildThreads;
        if (k < cap && slots[k].w0 != 0) ++c;
    }
    for (int off = 32; off > 0; off >>= 1) c += __shfl_down(c, off);
    if ((threadIdx.x & 63) == 0 && c) atomicAdd(&s_c, c);
    __syncthreads();
    if (threadIdx.x == 0 && s_c) atomicAdd(used, (unsigned long long)s_c);
}

// Gives the entry of `key` kExtBit, inserting a marker when the key has no
// entry.  A marker slot is claimed in three steps: its first key word goes
// from 0 to kBusy (no key has length field 15), the rest of the key and the
// id are written, and only then is the first word set to the key with
// release order.  A thread that reads its key in the first word and then
// takes an acquire fence therefore also sees that key's second word, so it
// never takes a half-written slot for its own key; a slot still kBusy counts
// as another key (at worst a second, identical marker).
constexpr uint64_t kBusy = 0xF;

template <int SB>
__device__ __forceinline__ void mark_suffix(typename SlotOps<SB>::Slot* slots, uint64_t mask,
                                            const Key& key, unsigned* status) {
    uint64_t s = home_slot(key, mask, Bucket<SB>::kSlots);
    for (uint64_t step = 0; step <= mask; ++step) {
        unsigned long long* w0p = reinterpret_cast<unsigned long long*>(&slots[s].w0);
        uint64_t w0 = __hip_atomic_load(w0p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (w0 == 0) {
            w0 = atomicCAS(w0p, 0ull, (unsigned long long)kBusy);
            if (w0 == 0) {
                SlotOps<SB>::write_rest(slots, s, key, (int32_t)(kMarkerId | kExtBit));
                __hip_atomic_store(w0p, (unsigned long long)key.w0, __ATOMIC_RELEASE,
                                   __HIP_MEMORY_SCOPE_AGENT);
                return;
            }
            w0 = __hip_atomic_load(w0p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (w0 == key.w0) {
            // the release store that published this key word happened before:
            // an acquire fence makes the rest of the slot visible
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            uint64_t w1;
            if (SB == 16)
                w1 = __hip_atomic_load(reinterpret_cast<uint32_t*>(&slots[s]) + 2,
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            else
                w1 = __hip_atomic_load(reinterpret_cast<unsigned long long*>(&slots[s]) + 1,
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (w1 == key.w1) {
                // common suffixes end many f-grams: skip the atomic once the bit is set
                unsigned* idp = reinterpret_cast<unsigned*>(&slots[s].id);
                if (!(__hip_atomic_load(idp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) &
                      kExtBit))
                    atomicOr(idp, kExtBit);
                return;
            }
        }
        s = (s + 1) & mask;
    }
    atomicOr(status, err_bit(SCONE_EFULL));
}

template <int SB>
__global__ __launch_bounds__(kBuildThreads) void k_mark(
    const int32_t* __restrict__ fgrams, const int32_t* __restrict__ lengths, int64_t n,
    int max_len, typename SlotOps<SB>::Slot* __restrict__ slots, uint64_t mask,
    const int64_t* __restrict__ slot_of, unsigned* __restrict__ status, int64_t block0) {
    const int64_t k = block_index(block0) * kBuildThreads + threadIdx.x;
    if (k >= n || slot_of[k] < 0) return;  // rejected f-grams were reported
    const int len = lengths[k];
    const int32_t* tok = fgrams + k * (int64_t)max_len;
    if (len >= 4) mark_suffix<SB>(slots, mask, pack_key(tok + len - 3, 3), status);
    if (len >= 6) mark_suffix<SB>(slots, mask, pack_key(tok + len - 5, 5), status);
}

template <int SB>
hipError_t launch_build(const int32_t* fgrams, const int32_t* lengths, const int32_t* ids,
                        int64_t n, int max_len, void* slots, uint64_t mask, int64_t* slot_of,
                        unsigned* status, hipStream_t st) {
    using Slot = typename SlotOps<SB>::Slot;
    const int64_t blocks = (n + kBuildThreads - 1) / kBuildThreads;
    const hipError_t e = launch_blocks(blocks, kBuildThreads, [&](int64_t b0, dim3 grid) {
        hipLaunchKernelGGL(k_insert<SB>, grid, dim3(kBuildThreads), 0, st, fgrams, lengths, ids,
                           n, max_len, static_cast<Slot*>(slots), mask, slot_of, status, b0);
    });
    if (e != hipSuccess) return e;
    const hipError_t e2 = launch_blocks(blocks, kBuildThreads, [&](int64_t b0, dim3 grid) {
        hipLaunchKernelGGL(k_verify<SB>, grid, dim3(kBuildThreads), 0, st, fgrams, lengths, n,
                           max_len, static_cast<const Slot*>(slots), mask, slot_of, status, b0);
    });
    if (e2 != hipSuccess || max_len < 4) return e2;
    return launch_blocks(blocks, kBuildThreads, [&](int64_t b0, dim3 grid) {
        hipLaunchKernelGGL(k_mark<SB>, grid, dim3(kBuildThreads), 0, st, fgrams, lengths, n,
                           max_len, static_cast<Slot*>(slots), mask, slot_of, status, b0);
    });
}

}  // namespace
}  // namespace scone

extern "C" int scone_build_fgram_table(const int32_t* fgrams, const int32_t* lengths,
                                       const int32_t* ids, int64_t n, int32_t max_len,
                                       double max_load, void* stream, scone_table_t** out) {
    using namespace scone;
    if (!out) return SCONE_EINVAL;
    *out = nullptr;
    if (n < 0 || max_len < 2 || max_len > SCONE_MAX_FGRAM_LEN) return SCONE_EINVAL;
    if (!(max_load > 0.0 && max_load <= 0.9)) return SCONE_EINVAL;
    if (n > 0 && (!fgrams || !lengths || !ids)) return SCONE_EINVAL;
    // At most n entries plus one suffix entry per f-gram of length >= 4 and
    // one more per f-gram of length >= 6, so n * 3 bounds them.
    if (std::ceil(3.0 * (double)n / max_load) > (double)(1ull << 40)) return SCONE_EINVAL;
    const int slot_bytes = max_len <= kMaxLenSlot16 ? 16 : 32;

    hipStream_t st = static_cast<hipStream_t>(stream);
    int dev = 0;
    SCONE_HIP_TRY(hipGetDevice(&dev));

    void* slots = nullptr;
    // status word at offset 0, counts of f-grams of length >= 4 and >= 6 at 8,
    // 16, slots in use after the build at 24
    void* aux = nullptr;
    int64_t* slot_of = nullptr;
    int rc = SCONE_OK;
    unsigned long long haux[4] = {0, 0, 0, 0};
    unsigned hstatus = 0;
    unsigned long long hcount[2] = {0, 0};
    uint64_t cap = 64;
    unsigned* status = nullptr;
    if (hipMalloc(&aux, 32) != hipSuccess) {
        (void)hipGetLastError();
        return SCONE_ENOMEM;
    }
    status = static_cast<unsigned*>(aux);
    if (hipMemsetAsync(aux, 0, 32, st) != hipSuccess) {
        rc = SCONE_EHIP;
        goto fail;
    }
    if (n > 0 && max_len >= 4) {
        unsigned long long* counts =
            reinterpret_cast<unsigned long long*>(static_cast<uint8_t*>(aux) + 8);
        const hipError_t e = launch_blocks((n + kBuildThreads - 1) / kBuildThreads, kBuildThreads,
                                           [&](int64_t b0, dim3 grid) {
            hipLaunchKernelGGL(k_count_long, grid, dim3(kBuildThreads), 0, st, lengths, n,
                               (int)max_len, counts, b0);
        });
        if (e != hipSuccess ||
            hipMemcpyAsync(hcount, counts, sizeof(hcount), hipMemcpyDeviceToHost, st) !=
                hipSuccess ||
            hipStreamSynchronize(st) != hipSuccess) {
            rc = SCONE_EHIP;
            goto fail;
        }
    }
    {
        // Slot count: smallest power of two >= max(64, entries / max_load).
        const double entries = (double)n + (double)hcount[0] + (double)hcount[1];
        const double want = std::max(64.0, std::ceil(entries / max_load));
        while ((double)cap < want) cap <<= 1;
    }
    if (hipMalloc(&slots, cap * (uint64_t)slot_bytes) != hipSuccess ||
        (n > 0 && hipMalloc(&slot_of, sizeof(int64_t) * (size_t)n) != hipSuccess)) {
        (void)hipGetLastError();
        rc = SCONE_ENOMEM;
        goto fail;
    }
    if (hipMemsetAsync(slots, 0, cap * (uint64_t)slot_bytes, st) != hipSuccess) {
        rc = SCONE_EHIP;
        goto fail;
    }
    if (n > 0) {
        const hipError_t e =
            slot_bytes == 16
                ? launch_build<16>(fgrams, lengths, ids, n, max_len, slots, cap - 1, slot_of,
                                   status, st)
                : launch_build<32>(fgrams, lengths, ids, n, max_len, slots, cap - 1, slot_of,
                                   status, st);
        if (e != hipSuccess) {
            rc = SCONE_EHIP;
            goto fail;
        }
    }
    {
        unsigned long long* used =
            reinterpret_cast<unsigned long long*>(static_cast<uint8_t*>(aux) + 24);
        const int64_t per = (int64_t)kBuildThreads * kUsedPer;
        const hipError_t e = launch_blocks(((int64_t)cap + per - 1) / per, kBuildThreads,
                                           [&](int64_t b0, dim3 grid) {
            if (slot_bytes == 16)
                hipLaunchKernelGGL(k_count_used<16>, grid, dim3(kBuildThreads), 0, st,
                                   static_cast<const Slot16*>(slots), (int64_t)cap, used, b0);
            else
                hipLaunchKernelGGL(k_count_used<32>, grid, dim3(kBuildThreads), 0, st,
                                   static_cast<const Slot32*>(slots), (int64_t)cap, used, b0);
        });
        if (e != hipSuccess ||
            hipMemcpyAsync(haux, aux, sizeof(haux), hipMemcpyDeviceToHost, st) != hipSuccess ||
            hipStreamSynchronize(st) != hipSuccess) {
            rc = SCONE_EHIP;
            goto fail;
        }
        hstatus = (unsigned)(haux[0] & 0xffffffffu);
    }
    if (hstatus) {
        // Report argument-like data errors before structural ones.
        const int order[] = {SCONE_ELEN, SCONE_EID, SCONE_ETOKEN, SCONE_EDUP, SCONE_EFULL};
        rc = SCONE_EFULL;
        for (int c : order)
            if (hstatus & err_bit(c)) {
                rc = c;
                break;
            }
        goto fail;
    }
    (void)hipFree(aux);
    if (slot_of) (void)hipFree(slot_of);
    {
        scone_table* t = new (std::nothrow) scone_table();
        if (!t) {
            (void)hipFree(slots);
            return SCONE_ENOMEM;
        }
        t->device = dev;
        t->max_len = max_len;
        t->slot_bytes = slot_bytes;
        t->n = n;
        t->capacity = (int64_t)cap;
        t->entries = (int64_t)haux[3];
        t->slots = slots;
        *out = t;
    }
    return SCONE_OK;

fail:
    (void)hipStreamSynchronize(st);
    if (slots) (void)hipFree(slots);
    if (aux) (void)hipFree(aux);
    if (slot_of) (void)hipFree(slot_of);
    return rc;
}
