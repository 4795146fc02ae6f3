// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "scone.h"

namespace scone {

// ---------------------------------------------------------------- errors ---

__host__ __device__ constexpr unsigned err_bit(int code) { return 1u << code; }

// Lowest status code whose bit is set in `word` (SCONE_OK for 0).
int code_from_bits(unsigned word);

// The current device's 4-byte error word (a device variable of the library,
// looked up once per device), or null if the lookup failed.
unsigned* device_error_word();

#define SCONE_HIP_TRY(expr)                                \
    do {                                                   \
        if ((expr) != hipSuccess) return SCONE_EHIP;       \
    } while (0)

// Status of a sequence of launches: a grid the device cannot run is an
// argument error; any other runtime failure is SCONE_EHIP.
inline int status_of(hipError_t e) {
    return e == hipSuccess ? SCONE_OK
           : e == hipErrorInvalidConfiguration ? SCONE_EINVAL : SCONE_EHIP;
}

// n * size in bytes, saturated at 2^62 (sizes are validated against that bound).
inline int64_t span_bytes(int64_t n, int64_t size) {
    if (n <= 0 || size <= 0) return 0;
    return n > ((int64_t)1 << 62) / size ? ((int64_t)1 << 62) : n * size;
}

// True when the byte ranges [a, a + a_bytes) and [b, b + b_bytes) share a
// byte; a null pointer or an empty range shares nothing.  Used to reject
// outputs that alias inputs a concurrent workgroup still reads.
inline bool overlaps(const void* a, int64_t a_bytes, const void* b, int64_t b_bytes) {
    if (!a || !b || a_bytes <= 0 || b_bytes <= 0) return false;
    const uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b;
    return pa < pb + (uintptr_t)b_bytes && pb < pa + (uintptr_t)a_bytes;
}

// ------------------------------------------------------------- launches ----
// A dispatch states its grid as a count of work-items held in 32 bits per
// dimension, so a one-dimensional launch of 2^32 work-items or more would
// wrap around and run only the remainder, without an error.  Every kernel
// therefore takes the index of its first workgroup, `block0`, and launches go
// through launch_blocks, which issues consecutive launches of at most
// kMaxLaunchItems work-items each.

constexpr int64_t kMaxLaunchItems = (int64_t)1 << 31;

// Issues `blocks` workgroups of `threads` work-items: one(b0, grid) launches
// workgroups b0 .. b0 + grid.x - 1.  Returns the first launch error.
template <typename F>
hipError_t launch_blocks(int64_t blocks, int threads, F&& one) {
    const int64_t per = kMaxLaunchItems / threads;
    for (int64_t b0 = 0; b0 < blocks; b0 += per) {
        const int64_t n = blocks - b0 < per ? blocks - b0 : per;
        one(b0, dim3((unsigned)n));
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// This workgroup's index in the whole grid of a launch_blocks call.
__device__ __forceinline__ int64_t block_index(int64_t block0) {
    return block0 + (int64_t)blockIdx.x;
}

// ---------------------------------------------------------- f-gram keys ----
// An f-gram of n <= 7 tokens, each < 2^16, is one bit string:
//   bits [0, 4)              the length n
//   bits [4 + 16k, 20 + 16k) token k, oldest first
// held in two 64-bit words.  n <= 5 uses at most 84 bits, so its second word
// fits 32 bits and the key fits a 16-byte slot next to a 32-bit id.  A valid
// key never has a zero first word (n >= 2), so zero marks an empty slot.

constexpr int kTokenBits = 16;
constexpr int kMaxLenSlot16 = 5;

struct Key {
    uint64_t w0;
    uint64_t w1;
};

// Pack tokens tok[0..n) (n <= 7); the caller guarantees every token is in
// [0, 2^16).
template <typename Tok>
__device__ __forceinline__ Key pack_key(const Tok* tok, int n) {
    Key k{(uint64_t)n, 0};
#pragma unroll
    for (int i = 0; i < SCONE_MAX_FGRAM_LEN; ++i) {
        if (i < n) {
            const uint64_t v = (uint64_t)(uint32_t)tok[i];
            const int p = 4 + kTokenBits * i;
            if (p < 64) {
                k.w0 |= v << p;
                if (p + kTokenBits > 64) k.w1 |= v >> (64 - p);
            } else {
                k.w1 |= v << (p - 64);
            }
        }
    }
    return k;
}

// MurmurHash3's 64-bit finalizer (Appleby), applied to the two key words.
__device__ __forceinline__ uint64_t fmix64(uint64_t x) {
    x ^= x >> 33;
    x *= 0xff51afd7ed558ccdULL;
    x ^= x >> 33;
    x *= 0xc4ceb9fe1a85ec53ULL;
    x ^= x >> 33;
    return x;
}

__device__ __forceinline__ uint64_t hash_key(const Key& k) {
    return fmix64(k.w0 ^ (k.w1 * 0x9E3779B97F4A7C15ULL));
}

// ---------------------------------------------------------------- slots ----

struct alignas(16) Slot16 {
    uint64_t w0;
    uint32_t w1;
    int32_t id;
};

struct alignas(32) Slot32 {
    uint64_t w0;
    uint64_t w1;
    int32_t id;
    int32_t pad[3];
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <int SB>
struct SlotOps;

template <>
struct SlotOps<16> {
    using Slot = Slot16;
    // One 16-byte load returns the whole slot.
    __device__ __forceinline__ static void read(const Slot16* base, uint64_t s, uint64_t& w0,
                                                uint64_t& w1, int32_t& id) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(base + s);
        w0 = (uint64_t)v.x | ((uint64_t)v.y << 32);
        w1 = v.z;
        id = (int32_t)v.w;
    }
    __device__ __forceinline__ static void write_rest(Slot16* base, uint64_t s, const Key& k,
                                                      int32_t id) {
        base[s].w1 = (uint32_t)k.w1;
        base[s].id = id;
    }
};

template <>
struct SlotOps<32> {
    using Slot = Slot32;
    __device__ __forceinline__ static void read(const Slot32* base, uint64_t s, uint64_t& w0,
                                                uint64_t& w1, int32_t& id) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(base + s);
        const uint32_t c = reinterpret_cast<const uint32_t*>(base + s)[4];
        w0 = (uint64_t)a.x | ((uint64_t)a.y << 32);
        w1 = (uint64_t)a.z | ((uint64_t)a.w << 32);
        id = (int32_t)c;
    }
    __device__ __forceinline__ static void write_rest(Slot32* base, uint64_t s, const Key& k,
                                                      int32_t id) {
        base[s].w1 = k.w1;
        base[s].id = id;
    }
};

// Probing is linear, slot by slot, but starts at the first slot of the
// key's 64-byte bucket (the aligned group of 64 / SB slots that holds its
// hash slot).  Insertion claims the first empty slot in that order, so a
// lookup can read a whole bucket at once: a match anywhere in it is the key,
// and an empty slot in it (with no match) means the key is absent, because
// nothing is ever removed.  One round of independent loads usually settles
// a probe, instead of a chain of dependent single-slot loads.
template <int SB>
struct Bucket {
    static constexpr int kSlots = 64 / SB;
};

__device__ __forceinline__ uint64_t home_slot(const Key& k, uint64_t mask, int bucket_slots) {
    return (hash_key(k) & mask) & ~(uint64_t)(bucket_slots - 1);
}

// The id word of a slot.  Bits 0..30 hold the f-gram's row id, or
// kMarkerId for a marker: an entry that is not an f-gram but the suffix of
// one (see kExtBit).  Bit 31, kExtBit, is set on the entry of a length-3 key
// when some f-gram of length 4 or more ends with those three tokens, and on
// the entry of a length-5 key when some f-gram of length 6 or more ends with
// those five; every such suffix has an entry (the f-gram itself or a marker).
// A lookup can therefore skip the probes of lengths 4-5 (6-7) at a position
// whose length-3 (length-5) suffix has no entry with the bit, and the result
// is the same as probing every length.
constexpr uint32_t kExtBit = 0x80000000u;
constexpr int32_t kIdMask = 0x7FFFFFFF;
constexpr int32_t kMarkerId = 0x7FFFFFFF;  // a row id the build rejects

__device__ __forceinline__ bool entry_is_fgram(int32_t raw) { return (raw & kIdMask) != kMarkerId; }
__device__ __forceinline__ bool entry_extends(int32_t raw) { return raw < 0; }

// Returns true and the slot's raw id word when the key has an entry (an
// f-gram or a marker).  Bounded by the slot count.
template <int SB>
__device__ __forceinline__ bool probe_raw(const typename SlotOps<SB>::Slot* slots, uint64_t mask,
                                          const Key& k, int32_t& raw_out) {
    constexpr int BW = Bucket<SB>::kSlots;
    uint64_t s = home_slot(k, mask, BW);
    for (uint64_t step = 0; step <= mask; step += BW) {
        uint64_t w0[BW], w1[BW];
        int32_t id[BW];
#pragma unroll
        for (int i = 0; i < BW; ++i) SlotOps<SB>::read(slots, s + i, w0[i], w1[i], id[i]);
        bool empty = false;
#pragma unroll
        for (int i = 0; i < BW; ++i) {
            if (w0[i] == k.w0 && w1[i] == k.w1) {
                raw_out = id[i];
                return true;
            }
            empty |= w0[i] == 0;
        }
        if (empty) return false;
        s = (s + BW) & mask;
    }
    return false;
}

// Returns true and the row id when the key is an f-gram of the table.
template <int SB>
__device__ __forceinline__ bool probe(const typename SlotOps<SB>::Slot* slots, uint64_t mask,
                                      const Key& k, int32_t& id_out) {
    int32_t raw = 0;
    if (!probe_raw<SB>(slots, mask, k, raw) || !entry_is_fgram(raw)) return false;
    id_out = raw & kIdMask;
    return true;
}

}  // namespace scone

struct scone_table;

namespace scone {
// Launch the lookup kernel (max_n already clamped to the table's K); a null
// `ids`, `lens` or `hist` output is skipped.  `hist` accumulates, per matched
// length 1..K, the number of positions (index = length).
hipError_t launch_lookup(const scone_table* tb, const int32_t* X, int64_t B, int64_t T,
                         int max_n, int32_t* ids, int8_t* lens, unsigned* err, hipStream_t st,
                         unsigned long long* hist = nullptr);
// Zero `bytes` of device memory with a kernel and raise SCONE_EROW (a table
// without rows has no valid row id).
hipError_t launch_zero_rows(void* out, int64_t bytes, unsigned* err, hipStream_t st);
// Launch the gather kernel that suits the row width and alignment (the whole of
// scone_gather after its argument checks).
hipError_t launch_gather_any(const int32_t* ids, int64_t n_tok, const void* rows, int64_t n_rows,
                             int64_t row_bytes, void* out, unsigned* err, hipStream_t st);
}  // namespace scone

// The opaque table handle.
struct scone_table {
    int device;
    int32_t max_len;    // longest f-gram the table can hold (K)
    int32_t slot_bytes; // 16 or 32
    int64_t n;          // f-grams stored
    int64_t capacity;   // slots, a power of two
    int64_t entries;    // slots in use: the f-grams plus their suffix markers
    void* slots;        // device memory, capacity * slot_bytes
};
