// Split row placement with per-batch deduplication of off-accelerator rows.
//
// The paper keeps the token embedding layer T on the accelerator and offloads
// the f-gram layer F to main memory (Section 3.2; off-accelerator storage,
// Sections 2 and 4.3).  Here ids below `n_near` address `near` rows in device
// memory and ids from n_near up address `far` rows in host-mapped pinned
// memory.  A batch usually names the same f-gram several times, so every
// distinct far id crosses PCIe once:
//   1. k_split_clear  - reset the dedupe set and the counter (a kernel, so the
//                       call can sit in a captured graph),
//   2. k_split_insert - put every far id of the batch into an open-addressing
//                       set (compare-and-swap on the id itself),
//   3. k_split_number - give every occupied set slot a staging index,
//   4. k_split_fetch  - copy each distinct far row from host memory into the
//                       device staging area, one wavefront per row,
//   5. k_split_gather - out[k] = near[id] or staged[index of id], from HBM.
#include <mutex>

#include "scone_internal.h"

namespace scone {
namespace {

constexpr int kThreads = 256;
constexpr int32_t kEmpty = -1;

__device__ __forceinline__ uint64_t id_hash(int32_t id) {
    return fmix64((uint64_t)(uint32_t)id * 0x9E3779B97F4A7C15ULL);
}

__global__ __launch_bounds__(kThreads) void k_split_clear(int32_t* keys, uint64_t cap,
                                                          unsigned* count, int64_t block0) {
    const uint64_t i = (uint64_t)block_index(block0) * kThreads + threadIdx.x;
    if (i < cap) keys[i] = kEmpty;
    if (i == 0) *count = 0;
}

__global__ __launch_bounds__(kThreads) void k_split_insert(const int32_t* __restrict__ ids,
                                                           int64_t n_tok, int64_t n_near,
                                                           int64_t n_far, int32_t* keys,
                                                           uint64_t mask, int64_t block0) {
    const int64_t k = block_index(block0) * kThreads + threadIdx.x;
    if (k >= n_tok) return;
    const int32_t id = ids[k];
    if ((int64_t)id < n_near || (int64_t)id >= n_near + n_far) return;  // near or bad
    uint64_t s = id_hash(id) & mask;
    for (uint64_t step = 0; step <= mask; ++step) {
        const int32_t old = atomicCAS(keys + s, kEmpty, id);
        if (old == kEmpty || old == id) return;
        s = (s + 1) & mask;
    }
}

__global__ __launch_bounds__(kThreads) void k_split_number(const int32_t* __restrict__ keys,
                                                           int32_t* __restrict__ index,
                                                           int32_t* __restrict__ unique,
                                                           uint64_t cap, unsigned* count,
                                                           int64_t block0) {
    const uint64_t s = (uint64_t)block_index(block0) * kThreads + threadIdx.x;
    if (s >= cap) return;
    const int32_t id = keys[s];
    if (id == kEmpty) return;
    const unsigned u = atomicAdd(count, 1u);
    index[s] = (int32_t)u;
    unique[u] = id;
}

// One wavefront per distinct far row; rows are row_bytes / 16 units.
__global__ __launch_bounds__(kThreads) void k_split_fetch(const int32_t* __restrict__ unique,
                                                          const unsigned* __restrict__ count,
                                                          int64_t n_near, const u32x4* far,
                                                          int64_t upr, u32x4* __restrict__ staging,
                                                          int32_t* __restrict__ n_unique,
                                                          int64_t block0) {
    const int64_t u = block_index(block0) * (kThreads / 64) +
                      __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const unsigned total = *count;
    if (u == 0 && threadIdx.x == 0 && n_unique) *n_unique = (int32_t)total;
    if (u >= (int64_t)total) return;  // wave-uniform
    const int lane = threadIdx.x & 63;
    const u32x4* src = far + ((int64_t)unique[u] - n_near) * upr;
    u32x4* dst = staging + u * upr;
    for (int64_t c = lane; c < upr; c += 4 * 64) {
        u32x4 v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (c + j * 64 < upr) v[j] = src[c + j * 64];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (c + j * 64 < upr) dst[c + j * 64] = v[j];
    }
}

// One wavefront per output row.
__global__ __launch_bounds__(kThreads) void k_split_gather(
    const int32_t* __restrict__ ids, int64_t n_tok, const u32x4* __restrict__ near,
    int64_t n_near, int64_t n_far, const int32_t* __restrict__ keys,
    const int32_t* __restrict__ index, uint64_t mask, const u32x4* __restrict__ staging,
    int64_t upr, u32x4* __restrict__ out, unsigned* __restrict__ err, int64_t block0) {
    const int64_t r = block_index(block0) * (kThreads / 64) +
                      __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (r >= n_tok) return;  // wave-uniform
    const int lane = threadIdx.x & 63;
    const int32_t id = ids[r];
    const u32x4* src = nullptr;
    if (id >= 0 && (int64_t)id < n_near) {
        src = near + (int64_t)id * upr;
    } else if ((int64_t)id >= n_near && (int64_t)id < n_near + n_far) {
        uint64_t s = id_hash(id) & mask;
        for (uint64_t step = 0; step <= mask; ++step) {
            const int32_t key = keys[s];
            if (key == id) {
                src = staging + (int64_t)index[s] * upr;
                break;
            }
            if (key == kEmpty) break;  // cannot happen: every far id was inserted
            s = (s + 1) & mask;
        }
    }
    u32x4* dst = out + r * upr;
    if (src) {
        for (int64_t c = lane; c < upr; c += 4 * 64) {
            u32x4 v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (c + j * 64 < upr) v[j] = src[c + j * 64];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (c + j * 64 < upr) __builtin_nontemporal_store(v[j], dst + c + j * 64);
        }
    } else {
        for (int64_t c = lane; c < upr; c += 64) dst[c] = u32x4{};
        if (lane == 0) atomicOr(err, err_bit(SCONE_EROW));
    }
}

// Workspace layout for n_tok tokens of row_bytes each (all parts 256-byte
// aligned): the dedupe set's keys and staging indices ([cap] each, cap the
// smallest power of two >= 2 * n_tok), the distinct far ids in staging order
// ([n_tok]), the counter, and the staged rows ([n_tok, row_bytes]).
struct Layout {
    uint64_t cap;
    int64_t keys, index, unique, count, staging, total;
};

Layout layout(int64_t n_tok, int64_t row_bytes) {
    auto up = [](int64_t x) { return (x + 255) & ~(int64_t)255; };
    Layout l;
    l.cap = 64;
    while ((int64_t)l.cap < 2 * n_tok) l.cap <<= 1;
    l.keys = 0;
    l.index = up(l.keys + 4 * (int64_t)l.cap);
    l.unique = up(l.index + 4 * (int64_t)l.cap);
    l.count = up(l.unique + 4 * n_tok);
    l.staging = up(l.count + 4);
    l.total = up(l.staging + n_tok * row_bytes);
    return l;
}

}  // namespace
}  // namespace scone

extern "C" int64_t scone_gather_split_workspace(int64_t n_tok, int64_t row_bytes) {
    if (n_tok < 0 || row_bytes <= 0 || n_tok > ((int64_t)1 << 40) / row_bytes) return -1;
    return scone::layout(n_tok, row_bytes).total;
}

namespace scone {
namespace {

// Everything of scone_gather_split after the workspace is known.
int split_run(const int32_t* fgram_ids, int64_t n_tok, const void* near_rows, int64_t n_near,
              const void* far_rows, int64_t n_far, int64_t row_bytes, void* out,
              void* workspace, int64_t workspace_bytes, int32_t* n_unique, void* stream) {
    const Layout l = layout(n_tok, row_bytes);
    if (workspace_bytes < l.total) return SCONE_EINVAL;
    unsigned* err = device_error_word();
    if (!err) return SCONE_EHIP;
    hipStream_t st = static_cast<hipStream_t>(stream);
    uint8_t* ws = static_cast<uint8_t*>(workspace);
    int32_t* keys = reinterpret_cast<int32_t*>(ws + l.keys);
    int32_t* index = reinterpret_cast<int32_t*>(ws + l.index);
    int32_t* unique = reinterpret_cast<int32_t*>(ws + l.unique);
    unsigned* count = reinterpret_cast<unsigned*>(ws + l.count);
    u32x4* staging = reinterpret_cast<u32x4*>(ws + l.staging);
    const int64_t upr = row_bytes / 16;
    const uint64_t mask = l.cap - 1;
    const int64_t g_cap = ((int64_t)l.cap + kThreads - 1) / kThreads;
    const int64_t g_tok = (n_tok + kThreads - 1) / kThreads;
    const int64_t g_rows = (n_tok + 3) / 4;
    const dim3 block(kThreads);
    hipError_t e = launch_blocks(g_cap, kThreads, [&](int64_t b0, dim3 grid) {
        hipLaunchKernelGGL(k_split_clear, grid, block, 0, st, keys, l.cap, count, b0);
    });
    if (e == hipSuccess)
        e = launch_blocks(g_tok, kThreads, [&](int64_t b0, dim3 grid) {
            hipLaunchKernelGGL(k_split_insert, grid, block, 0, st, fgram_ids, n_tok, n_near,
                               n_far, keys, mask, b0);
        });
    if (e == hipSuccess)
        e = launch_blocks(g_cap, kThreads, [&](int64_t b0, dim3 grid) {
            hipLaunchKernelGGL(k_split_number, grid, block, 0, st, keys, index, unique, l.cap,
                               count, b0);
        });
    if (e == hipSuccess)
        e = launch_blocks(g_rows, kThreads, [&](int64_t b0, dim3 grid) {
            hipLaunchKernelGGL(k_split_fetch, grid, block, 0, st, unique, count, n_near,
                               static_cast<const u32x4*>(far_rows), upr, staging, n_unique, b0);
        });
    if (e == hipSuccess)
        e = launch_blocks(g_rows, kThreads, [&](int64_t b0, dim3 grid) {
            hipLaunchKernelGGL(k_split_gather, grid, block, 0, st, fgram_ids, n_tok,
                               static_cast<const u32x4*>(near_rows), n_near, n_far, keys, index,
                               mask, staging, upr, static_cast<u32x4*>(out), err, b0);
        });
    return status_of(e);
}

// Argument checks shared by both entry points (the workspace is checked by
// each); SCONE_OK means the call has work to do.
int split_args(const int32_t* fgram_ids, int64_t n_tok, const void* near_rows, int64_t n_near,
               const void* far_rows, int64_t n_far, int64_t row_bytes, const void* out,
               const int32_t* n_unique) {
    if (n_tok < 0 || n_near < 0 || n_far < 0 || row_bytes <= 0) return SCONE_EINVAL;
    if (row_bytes % 16 != 0 ||
        ((uintptr_t)near_rows | (uintptr_t)far_rows | (uintptr_t)out) % 16 != 0)
        return SCONE_EINVAL;
    if (n_near + n_far > ((int64_t)1 << 31) || n_tok > ((int64_t)1 << 40) / row_bytes)
        return SCONE_EINVAL;
    if (n_tok > 0 && (!fgram_ids || !out || (n_near > 0 && !near_rows) ||
                      (n_far > 0 && !far_rows)))
        return SCONE_EINVAL;
    if (overlaps(out, n_tok * row_bytes, fgram_ids, span_bytes(n_tok, 4)) ||
        overlaps(out, n_tok * row_bytes, near_rows, span_bytes(n_near, row_bytes)))
        return SCONE_EINVAL;
    // n_unique is written by the fetch kernel while the gather kernel still
    // reads the ids and writes out.
    if (overlaps(n_unique, 4, out, n_tok * row_bytes) ||
        overlaps(n_unique, 4, fgram_ids, span_bytes(n_tok, 4)))
        return SCONE_EINVAL;
    return SCONE_OK;
}

}  // namespace
}  // namespace scone

extern "C" int scone_gather_split(const int32_t* fgram_ids, int64_t n_tok, const void* near_rows,
                                  int64_t n_near, const void* far_rows, int64_t n_far,
                                  int64_t row_bytes, void* out, void* workspace,
                                  int64_t workspace_bytes, int32_t* n_unique, void* stream) {
    using namespace scone;
    const int rc = split_args(fgram_ids, n_tok, near_rows, n_near, far_rows, n_far, row_bytes,
                              out, n_unique);
    if (rc != SCONE_OK) return rc;
    if ((uintptr_t)workspace % 16 != 0) return SCONE_EINVAL;
    if (n_tok == 0) return SCONE_OK;
    if (!workspace) return SCONE_EINVAL;
    // The kernels write the workspace while they read every input and write
    // out and n_unique: it may share memory with none of them.
    const int64_t used = layout(n_tok, row_bytes).total;
    if (overlaps(workspace, used, fgram_ids, span_bytes(n_tok, 4)) ||
        overlaps(workspace, used, near_rows, span_bytes(n_near, row_bytes)) ||
        overlaps(workspace, used, far_rows, span_bytes(n_far, row_bytes)) ||
        overlaps(workspace, used, out, n_tok * row_bytes) ||
        overlaps(workspace, used, n_unique, 4))
        return SCONE_EINVAL;
    return split_run(fgram_ids, n_tok, near_rows, n_near, far_rows, n_far, row_bytes, out,
                     workspace, workspace_bytes, n_unique, stream);
}

namespace scone {
namespace {

// The scratch of scone_gather_split_static: a fixed buffer in the library's
// own device data, one copy per GPU, held until the process ends.  Host code
// never uses this name as an address: each device's copy is looked up once
// with hipGetSymbolAddress and that pointer is passed to the kernels.
static __device__ __align__(256) uint8_t scratch[SCONE_SPLIT_STATIC_BYTES];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxScratchDevices] = {};

// This device's copy of `scratch`, or null if the lookup failed.
void* device_scratch() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxScratchDevices) return nullptr;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();
            return nullptr;
        }
        g_scratch[dev] = p;
    }
    return g_scratch[dev];
}

}  // namespace
}  // namespace scone

extern "C" int scone_gather_split_static(const int32_t* fgram_ids, int64_t n_tok,
                                         const void* near_rows, int64_t n_near,
                                         const void* far_rows, int64_t n_far, int64_t row_bytes,
                                         void* out, int32_t* n_unique, void* stream) {
    using namespace scone;
    const int rc = split_args(fgram_ids, n_tok, near_rows, n_near, far_rows, n_far, row_bytes,
                              out, n_unique);
    if (rc != SCONE_OK) return rc;
    if (n_tok == 0) return SCONE_OK;
    if (layout(n_tok, row_bytes).total > (int64_t)SCONE_SPLIT_STATIC_BYTES) return SCONE_ESCRATCH;
    void* ws = device_scratch();
    if (!ws) return SCONE_EHIP;
    return split_run(fgram_ids, n_tok, near_rows, n_near, far_rows, n_far, row_bytes, out, ws,
                     (int64_t)SCONE_SPLIT_STATIC_BYTES, n_unique, stream);
}
