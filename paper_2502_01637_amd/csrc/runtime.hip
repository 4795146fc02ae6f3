// Error word, status strings, pinned host memory and table bookkeeping.
#include <mutex>

#include "scone_internal.h"

namespace scone {

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_mu;
unsigned* g_err_word[kMaxDevices] = {};
// The error word lives in the library's own device data (one copy per GPU,
// zero when the code object loads), so raising and checking errors never
// allocates.  Host code reaches it only through hipGetSymbolAddress.
__device__ unsigned g_err_bits;
}  // namespace

int code_from_bits(unsigned word) {
    for (int c = 1; c < 32; ++c)
        if (word & err_bit(c)) return c;
    return SCONE_OK;
}

unsigned* device_error_word() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_err_word[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(g_err_bits)) != hipSuccess || !p) {
            (void)hipGetLastError();
            return nullptr;
        }
        g_err_word[dev] = static_cast<unsigned*>(p);
    }
    return g_err_word[dev];
}

namespace {
// Clears exactly the bits the host read, so that a bit another stream's
// kernel raised after the read survives until the next check.
__global__ void k_clear_bits(unsigned* word, unsigned bits) { atomicAnd(word, ~bits); }
}  // namespace

}  // namespace scone

extern "C" {

int scone_check(void* stream) {
    hipStream_t st = static_cast<hipStream_t>(stream);
    SCONE_HIP_TRY(hipStreamSynchronize(st));
    unsigned* w = scone::device_error_word();
    if (!w) return SCONE_EHIP;
    unsigned h = 0;
    SCONE_HIP_TRY(hipMemcpyAsync(&h, w, sizeof(h), hipMemcpyDeviceToHost, st));
    SCONE_HIP_TRY(hipStreamSynchronize(st));
    if (h) {
        hipLaunchKernelGGL(scone::k_clear_bits, dim3(1), dim3(1), 0, st, w, h);
        SCONE_HIP_TRY(hipGetLastError());
        SCONE_HIP_TRY(hipStreamSynchronize(st));
    }
    return scone::code_from_bits(h);
}

const char* scone_strerror(int code) {
    switch (code) {
        case SCONE_OK: return "ok";
        case SCONE_EINVAL: return "invalid argument";
        case SCONE_ELEN: return "f-gram length outside [2, max_len]";
        case SCONE_EID: return "f-gram id outside [0, 2^31 - 1)";
        case SCONE_EDUP: return "duplicate f-gram in build input";
        case SCONE_EFULL: return "hash table full";
        case SCONE_ENOMEM: return "out of memory";
        case SCONE_EHIP: return "HIP runtime error";
        case SCONE_ETOKEN: return "token outside [0, 65536)";
        case SCONE_EROW: return "row id outside [0, n_rows)";
        case SCONE_ESCRATCH: return "call exceeds the fixed scratch buffer";
        default: return "unknown status";
    }
}

int scone_host_alloc(int64_t bytes, void** host_ptr, void** device_ptr) {
    if (!host_ptr || !device_ptr || bytes <= 0) return SCONE_EINVAL;
    *host_ptr = nullptr;
    *device_ptr = nullptr;
    void* h = nullptr;
    // Mapped so kernels can read it; non-coherent so the GPU may cache it.
    if (hipHostMalloc(&h, (size_t)bytes, hipHostMallocMapped | hipHostMallocNonCoherent) !=
        hipSuccess)
        return SCONE_ENOMEM;
    void* d = nullptr;
    if (hipHostGetDevicePointer(&d, h, 0) != hipSuccess) {
        (void)hipHostFree(h);
        return SCONE_EHIP;
    }
    *host_ptr = h;
    *device_ptr = d;
    return SCONE_OK;
}

int scone_host_free(void* host_ptr) {
    if (!host_ptr) return SCONE_OK;
    SCONE_HIP_TRY(hipHostFree(host_ptr));
    return SCONE_OK;
}

void scone_table_destroy(scone_table_t* t) {
    if (!t) return;
    int cur = 0;
    const bool have_cur = hipGetDevice(&cur) == hipSuccess;
    if (have_cur && cur != t->device) (void)hipSetDevice(t->device);
    if (t->slots) (void)hipFree(t->slots);
    if (have_cur && cur != t->device) (void)hipSetDevice(cur);
    delete t;
}

int scone_table_info(const scone_table_t* t, int64_t* n, int64_t* capacity, int32_t* max_len,
                     int32_t* slot_bytes, int64_t* entries) {
    if (!t) return SCONE_EINVAL;
    if (n) *n = t->n;
    if (capacity) *capacity = t->capacity;
    if (max_len) *max_len = t->max_len;
    if (slot_bytes) *slot_bytes = t->slot_bytes;
    if (entries) *entries = t->entries;
    return SCONE_OK;
}

}  // extern "C"
