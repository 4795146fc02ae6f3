/*
 * scone_embed: the library's C ABI used from plain C with the HIP runtime
 * only (no Python, no PyTorch): build the f-gram dictionary, look up the
 * longest f-gram of every position, gather the rows, check the error word.
 *
 * Usage: scone_embed <dir>
 *   <dir>/meta.txt     "n K B T max_n n_rows row_bytes"
 *   <dir>/fgrams.bin   int32 [n, K], oldest token first, padded with -1
 *   <dir>/lengths.bin  int32 [n]
 *   <dir>/ids.bin      int32 [n]
 *   <dir>/tokens.bin   int32 [B, T]
 *   <dir>/rows.bin     uint8 [n_rows, row_bytes]
 * Writes <dir>/ids_out.bin (int32 [B, T]), <dir>/len_out.bin (int8 [B, T]),
 * <dir>/out.bin (uint8 [B, T, row_bytes]); exit status 0 on success.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <hip/hip_runtime_api.h>

#include "scone.h"

static void* read_file(const char* dir, const char* name, size_t bytes) {
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", dir, name);
    FILE* f = fopen(path, "rb");
    if (!f) return NULL;
    void* p = malloc(bytes ? bytes : 1);
    if (p && bytes && fread(p, 1, bytes, f) != bytes) {
        free(p);
        p = NULL;
    }
    fclose(f);
    return p;
}

static int write_file(const char* dir, const char* name, const void* p, size_t bytes) {
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", dir, name);
    FILE* f = fopen(path, "wb");
    if (!f) return 1;
    const int bad = bytes && fwrite(p, 1, bytes, f) != bytes;
    return fclose(f) != 0 || bad;
}

static void* to_device(const void* host, size_t bytes) {
    void* d = NULL;
    if (hipMalloc(&d, bytes ? bytes : 16) != hipSuccess) return NULL;
    if (bytes && hipMemcpy(d, host, bytes, hipMemcpyHostToDevice) != hipSuccess) return NULL;
    return d;
}

#define CHECK(call)                                                                  \
    do {                                                                             \
        const int rc_ = (call);                                                      \
        if (rc_ != SCONE_OK) {                                                       \
            fprintf(stderr, "%s: %s\n", #call, scone_strerror(rc_));                  \
            return 2;                                                                \
        }                                                                            \
    } while (0)

int main(int argc, char** argv) {
    if (argc != 2) {
        fprintf(stderr, "usage: %s <dir>\n", argv[0]);
        return 1;
    }
    const char* dir = argv[1];
    char path[4096];
    snprintf(path, sizeof path, "%s/meta.txt", dir);
    FILE* mf = fopen(path, "r");
    long long n, K, B, T, max_n, n_rows, row_bytes;
    if (!mf || fscanf(mf, "%lld %lld %lld %lld %lld %lld %lld", &n, &K, &B, &T, &max_n, &n_rows,
                      &row_bytes) != 7) {
        fprintf(stderr, "cannot read %s\n", path);
        return 1;
    }
    fclose(mf);
    const size_t n_tok = (size_t)(B * T);
    int32_t* fgrams = read_file(dir, "fgrams.bin", (size_t)(n * K) * 4);
    int32_t* lengths = read_file(dir, "lengths.bin", (size_t)n * 4);
    int32_t* ids = read_file(dir, "ids.bin", (size_t)n * 4);
    int32_t* tokens = read_file(dir, "tokens.bin", n_tok * 4);
    uint8_t* rows = read_file(dir, "rows.bin", (size_t)(n_rows * row_bytes));
    if (!fgrams || !lengths || !ids || !tokens || !rows) {
        fprintf(stderr, "cannot read the inputs in %s\n", dir);
        return 1;
    }

    void* d_fg = to_device(fgrams, (size_t)(n * K) * 4);
    void* d_len = to_device(lengths, (size_t)n * 4);
    void* d_ids = to_device(ids, (size_t)n * 4);
    void* d_tok = to_device(tokens, n_tok * 4);
    void* d_rows = to_device(rows, (size_t)(n_rows * row_bytes));
    void *d_fid = NULL, *d_ml = NULL, *d_out = NULL;
    if (!d_fg || !d_len || !d_ids || !d_tok || !d_rows ||
        hipMalloc(&d_fid, n_tok * 4 + 16) != hipSuccess ||
        hipMalloc(&d_ml, n_tok + 16) != hipSuccess ||
        hipMalloc(&d_out, n_tok * (size_t)row_bytes + 16) != hipSuccess) {
        fprintf(stderr, "device allocation failed\n");
        return 1;
    }
    hipStream_t stream;
    if (hipStreamCreate(&stream) != hipSuccess) return 1;

    scone_table_t* table = NULL;
    CHECK(scone_build_fgram_table(d_fg, d_len, d_ids, n, (int32_t)K, 0.5, stream, &table));
    int64_t stored = 0, capacity = 0;
    int32_t klen = 0, slot_bytes = 0;
    CHECK(scone_table_info(table, &stored, &capacity, &klen, &slot_bytes, NULL));
    CHECK(scone_lookup(table, d_tok, B, T, (int32_t)max_n, d_fid, d_ml, stream));
    CHECK(scone_gather(d_fid, (int64_t)n_tok, d_rows, n_rows, row_bytes, d_out, SCONE_PLACE_HBM,
                       stream));
    CHECK(scone_check(stream));

    int32_t* fid = malloc(n_tok * 4 + 4);
    int8_t* ml = malloc(n_tok + 1);
    uint8_t* out = malloc(n_tok * (size_t)row_bytes + 1);
    if (!fid || !ml || !out ||
        hipMemcpy(fid, d_fid, n_tok * 4, hipMemcpyDeviceToHost) != hipSuccess ||
        hipMemcpy(ml, d_ml, n_tok, hipMemcpyDeviceToHost) != hipSuccess ||
        hipMemcpy(out, d_out, n_tok * (size_t)row_bytes, hipMemcpyDeviceToHost) != hipSuccess)
        return 1;
    if (write_file(dir, "ids_out.bin", fid, n_tok * 4) ||
        write_file(dir, "len_out.bin", ml, n_tok) ||
        write_file(dir, "out.bin", out, n_tok * (size_t)row_bytes))
        return 1;
    printf("scone_embed: %lld f-grams in %lld slots of %d bytes, %zu positions\n",
           (long long)stored, (long long)capacity, slot_bytes, n_tok);
    scone_table_destroy(table);
    hipStreamDestroy(stream);
    hipFree(d_fg); hipFree(d_len); hipFree(d_ids); hipFree(d_tok); hipFree(d_rows);
    hipFree(d_fid); hipFree(d_ml); hipFree(d_out);
    free(fgrams); free(lengths); free(ids); free(tokens); free(rows);
    free(fid); free(ml); free(out);
    return 0;
}
