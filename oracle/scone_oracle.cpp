// CPU oracle for SCONE's inference-time f-gram embedding (test infrastructure).
//
// This file is test infrastructure only.  It is used by the test suite, by the
// package's smoke check and by the benchmark's CPU-baseline leg; the product
// path never calls it.  It shares no code, header, table or constant with the
// GPU library: keys here are the raw bytes of the f-gram's int32 tokens held in
// a std::unordered_map, and rows are copied with memcpy.
//
// What it computes (Algorithm 1, inference branch, of "Scaling Embedding
// Layers in Language Models"):  for position i of a sequence, j is the
// smallest j' < i such that the n-gram (sigma_j', ..., sigma_i) is an f-gram;
// if no such j' exists, j = i.  If j = i the output is the token's own
// embedding T(sigma_i), otherwise the f-gram embedding F(sigma_j..sigma_i).
// With 0-based position t and n = t - j + 1 this reads: the largest
// n in [2, min(max_n, t + 1)] whose suffix of length n is in the f-gram set.
// The f-gram set is a subset of V^[2, K] (Section 3), so length-1 entries are
// rejected.  Matches never look before the start of the row (Algorithm 1 runs
// on one sequence).  The row table is a single matrix: rows 0..V-1 hold the
// token embeddings T and each f-gram row is addressed by its caller-given id
// (Section 2 stores F as a dense matrix plus a dictionary to row indices).
//
// Single-threaded by definition.
#include <cstdint>
#include <cstring>
#include <string>
#include <unordered_map>
#include <new>

namespace {

// Oracle status codes (independent of the GPU library's codes).
enum : int {
    OR_OK = 0,
    OR_BAD_ARG = 1,
    OR_BAD_LENGTH = 2,
    OR_BAD_ID = 3,
    OR_DUPLICATE = 4,
    OR_BAD_ROW = 5,
};

struct OracleSet {
    std::unordered_map<std::string, int32_t> dict;  // f-gram bytes -> row id
    int32_t longest = 0;                            // K of this set
};

std::string key_of(const int32_t* toks, int32_t n) {
    return std::string(reinterpret_cast<const char*>(toks), sizeof(int32_t) * (size_t)n);
}

}  // namespace

extern "C" {

// Build the dictionary from n f-grams.  fgrams is [n, stride] row-major; row k
// holds lengths[k] tokens (the rest is ignored).  Returns OR_BAD_LENGTH for a
// length outside [2, stride], OR_BAD_ID for a negative id, OR_DUPLICATE when an
// f-gram occurs twice (a set holds each element once).  On success *out owns
// the dictionary until oracle_destroy.
int oracle_build(const int32_t* fgrams, const int32_t* lengths, const int32_t* ids,
                 int64_t n, int32_t stride, void** out) {
    if (!out || n < 0 || stride < 1 || (n > 0 && (!fgrams || !lengths || !ids)))
        return OR_BAD_ARG;
    *out = nullptr;
    OracleSet* s = new (std::nothrow) OracleSet();
    if (!s) return OR_BAD_ARG;
    s->dict.reserve((size_t)n);
    for (int64_t k = 0; k < n; ++k) {
        int32_t len = lengths[k];
        if (len < 2 || len > stride) { delete s; return OR_BAD_LENGTH; }
        if (ids[k] < 0) { delete s; return OR_BAD_ID; }
        auto ins = s->dict.emplace(key_of(fgrams + k * (int64_t)stride, len), ids[k]);
        if (!ins.second) { delete s; return OR_DUPLICATE; }
        if (len > s->longest) s->longest = len;
    }
    *out = s;
    return OR_OK;
}

void oracle_destroy(void* h) { delete static_cast<OracleSet*>(h); }

int64_t oracle_size(const void* h) {
    return h ? (int64_t)static_cast<const OracleSet*>(h)->dict.size() : -1;
}

// Longest-suffix lookup over a [B, T] token matrix (Algorithm 1's choice of
// j).  For every (b, t): ids[b,t] = F[suffix of length n] for the largest n in
// [2, min(max_n, t+1)] whose suffix is in the set, and match_len[b,t] = n;
// otherwise ids[b,t] = X[b,t] and match_len[b,t] = 1.  Every n is tested
// independently (the set need not be closed under taking suffixes).
// match_len may be null.  Returns the number of dictionary queries made, or
// -1 on a bad argument.
int64_t oracle_lookup(const void* h, const int32_t* X, int64_t B, int64_t T, int32_t max_n,
                      int32_t* ids, int8_t* match_len) {
    const OracleSet* s = static_cast<const OracleSet*>(h);
    if (!s || B < 0 || T < 0 || max_n < 1 || (B * T > 0 && (!X || !ids))) return -1;
    int64_t queries = 0;
    for (int64_t b = 0; b < B; ++b) {
        const int32_t* row = X + b * T;
        for (int64_t t = 0; t < T; ++t) {
            int32_t id = row[t];
            int32_t len = 1;
            int64_t top = max_n < t + 1 ? (int64_t)max_n : t + 1;
            for (int64_t n = top; n >= 2; --n) {
                ++queries;
                auto it = s->dict.find(key_of(row + (t - n + 1), (int32_t)n));
                if (it != s->dict.end()) { id = it->second; len = (int32_t)n; break; }
            }
            ids[b * T + t] = id;
            if (match_len) match_len[b * T + t] = (int8_t)len;
        }
    }
    return queries;
}

// Row gather: out[k, :] = table[ids[k], :] as raw bytes (the embedding layer
// is a pure memory fetch).  Returns OR_BAD_ROW if an id is outside
// [0, n_rows); rows before the offending one are already written.
int oracle_gather(const int32_t* ids, int64_t n_tok, const uint8_t* table, int64_t n_rows,
                  int64_t row_bytes, uint8_t* out) {
    if (n_tok < 0 || n_rows < 0 || row_bytes < 1 || (n_tok > 0 && (!ids || !table || !out)))
        return OR_BAD_ARG;
    for (int64_t k = 0; k < n_tok; ++k) {
        int64_t r = ids[k];
        if (r < 0 || r >= n_rows) return OR_BAD_ROW;
        std::memcpy(out + k * row_bytes, table + r * row_bytes, (size_t)row_bytes);
    }
    return OR_OK;
}

}  // extern "C"
