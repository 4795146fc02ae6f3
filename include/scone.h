/*
 * scone.h: C ABI of the MI355X f-gram embedding library (libscone.so).
 *
 * The library implements the inference branch of the SCONE embedding
 * (Algorithm 1 of "Scaling Embedding Layers in Language Models"): for each
 * token it finds the longest f-gram that ends at that token, maps it to a row
 * id, and copies that row of a precomputed embedding table; when no f-gram
 * matches it copies the token's own row.  The f-gram layer is a key-value
 * store from f-grams to rows (Section 2: a dense matrix plus a hash
 * dictionary to row indices), and the rows live either in HBM or in
 * host-pinned memory read over PCIe (the off-accelerator placement of
 * Sections 2 and 3.2).
 *
 * Conventions for every call:
 *  - Pointers are device pointers unless stated otherwise; "host-mapped"
 *    means a device-accessible pointer to pinned host memory (see
 *    scone_host_alloc).
 *  - `stream` is a hipStream_t passed as void*; NULL is the default stream.
 *    Calls run on the calling thread's current HIP device.
 *  - Every call returns a scone_status.  Argument errors are detected on the
 *    host before any launch and change nothing.  Errors that depend on
 *    device data (SCONE_ETOKEN, SCONE_EROW) cannot be seen by the host
 *    without a sync: asynchronous calls raise them in the device's error
 *    word and report them through scone_check().  After such an error the
 *    contents of the outputs are unspecified.
 *  - No call allocates device memory except scone_build_fgram_table,
 *    scone_host_alloc and the synchronous offline calls
 *    scone_discover_fgrams (when given no workspace) and
 *    scone_fgram_model_forward.  The device error word is a variable of the
 *    library's own code object (one per GPU), not an allocation.
 *  - All buffers are owned by the caller except the table handle, which the
 *    library owns until scone_table_destroy.
 */
#ifndef SCONE_H
#define SCONE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct scone_table scone_table_t;

enum scone_status {
    SCONE_OK = 0,
    SCONE_EINVAL = 1,  /* bad argument: null pointer, negative size, bad window ... */
    SCONE_ELEN = 2,    /* an f-gram length outside [2, max_len] */
    SCONE_EID = 3,     /* an f-gram id outside [0, 2^31 - 1) */
    SCONE_EDUP = 4,    /* the same f-gram appears twice in the build input */
    SCONE_EFULL = 5,   /* hash table has no free slot (cannot happen for max_load <= 0.9) */
    SCONE_ENOMEM = 6,  /* device or pinned host allocation failed */
    SCONE_EHIP = 7,    /* a HIP runtime call failed */
    SCONE_ETOKEN = 8,  /* a token outside [0, SCONE_TOKEN_LIMIT) */
    SCONE_EROW = 9,    /* a row id outside [0, n_rows) */
    SCONE_ESCRATCH = 10 /* the call needs more than the library's fixed scratch buffer */
};

enum scone_placement {
    SCONE_PLACE_HBM = 0,   /* `rows` is device memory */
    SCONE_PLACE_HOST = 1   /* `rows` is host-mapped pinned memory, read over PCIe */
};

#define SCONE_MAX_FGRAM_LEN 7     /* longest f-gram a table can hold */
#define SCONE_TOKEN_LIMIT 65536   /* tokens are packed as 16-bit fields */

/*
 * Build the f-gram dictionary (the key-value store F of Algorithm 1, whose
 * keys are the set V_fgram of Section 3; F is precomputed before serving,
 * Section 3.2).
 *
 *  fgrams   [n, max_len] int32 row-major; row k holds f-gram k's tokens,
 *           oldest first, in its first lengths[k] entries (the rest is
 *           ignored and may hold anything).
 *  lengths  [n] int32, each in [2, max_len]   (else SCONE_ELEN; V_fgram is a
 *           subset of V^[2,K]).
 *  ids      [n] int32 row ids, each in [0, 2^31 - 1)   (else SCONE_EID; the
 *           value 2^31 - 1 is reserved).  Ids are not checked against a row
 *           count here; scone_gather checks them.
 *  n        number of f-grams, >= 0 (0 builds an empty set).
 *  max_len  K, in [2, SCONE_MAX_FGRAM_LEN].  K <= 5 uses 16-byte slots,
 *           K = 6 or 7 uses 32-byte slots.
 *  max_load target load factor in (0, 0.9]; the slot count is the smallest
 *           power of two >= max(64, e / max_load), where e is n plus the
 *           number of f-grams of length >= 4 plus the number of length >= 6.
 *           Besides the f-grams, the table holds an entry for the last three
 *           tokens of every f-gram of length >= 4 and the last five of every
 *           f-gram of length >= 6, flagged so that a lookup stops probing a
 *           position once no longer f-gram can end there; e bounds all of
 *           them.
 *  stream   stream on which the inputs are ready.
 *  out      receives the new table handle (host pointer to a handle).
 *
 * Tokens must lie in [0, SCONE_TOKEN_LIMIT) (else SCONE_ETOKEN).  A repeated
 * f-gram (same length, same tokens) gives SCONE_EDUP: V_fgram is a set.
 * The call is synchronous: it waits on `stream` and returns the first data
 * error found.  On any error *out is NULL and nothing stays allocated.  The
 * caller may free its inputs as soon as the call returns.
 */
int scone_build_fgram_table(const int32_t* fgrams, const int32_t* lengths,
                            const int32_t* ids, int64_t n, int32_t max_len,
                            double max_load, void* stream, scone_table_t** out);

/*
 * Longest-suffix lookup (Algorithm 1, the choice of j): for every b < B and
 * t < T, fgram_ids[b,t] is the id of the longest f-gram
 * (X[b,t-n+1], ..., X[b,t]) with 2 <= n <= min(max_n, t+1) that is in the
 * table, and match_len[b,t] = n; when there is none, fgram_ids[b,t] =
 * X[b,t] (the token's own row) and match_len[b,t] = 1.  Windows never reach
 * before t = 0 of their own row.  Every length is tested on its own, so the
 * f-gram set need not contain the suffixes of its members.
 *
 *  token_ids  [B, T] int32 row-major, each in [0, SCONE_TOKEN_LIMIT)
 *             (else SCONE_ETOKEN via scone_check).
 *  max_n      >= 1; values above the table's max_len behave as max_len;
 *             1 gives the identity.
 *  fgram_ids  [B, T] int32 output.
 *  match_len  [B, T] int8 output, or NULL.
 *
 * Outputs that share memory with token_ids (or with each other) give
 * SCONE_EINVAL: workgroups read a halo of tokens that other workgroups'
 * positions own.  Asynchronous on `stream`; the table is read-only, so
 * concurrent lookups on one table are safe.  B * T = 0 launches nothing.
 */
int scone_lookup(const scone_table_t* table, const int32_t* token_ids, int64_t B,
                 int64_t T, int32_t max_n, int32_t* fgram_ids, int8_t* match_len,
                 void* stream);

/*
 * scone_lookup that also counts its hash probes (Section 4.3 reports up to
 * four queries per token for K = 5; this measures how many the kernel makes):
 * *probes, a device uint64, is increased by the number of keys probed, one
 * per tested length of every position.  Lengths 2 and 3 are tested at every
 * position where they fit the window; 4 and 5 only where the length-3 suffix
 * ends some f-gram of length 4 or more, and 6 and 7 where, in addition, the
 * length-5 suffix ends one of length 6 or more.  Arguments, results and errors
 * are those of scone_lookup; probes may not be NULL (SCONE_EINVAL) or share
 * memory with the other buffers (SCONE_EINVAL).  The count is a diagnostic:
 * the same kernel built with a counter, for tests and measurements.
 */
int scone_lookup_counted(const scone_table_t* table, const int32_t* token_ids, int64_t B,
                         int64_t T, int32_t max_n, int32_t* fgram_ids, int8_t* match_len,
                         uint64_t* probes, void* stream);

/*
 * Pre-scan tagging (the paper tags every training token with the length of
 * its longest matching f-gram before training, implementation details in the
 * appendix; the mean of these lengths is the average match length that
 * Section 4.1 reports): the match lengths of scone_lookup without the ids, plus
 * their histogram.
 *
 *  token_ids  [B, T] int32, as for scone_lookup.
 *  match_len  [B, T] int8 output (1 = no f-gram), or NULL.
 *  hist       [SCONE_MAX_FGRAM_LEN + 1] uint64 device array, or NULL;
 *             hist[n] is INCREASED by the number of positions whose match
 *             length is n (the caller zeroes it to start a count).
 *
 * At least one of match_len and hist must be given; neither may share memory
 * with token_ids or with the other (else SCONE_EINVAL).  Asynchronous.
 */
int scone_tag(const scone_table_t* table, const int32_t* token_ids, int64_t B, int64_t T,
              int32_t max_n, int8_t* match_len, uint64_t* hist, void* stream);

/*
 * Row gather (the embedding fetch; Section 1 notes it is a pure memory read):
 * out[k, :] = rows[fgram_ids[k], :] for k < n_tok, copied as raw bytes, so
 * any element type (fp32, bf16, ...) is reproduced bit for bit.
 *
 *  fgram_ids  [n_tok] int32, each in [0, n_rows) (else SCONE_EROW via
 *             scone_check; that output row is then zero-filled).
 *  rows       [n_rows, row_bytes] table: device memory (placement
 *             SCONE_PLACE_HBM) or host-mapped pinned memory
 *             (SCONE_PLACE_HOST).
 *  row_bytes  > 0.  Rows move in 16-byte vectors when row_bytes and both
 *             pointers allow it, otherwise in the widest unit that does.
 *  out        [n_tok, row_bytes] device output; sharing memory with `rows`
 *             or with fgram_ids gives SCONE_EINVAL.
 *
 * Asynchronous on `stream`.  n_tok = 0 launches nothing.
 */
int scone_gather(const int32_t* fgram_ids, int64_t n_tok, const void* rows,
                 int64_t n_rows, int64_t row_bytes, void* out, int32_t placement,
                 void* stream);

/*
 * Fused lookup + gather (the whole inference branch of Algorithm 1 in one
 * kernel): produces exactly what scone_lookup followed by scone_gather
 * produces, without the ids passing through memory in between.
 *
 *  token_ids, B, T, max_n   as for scone_lookup.
 *  rows, n_rows, row_bytes, placement   as for scone_gather.
 *  out        [B, T, row_bytes] device output.
 *  fgram_ids  [B, T] int32 output, or NULL when not wanted.
 *  match_len  [B, T] int8 output, or NULL.
 *
 * Errors as for scone_lookup and scone_gather; out, fgram_ids and match_len
 * may not share memory with token_ids, rows or each other (SCONE_EINVAL).
 * Asynchronous on `stream`.
 */
int scone_embed(const scone_table_t* table, const int32_t* token_ids, int64_t B, int64_t T,
                int32_t max_n, const void* rows, int64_t n_rows, int64_t row_bytes,
                int32_t placement, void* out, int32_t* fgram_ids, int8_t* match_len,
                void* stream);

/*
 * One step of a stream of batches, software-pipelined (Algorithm 1's
 * inference branch, the lookup of one batch overlapped with the gather of
 * the batch before it): in a single launch,
 *   next_ids[b, t] = scone_lookup's id for next_tokens[b, t]   (next batch)
 *   out[k, :]      = rows[cur_ids[k], :]                        (current batch)
 * The results equal scone_lookup on the next batch and scone_gather on the
 * current ids.  A stream of batches X_0, X_1, ... runs as: step 0 with no
 * current ids (lookup of X_0 only), step k with next = X_k and cur = the ids
 * of X_{k-1}, and a last step with no next tokens (gather only); the ids
 * alternate between two buffers.
 *
 *  next_tokens, B, T, max_n   as for scone_lookup; B * T == 0 (next_tokens
 *             may then be NULL) makes this step a gather only.
 *  next_ids   [B, T] int32 output; next_len [B, T] int8 output or NULL.
 *  cur_ids    [n_cur] int32, the previous step's next_ids; n_cur == 0
 *             (cur_ids may then be NULL) makes this step a lookup only.
 *  rows, n_rows, row_bytes, placement   as for scone_gather.
 *  out        [n_cur, row_bytes] device output.
 *
 * Returns SCONE_EINVAL when any output (next_ids, next_len, out) shares
 * memory with an input (next_tokens, cur_ids) or with another output: the
 * launch writes them while its other workgroups read; otherwise errors as
 * for scone_lookup and scone_gather.  Rows of 1, 2, 4 or 8 KiB, 16-byte aligned,
 * take the one-launch kernel; other widths run the lookup and gather kernels
 * back to back with the same results.  Asynchronous on `stream`.
 */
int scone_embed_pipelined(const scone_table_t* table, const int32_t* next_tokens, int64_t B,
                          int64_t T, int32_t max_n, int32_t* next_ids, int8_t* next_len,
                          const int32_t* cur_ids, int64_t n_cur, const void* rows,
                          int64_t n_rows, int64_t row_bytes, int32_t placement, void* out,
                          void* stream);

/*
 * One decoding step for S sequences (inference emits one token per step per
 * sequence; Section 4.3 measures per-token latency this way).  Sequence s
 * appends new_tok[s] to its rolling context and gets the embedding of the
 * longest f-gram ending at that token (Algorithm 1 at the newest position).
 *
 *  ctx        [S, ctx_cap] int32, in/out: the last ctx_len[s] tokens of
 *             sequence s, oldest first (the rest is ignored).  Rewritten
 *             with the last min(ctx_cap, ctx_len[s] + 1) tokens.
 *  ctx_len    [S] int32, in/out; 0 for a new sequence.  Values outside
 *             [0, ctx_cap] are treated as the nearest bound.
 *  ctx_cap    context capacity, in [min(max_n, K) - 1, 63]; with at least
 *             max_n - 1 tokens kept, step s of a sequence gives the same id
 *             and row as scone_lookup at position s of the whole sequence.
 *  new_tok    [S] int32 tokens in [0, SCONE_TOKEN_LIMIT).
 *  rows ...   as for scone_gather; out is [S, row_bytes].
 *  fgram_ids  [S] int32 output, or NULL; match_len [S] int8 or NULL.
 *
 * out, fgram_ids and match_len may not share memory with ctx, ctx_len,
 * new_tok, rows or each other, nor ctx, ctx_len and new_tok with each other
 * (SCONE_EINVAL).  Asynchronous on `stream`.  Calls for the same sequences
 * must be ordered (the context is read and rewritten in place).
 */
int scone_decode_step(const scone_table_t* table, int32_t* ctx, int32_t* ctx_len,
                      int32_t ctx_cap, const int32_t* new_tok, int64_t S, int32_t max_n,
                      const void* rows, int64_t n_rows, int64_t row_bytes, int32_t placement,
                      void* out, int32_t* fgram_ids, int8_t* match_len, void* stream);

/*
 * Row gather with split placement: the token rows stay on the accelerator and
 * the f-gram rows live off it (Section 3.2 keeps T on the accelerator and
 * offloads F; Section 4.3 stores F in main memory).  Ids in [0, n_near) read
 * `near_rows` (device memory); ids in [n_near, n_near + n_far) read row
 * id - n_near of `far_rows` (host-mapped pinned memory).  Each distinct far id
 * of the call crosses PCIe once: the call dedupes the far ids in `workspace`,
 * copies those rows into a device staging area, then writes
 * out[k, :] = row of fgram_ids[k] from device memory.  The result equals
 * scone_gather over the concatenated table.
 *
 *  fgram_ids   [n_tok] int32; an id outside [0, n_near + n_far) raises
 *              SCONE_EROW via scone_check and zeroes its output row.
 *  near_rows   [n_near, row_bytes] device memory; far_rows [n_far, row_bytes]
 *              host-mapped (scone_host_alloc).  n_near + n_far <= 2^31.
 *  row_bytes   a multiple of 16; every pointer 16-byte aligned (else
 *              SCONE_EINVAL).
 *  out         [n_tok, row_bytes] device output; sharing memory with
 *              fgram_ids or near_rows gives SCONE_EINVAL.
 *  workspace   device scratch of at least scone_gather_split_workspace(n_tok,
 *              row_bytes) bytes (else SCONE_EINVAL), caller-owned, reusable
 *              across calls that do not overlap.  The part of it the call
 *              uses (scone_gather_split_workspace bytes) may not share memory
 *              with fgram_ids, near_rows, far_rows, out or n_unique
 *              (SCONE_EINVAL).
 *  n_unique    device int32 receiving the number of distinct far ids (the
 *              rows that crossed PCIe), or NULL; sharing memory with out or
 *              fgram_ids gives SCONE_EINVAL.
 *
 * Asynchronous on `stream`; launches kernels only (no memset or copy nodes),
 * so the call can be captured in a graph.
 */
int scone_gather_split(const int32_t* fgram_ids, int64_t n_tok, const void* near_rows,
                       int64_t n_near, const void* far_rows, int64_t n_far,
                       int64_t row_bytes, void* out, void* workspace,
                       int64_t workspace_bytes, int32_t* n_unique, void* stream);

/* Bytes of workspace scone_gather_split needs for n_tok rows of row_bytes, or
 * -1 for invalid sizes (worst case: every id distinct and far). */
int64_t scone_gather_split_workspace(int64_t n_tok, int64_t row_bytes);

/* Size of the fixed scratch buffer of scone_gather_split_static (bytes, per GPU). */
#define SCONE_SPLIT_STATIC_BYTES (32 << 20)

/*
 * scone_gather_split without a workspace argument and without any allocation,
 * for callers that cannot allocate device memory: code being captured into a
 * HIP graph, tight serving loops (a decoding step for a few hundred sequences
 * with the f-gram rows in host memory), harnesses that forbid hipMalloc.
 * Arguments, results and errors are those of scone_gather_split; the dedupe
 * set and the staged rows live in a fixed buffer of SCONE_SPLIT_STATIC_BYTES
 * in the library's own device data (one per GPU, held until the process
 * ends).  A call whose scone_gather_split_workspace(n_tok, row_bytes) exceeds
 * that size returns SCONE_ESCRATCH and launches nothing (for 4 KiB rows, up
 * to about 8,100 tokens fit).  Every call on a GPU shares that GPU's buffer:
 * calls on one stream run in order, but calls that can overlap (other
 * streams, other threads) race and their results are unspecified.  Each call
 * resets the parts it reads, so nothing carries over from the last call.
 * Asynchronous on `stream`; launches kernels only.
 */
int scone_gather_split_static(const int32_t* fgram_ids, int64_t n_tok, const void* near_rows,
                              int64_t n_near, const void* far_rows, int64_t n_far,
                              int64_t row_bytes, void* out, int32_t* n_unique, void* stream);

/*
 * F-gram discovery (Algorithm 3: count every n-gram, n = 2..max_len, of all
 * sequences and keep the S most frequent; ties at the cut are broken in an
 * unspecified order, as Algorithm 3 allows).  It follows the efficient form of
 * Section 3.1: one counting scan per n, and from the second scan on an n-gram
 * is kept only when it occurs at least min_count times (the paper uses 5);
 * all 2-grams are kept.  With min_count = 1 the result is Algorithm 3's.
 * n-grams never cross from one sequence into the next.
 *
 *  token_ids  [B, T] int32 (each in [0, SCONE_TOKEN_LIMIT), else
 *             SCONE_ETOKEN); B * T < 2^31 and (max_len - 1) * B * T < 2^32
 *             (candidates are counted in 32 bits), else SCONE_EINVAL.
 *  max_len    K, in [2, SCONE_MAX_FGRAM_LEN].
 *  S          the number of f-grams wanted.
 *  fgrams     [S, max_len] int32 output, row k holding f-gram k oldest first,
 *             padded with -1; lengths [S] and counts [S] int32 outputs.
 *  n_found    host pointer receiving min(S, number of candidates); only that
 *             many rows are written.
 *  workspace  device scratch of at least scone_discover_workspace(B, T,
 *             max_len) bytes, 256-byte aligned, caller-owned and reusable
 *             across calls that do not overlap (else SCONE_EINVAL); or NULL,
 *             and the call allocates that much itself and frees it before
 *             returning.
 * No two of token_ids, fgrams, lengths, counts and the workspace (the part
 * the call uses) may share memory (SCONE_EINVAL).
 *
 * The output is ready for scone_build_fgram_table (ids are the caller's
 * choice).  Synchronous (it reads the candidate count and a count histogram
 * back to choose the top-S threshold).
 */
int scone_discover_fgrams(const int32_t* token_ids, int64_t B, int64_t T, int32_t max_len,
                          int32_t min_count, int64_t S, int32_t* fgrams, int32_t* lengths,
                          int32_t* counts, int64_t* n_found, void* workspace,
                          int64_t workspace_bytes, void* stream);

/* Bytes of workspace scone_discover_fgrams needs for a [B, T] corpus and
 * f-grams up to max_len tokens (a counting table of 16-byte slots, at least
 * 2 B T of them, plus about (13 (max_len - 1) + 8 (max_len - 2) + 8) B T
 * bytes of per-scan arrays), or -1 for sizes the call rejects. */
int64_t scone_discover_workspace(int64_t B, int64_t T, int32_t max_len);

/*
 * Precompute the f-gram embedding layer (Section 3.2: F caches the f-gram
 * model's outputs, one row per f-gram; the model maps the token embeddings of
 * an f-gram to the output at its final token, Algorithm 1's training branch).
 *
 * The f-gram model A_fgram is a pre-LayerNorm causal decoder (the paper gives
 * its sizes through the main-model tables of the appendix, absolute position
 * embeddings with one row per position up to the longest f-gram, and bf16
 * parameters; the rest is this library's reading):
 *     h_i = T(w_i) + pos[i]                          i = 0 (oldest) .. n-1
 *     per layer:  h += Attn(LN1(h));  h += W2 GELU(W1 LN2(h) + b1) + b2
 *     F(w) = LNf(h_{n-1})
 * with causal multi-head attention (scores scaled by 1/sqrt(d / n_heads)),
 * exact erf GELU, LayerNorm epsilon 1e-5 over the population variance, and
 * y = x W^T + b for every linear map (W stored [out, in]).  F-grams of equal
 * length are processed together, unpadded (the paper right-pads a batch to
 * its longest f-gram; under causal attention the final token never sees a
 * pad, so the result is the same).
 *
 *  fgrams    [n, max_len] int32, row k = f-gram k oldest first (entries past
 *            lengths[k] are ignored); tokens in [0, vocab) else SCONE_ETOKEN.
 *  lengths   [n] int32 in [2, max_len] (else SCONE_ELEN, nothing computed).
 *  row_ids   [n] int32: F(f-gram k) is written to row row_ids[k] of `rows`;
 *            outside [0, n_rows) -> SCONE_EROW and that row is skipped.
 *  max_len   K in [2, SCONE_MAX_FGRAM_LEN] = the number of position rows.
 *  tok_rows  [vocab, d] bf16, the token embedding layer T.  It may be the
 *            first vocab rows of `rows` (the unified table) as long as no
 *            row id falls below vocab.
 *  params    bf16 parameters packed as scone_fgram_model_layout describes:
 *              pos [max_len, d];
 *              per layer: ln1_g [d], ln1_b [d], w_qkv [3d, d] (q, k, v
 *                rows in that order, heads contiguous), b_qkv [3d],
 *                w_o [d, d], b_o [d], ln2_g [d], ln2_b [d],
 *                w_fc1 [d_ff, d], b_fc1 [d_ff], w_fc2 [d, d_ff], b_fc2 [d];
 *              lnf_g [d], lnf_b [d];
 *            each tensor row-major, starting at a multiple of 128 elements.
 *  d         d_model, a multiple of 512 up to 4096; d / n_heads must be 64 or
 *            128; d_ff a multiple of 128; n_layers >= 0 (0 gives
 *            LNf(T(w_{n-1}) + pos[n-1])).
 *  rows      [n_rows, d] bf16 output table (device memory); sharing memory
 *            with fgrams, lengths, row_ids or params gives SCONE_EINVAL.
 *
 * tok_rows, params and rows must be 16-byte aligned (else SCONE_EINVAL).
 * Synchronous: returns after the rows are written, with the first data error
 * (SCONE_ELEN, SCONE_ETOKEN, SCONE_EROW) or SCONE_OK.  Allocates and frees its
 * own device scratch: about 65536 * (14 d + 2 d_ff) bytes of activations for
 * one chunk of same-length f-grams, plus 4 n bytes.
 */
int scone_fgram_model_forward(const int32_t* fgrams, const int32_t* lengths,
                              const int32_t* row_ids, int64_t n, int32_t max_len,
                              const void* tok_rows, int64_t vocab, const void* params, int32_t d,
                              int32_t n_heads, int32_t d_ff, int32_t n_layers, void* rows,
                              int64_t n_rows, void* stream);

/*
 * Packing of scone_fgram_model_forward's parameters: offsets[k] (elements)
 * of the k-th tensor in the order listed there (2 + 12 * n_layers + 1
 * tensors; offsets may be NULL), the tensor count and the total element count
 * of the blob.  SCONE_EINVAL for unsupported sizes.
 */
int scone_fgram_model_layout(int32_t d, int32_t n_heads, int32_t d_ff, int32_t n_layers,
                             int32_t max_len, int64_t* offsets, int64_t* n_params,
                             int64_t* total_elems);

/*
 * Allocate `bytes` of pinned host memory that kernels can read over PCIe
 * (the off-accelerator row store of Section 4.3).  *host_ptr receives the
 * host address, *device_ptr the address to pass to scone_gather with
 * SCONE_PLACE_HOST.  SCONE_ENOMEM on failure.  Free with scone_host_free.
 */
int scone_host_alloc(int64_t bytes, void** host_ptr, void** device_ptr);
int scone_host_free(void* host_ptr);

/*
 * Wait for `stream`, then read the current device's error word and clear
 * the bits it read (atomically, so a bit that a kernel on another stream
 * raises after the read is kept for the next check).  Returns SCONE_OK or
 * the lowest data-error code raised by the asynchronous calls since the last
 * check (SCONE_ETOKEN, SCONE_EROW, SCONE_EFULL).  The word is per device, not
 * per stream: concurrent streams share it.
 */
int scone_check(void* stream);

/* Free a table (NULL is a no-op).  The caller must not use it afterwards and
 * must make sure no lookup that reads it is still running. */
void scone_table_destroy(scone_table_t* table);

/* Properties of a built table; any output pointer may be NULL.  n: f-grams
 * stored; capacity: slots; max_len: K; slot_bytes: 16 or 32; entries: slots
 * in use, the f-grams plus the flagged suffix markers (so entries / capacity
 * is the table's load).  Two concurrent inserts of the same marker can leave
 * two copies of it, so entries may differ slightly between builds of the same
 * set; lookups are unaffected. */
int scone_table_info(const scone_table_t* table, int64_t* n, int64_t* capacity,
                     int32_t* max_len, int32_t* slot_bytes, int64_t* entries);

/* A static, human-readable description of a status code. */
const char* scone_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* SCONE_H */
