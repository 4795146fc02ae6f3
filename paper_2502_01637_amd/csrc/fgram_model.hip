// Precomputing the f-gram embedding layer: F(w) = A_fgram(T(w_0..w_{n-1})),
// the f-gram model's output at the last token, for every f-gram w (Section
// 3.2; Algorithm 1's training branch is the same map).  The model is a
// pre-LayerNorm causal decoder with absolute position embeddings of one row
// per position up to the longest f-gram (implementation appendix), biases on
// every linear map, exact GELU, LayerNorm epsilon 1e-5, and a final LayerNorm.
//
// The paper pads the f-grams of a batch to the longest one.  Here the f-grams
// are bucketed by length instead (a counting sort on the device) and each
// bucket runs unpadded: with causal attention and right padding the last
// token never sees a pad position, so the result is the same and no work is
// spent on pads.  A chunk holds up to kChunkTokens tokens of one length, laid
// out f-gram-major (token i of the chunk's f-gram g is row g * n + i):
//
//   k_embed_ln   h = T[w_i] + P[i] (f32),  a = LN1_0(h) (bf16)
//   per layer:   [k_ln a = LN1(h)]  qkv = a Wqkv^T + b       (MFMA)
//                o = causal attention(qkv)                    (k_attn)
//                h += o Wo^T + b                              (MFMA, fused residual)
//                a = LN2(h);  f = GELU(a W1^T + b1)           (MFMA, fused GELU)
//                h += f W2^T + b2                             (MFMA, fused residual)
//   k_final      rows[row_id] = bf16(LNf(h at the last token))
//
// Matrix products run on the matrix cores (gemm_bf16.h); the rest is
// bandwidth-bound and one wavefront handles one row or one f-gram.
#include "gemm_bf16.h"

#include <algorithm>
#include <vector>

namespace scone {
namespace {

using gemm::bf16_to_f32;
using gemm::f32_to_bf16;

constexpr int kThreads = 256;
constexpr int64_t kChunkTokens = 65536;
constexpr float kLnEps = 1e-5f;

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// ---------------------------------------------------------------- sorting --

// Length histogram (counts[0..7]); lengths outside [2, max_len] raise ELEN.
// Counts are summed per workgroup in LDS first, so each workgroup adds at
// most one value per length to the global counters.
__global__ __launch_bounds__(kThreads) void k_len_count(const int32_t* __restrict__ lengths,
                                                        int64_t n, int max_len,
                                                        unsigned* __restrict__ counts,
                                                        unsigned* __restrict__ status) {
    __shared__ unsigned s_cnt[8];
    if (threadIdx.x < 8) s_cnt[threadIdx.x] = 0;
    __syncthreads();
    const int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (g < n) {
        const int32_t L = lengths[g];
        if (L < 2 || L > max_len)
            atomicOr(status, err_bit(SCONE_ELEN));
        else
            atomicAdd(s_cnt + L, 1u);
    }
    __syncthreads();
    if (threadIdx.x < 8 && s_cnt[threadIdx.x]) atomicAdd(counts + threadIdx.x, s_cnt[threadIdx.x]);
}

// order[base[L] + k] = g for the f-grams of length L (any order inside a
// bucket).  A workgroup ranks its f-grams per length in LDS and reserves each
// length's run with one global atomic.
__global__ __launch_bounds__(kThreads) void k_len_scatter(const int32_t* __restrict__ lengths,
                                                          int64_t n, int max_len,
                                                          const int64_t* __restrict__ base,
                                                          unsigned* __restrict__ cursor,
                                                          int32_t* __restrict__ order) {
    __shared__ unsigned s_cnt[8], s_off[8];
    if (threadIdx.x < 8) s_cnt[threadIdx.x] = 0;
    __syncthreads();
    const int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    int32_t L = 0;
    unsigned rank = 0;
    if (g < n) {
        L = lengths[g];
        if (L >= 2 && L <= max_len) rank = atomicAdd(s_cnt + L, 1u);
        else L = 0;
    }
    __syncthreads();
    if (threadIdx.x < 8 && s_cnt[threadIdx.x])
        s_off[threadIdx.x] = atomicAdd(cursor + threadIdx.x, s_cnt[threadIdx.x]);
    __syncthreads();
    if (L) order[base[L] + s_off[L] + rank] = (int32_t)g;
}

// -------------------------------------------------------------- row kernels --
// One wavefront per row of d = 256 * R elements; lane holds elements
// c * 256 + lane * 4 + (0..3), c < R.

template <int R>
__device__ __forceinline__ void layer_norm_store(float (&x)[R][4], const uint16_t* __restrict__ g,
                                                 const uint16_t* __restrict__ b, int lane,
                                                 uint16_t* __restrict__ dst) {
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < R; ++c) s += (x[c][0] + x[c][1]) + (x[c][2] + x[c][3]);
    const float mean = wave_sum(s) * (1.0f / (256 * R));
    float q = 0.f;
#pragma unroll
    for (int c = 0; c < R; ++c)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float t = x[c][e] - mean;
            q += t * t;
        }
    const float rstd = rsqrtf(wave_sum(q) * (1.0f / (256 * R)) + kLnEps);
#pragma unroll
    for (int c = 0; c < R; ++c) {
        const int e0 = c * 256 + lane * 4;
        const u32x2 gg = *reinterpret_cast<const u32x2*>(g + e0);
        const u32x2 bb = *reinterpret_cast<const u32x2*>(b + e0);
        const float gv[4] = {bf16_to_f32(gg.x & 0xFFFFu), bf16_to_f32(gg.x >> 16),
                             bf16_to_f32(gg.y & 0xFFFFu), bf16_to_f32(gg.y >> 16)};
        const float bv[4] = {bf16_to_f32(bb.x & 0xFFFFu), bf16_to_f32(bb.x >> 16),
                             bf16_to_f32(bb.y & 0xFFFFu), bf16_to_f32(bb.y >> 16)};
        uint32_t o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = f32_to_bf16((x[c][e] - mean) * rstd * gv[e] + bv[e]);
        *reinterpret_cast<u32x2*>(dst + e0) = u32x2{o[0] | (o[1] << 16), o[2] | (o[3] << 16)};
    }
}

// h[r] = T[token] + P[pos]; a[r] = LN(h[r]).  Tokens outside [0, vocab) raise
// ETOKEN and use row 0.
template <int R>
__global__ __launch_bounds__(kThreads) void k_embed_ln(
    const int32_t* __restrict__ order, int64_t n_f, int n, const int32_t* __restrict__ fgrams,
    int max_len, const uint16_t* __restrict__ tok_rows, int64_t vocab,
    const uint16_t* __restrict__ pos, const uint16_t* __restrict__ g,
    const uint16_t* __restrict__ b, float* __restrict__ h, uint16_t* __restrict__ a,
    unsigned* __restrict__ status) {
    constexpr int d = 256 * R;
    const int64_t r = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (r >= n_f * n) return;
    const int lane = threadIdx.x & 63;
    const int64_t f = r / n;
    const int i = (int)(r - f * n);
    int32_t tok = fgrams[(int64_t)order[f] * max_len + i];
    if (tok < 0 || tok >= vocab) {
        if (lane == 0) atomicOr(status, err_bit(SCONE_ETOKEN));
        tok = 0;
    }
    const uint16_t* trow = tok_rows + (int64_t)tok * d;
    const uint16_t* prow = pos + (int64_t)i * d;
    float x[R][4];
#pragma unroll
    for (int c = 0; c < R; ++c) {
        const int e0 = c * 256 + lane * 4;
        const u32x2 tv = *reinterpret_cast<const u32x2*>(trow + e0);
        const u32x2 pv = *reinterpret_cast<const u32x2*>(prow + e0);
        x[c][0] = bf16_to_f32(tv.x & 0xFFFFu) + bf16_to_f32(pv.x & 0xFFFFu);
        x[c][1] = bf16_to_f32(tv.x >> 16) + bf16_to_f32(pv.x >> 16);
        x[c][2] = bf16_to_f32(tv.y & 0xFFFFu) + bf16_to_f32(pv.y & 0xFFFFu);
        x[c][3] = bf16_to_f32(tv.y >> 16) + bf16_to_f32(pv.y >> 16);
        *reinterpret_cast<float4*>(h + r * d + e0) =
            make_float4(x[c][0], x[c][1], x[c][2], x[c][3]);
    }
    layer_norm_store<R>(x, g, b, lane, a + r * d);
}

// a[r] = LN(h + r * ld) for r < rows (ld = d, or n * d to take every f-gram's
// last token from h + (n - 1) * d).
template <int R>
__global__ __launch_bounds__(kThreads) void k_ln(const float* __restrict__ h, int64_t rows,
                                                 int64_t ld, const uint16_t* __restrict__ g,
                                                 const uint16_t* __restrict__ b,
                                                 uint16_t* __restrict__ a) {
    constexpr int d = 256 * R;
    const int64_t r = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (r >= rows) return;
    const int lane = threadIdx.x & 63;
    float x[R][4];
#pragma unroll
    for (int c = 0; c < R; ++c) {
        const float4 v = *reinterpret_cast<const float4*>(h + r * ld + c * 256 + lane * 4);
        x[c][0] = v.x; x[c][1] = v.y; x[c][2] = v.z; x[c][3] = v.w;
    }
    layer_norm_store<R>(x, g, b, lane, a + r * d);
}

// rows[row_id] = bf16(LNf(h at the f-gram's last token)).  Row ids outside
// [0, n_rows) raise EROW and write nothing.
template <int R>
__global__ __launch_bounds__(kThreads) void k_final(const float* __restrict__ h,
                                                    const int32_t* __restrict__ order,
                                                    int64_t n_f, int n,
                                                    const int32_t* __restrict__ row_ids,
                                                    const uint16_t* __restrict__ g,
                                                    const uint16_t* __restrict__ b,
                                                    uint16_t* __restrict__ rows, int64_t n_rows,
                                                    unsigned* __restrict__ status) {
    constexpr int d = 256 * R;
    const int64_t f = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (f >= n_f) return;
    const int lane = threadIdx.x & 63;
    const int32_t id = row_ids[order[f]];
    if (id < 0 || id >= n_rows) {
        if (lane == 0) atomicOr(status, err_bit(SCONE_EROW));
        return;
    }
    const float* src = h + (f * n + n - 1) * d;
    float x[R][4];
#pragma unroll
    for (int c = 0; c < R; ++c) {
        const float4 v = *reinterpret_cast<const float4*>(src + c * 256 + lane * 4);
        x[c][0] = v.x; x[c][1] = v.y; x[c][2] = v.z; x[c][3] = v.w;
    }
    layer_norm_store<R>(x, g, b, lane, rows + (int64_t)id * d);
}

// ---------------------------------------------------------------- attention --
// One wavefront per f-gram of n tokens.  A pass covers 512 columns of the
// model: lane holds 8 consecutive columns, so a head of dh columns spans
// dh / 8 lanes and its dot products are reduced over that many lanes.
// qkv row r = [q | k | v], each d wide; o row r = concatenated heads.
// kLast: only the last position's output, written to o row f (the last
// layer needs nothing else).
template <int LPH, int N, bool kLast>  // lanes per head (dh / 8), f-gram length
__global__ __launch_bounds__(kThreads) void k_attn(const uint16_t* __restrict__ qkv,
                                                   uint16_t* __restrict__ o, int64_t n_f, int d,
                                                   float scale) {
    const int64_t f = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (f >= n_f) return;
    const int lane = threadIdx.x & 63;
    const int64_t r0 = f * N;
    const int64_t ld = 3 * (int64_t)d;
    for (int c0 = 0; c0 < d; c0 += 512) {
        const int col = c0 + lane * 8;
        u32x4 qq[N], kk[N], vv[N];
#pragma unroll
        for (int j = 0; j < N; ++j) {
            const uint16_t* row = qkv + (r0 + j) * ld + col;
            qq[j] = *reinterpret_cast<const u32x4*>(row);
            kk[j] = *reinterpret_cast<const u32x4*>(row + d);
            vv[j] = *reinterpret_cast<const u32x4*>(row + 2 * d);
        }
#pragma unroll
        for (int i = kLast ? N - 1 : 0; i < N; ++i) {
            float s[N];
            float mx = -3.0e38f;
#pragma unroll
            for (int j = 0; j <= i; ++j) {
                float t = 0.f;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    t += bf16_to_f32(qq[i][e] & 0xFFFFu) * bf16_to_f32(kk[j][e] & 0xFFFFu);
                    t += bf16_to_f32(qq[i][e] >> 16) * bf16_to_f32(kk[j][e] >> 16);
                }
#pragma unroll
                for (int w = LPH / 2; w >= 1; w >>= 1) t += __shfl_xor(t, w);
                s[j] = t * scale;
                mx = fmaxf(mx, s[j]);
            }
            float den = 0.f;
#pragma unroll
            for (int j = 0; j <= i; ++j) {
                s[j] = __expf(s[j] - mx);
                den += s[j];
            }
            const float inv = 1.0f / den;
            float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int j = 0; j <= i; ++j) {
                const float p = s[j] * inv;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc[2 * e] += p * bf16_to_f32(vv[j][e] & 0xFFFFu);
                    acc[2 * e + 1] += p * bf16_to_f32(vv[j][e] >> 16);
                }
            }
            u32x4 ov;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                ov[e] = f32_to_bf16(acc[2 * e]) | (f32_to_bf16(acc[2 * e + 1]) << 16);
            *reinterpret_cast<u32x4*>(o + (kLast ? f : r0 + i) * (int64_t)d + col) = ov;
        }
    }
}

template <int LPH, bool kLast>
hipError_t launch_attn(const uint16_t* qkv, uint16_t* o, int64_t n_f, int n, int d, float scale,
                       hipStream_t st) {
    const dim3 grid((unsigned)((n_f + 3) / 4)), block(kThreads);
    switch (n) {
#define SCONE_ATTN_CASE(NN)                                                                  \
    case NN:                                                                                 \
        hipLaunchKernelGGL((k_attn<LPH, NN, kLast>), grid, block, 0, st, qkv, o, n_f, d, scale); \
        break;
        SCONE_ATTN_CASE(2)
        SCONE_ATTN_CASE(3)
        SCONE_ATTN_CASE(4)
        SCONE_ATTN_CASE(5)
        SCONE_ATTN_CASE(6)
        SCONE_ATTN_CASE(7)
#undef SCONE_ATTN_CASE
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t attention(const uint16_t* qkv, uint16_t* o, int64_t n_f, int n, int d, int dh,
                     bool last, float scale, hipStream_t st) {
    if (dh == 64)
        return last ? launch_attn<8, true>(qkv, o, n_f, n, d, scale, st)
                    : launch_attn<8, false>(qkv, o, n_f, n, d, scale, st);
    return last ? launch_attn<16, true>(qkv, o, n_f, n, d, scale, st)
                : launch_attn<16, false>(qkv, o, n_f, n, d, scale, st);
}

// ------------------------------------------------------------------ layout --

constexpr int kPerLayer = 12;

int64_t align_up(int64_t x) { return (x + 127) & ~(int64_t)127; }

// Element counts of the parameters in packing order.
std::vector<int64_t> param_sizes(int64_t d, int64_t d_ff, int n_layers, int max_len) {
    std::vector<int64_t> s;
    s.push_back((int64_t)max_len * d);  // pos
    for (int l = 0; l < n_layers; ++l) {
        const int64_t per[kPerLayer] = {d,        d,    3 * d * d, 3 * d, d * d,    d,
                                        d,        d,    d_ff * d,  d_ff,  d * d_ff, d};
        for (int64_t v : per) s.push_back(v);
    }
    s.push_back(d);  // lnf_g
    s.push_back(d);  // lnf_b
    return s;
}

bool dims_ok(int32_t d, int32_t n_heads, int32_t d_ff, int32_t n_layers, int32_t max_len) {
    if (d <= 0 || d % 512 != 0 || d > 4096) return false;
    if (n_heads <= 0 || d % n_heads != 0) return false;
    const int dh = d / n_heads;
    if (dh != 64 && dh != 128) return false;
    if (d_ff <= 0 || d_ff % 128 != 0 || d_ff > 65536) return false;
    if (n_layers < 0 || n_layers > 1024) return false;
    if (max_len < 2 || max_len > SCONE_MAX_FGRAM_LEN) return false;
    return true;
}

struct Weights {
    const uint16_t* pos;
    struct Layer {
        const uint16_t *ln1_g, *ln1_b, *w_qkv, *b_qkv, *w_o, *b_o, *ln2_g, *ln2_b, *w_fc1,
            *b_fc1, *w_fc2, *b_fc2;
    };
    std::vector<Layer> layers;
    const uint16_t *lnf_g, *lnf_b;
};

Weights bind_weights(const uint16_t* blob, int64_t d, int64_t d_ff, int n_layers, int max_len) {
    const std::vector<int64_t> sz = param_sizes(d, d_ff, n_layers, max_len);
    std::vector<const uint16_t*> p;
    int64_t off = 0;
    for (int64_t s : sz) {
        p.push_back(blob + off);
        off += align_up(s);
    }
    Weights w;
    size_t k = 0;
    w.pos = p[k++];
    for (int l = 0; l < n_layers; ++l) {
        Weights::Layer L;
        L.ln1_g = p[k++]; L.ln1_b = p[k++]; L.w_qkv = p[k++]; L.b_qkv = p[k++];
        L.w_o = p[k++];   L.b_o = p[k++];   L.ln2_g = p[k++]; L.ln2_b = p[k++];
        L.w_fc1 = p[k++]; L.b_fc1 = p[k++]; L.w_fc2 = p[k++]; L.b_fc2 = p[k++];
        w.layers.push_back(L);
    }
    w.lnf_g = p[k++];
    w.lnf_b = p[k++];
    return w;
}

// ------------------------------------------------------------------ driver --

struct Buffers {
    float* h;
    uint16_t *a, *qkv, *f;
};

template <int R>
hipError_t run_chunk(const Weights& w, const int32_t* order, int64_t n_f, int n,
                     const int32_t* fgrams, int max_len, const uint16_t* tok_rows, int64_t vocab,
                     int d_ff, int n_heads, const int32_t* row_ids, uint16_t* rows,
                     int64_t n_rows, const Buffers& B, unsigned* status, hipStream_t st) {
    constexpr int d = 256 * R;
    const int64_t M = n_f * n;
    const unsigned g_rows = (unsigned)((M + 3) / 4);
    const unsigned g_f = (unsigned)((n_f + 3) / 4);
    const int n_layers = (int)w.layers.size();
    const uint16_t* ln_g = n_layers ? w.layers[0].ln1_g : w.lnf_g;
    const uint16_t* ln_b = n_layers ? w.layers[0].ln1_b : w.lnf_b;
    hipLaunchKernelGGL(k_embed_ln<R>, dim3(g_rows), dim3(kThreads), 0, st, order, n_f, n, fgrams,
                       max_len, tok_rows, vocab, w.pos, ln_g, ln_b, B.h, B.a, status);
    const int dh = d / n_heads;
    const float scale = 1.0f / sqrtf((float)dh);
    hipError_t e = hipGetLastError();
    for (int l = 0; l < n_layers && e == hipSuccess; ++l) {
        const Weights::Layer& L = w.layers[l];
        if (l > 0)
            hipLaunchKernelGGL(k_ln<R>, dim3(g_rows), dim3(kThreads), 0, st, B.h, M, (int64_t)d,
                               L.ln1_g, L.ln1_b, B.a);
        e = gemm::launch<gemm::kBias>(B.a, L.w_qkv, L.b_qkv, B.qkv, 3 * d, (int)M, 3 * d, d, st);
        if (e != hipSuccess) break;
        // Only the last token's state reaches F, so after the last layer's
        // attention every product runs on one row per f-gram: rows of h are
        // then taken with stride n * d from the last position.
        const bool last = l == n_layers - 1;
        const int64_t Mr = last ? n_f : M;
        float* hr = last ? B.h + (int64_t)(n - 1) * d : B.h;
        const int64_t ldh = last ? (int64_t)n * d : d;
        const unsigned g_r = (unsigned)((Mr + 3) / 4);
        // attention output overwrites a (its input to the qkv product is consumed)
        e = attention(B.qkv, B.a, n_f, n, d, dh, last, scale, st);
        if (e != hipSuccess) break;
        e = gemm::launch<gemm::kResid>(B.a, L.w_o, L.b_o, hr, ldh, (int)Mr, d, d, st);
        if (e != hipSuccess) break;
        hipLaunchKernelGGL(k_ln<R>, dim3(g_r), dim3(kThreads), 0, st, hr, Mr, ldh, L.ln2_g,
                           L.ln2_b, B.a);
        e = gemm::launch<gemm::kGelu>(B.a, L.w_fc1, L.b_fc1, B.f, d_ff, (int)Mr, d_ff, d, st);
        if (e != hipSuccess) break;
        e = gemm::launch<gemm::kResid>(B.f, L.w_fc2, L.b_fc2, hr, ldh, (int)Mr, d, d_ff, st);
    }
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_final<R>, dim3(g_f), dim3(kThreads), 0, st, B.h, order, n_f, n, row_ids,
                       w.lnf_g, w.lnf_b, rows, n_rows, status);
    return hipGetLastError();
}

typedef hipError_t (*ChunkFn)(const Weights&, const int32_t*, int64_t, int, const int32_t*, int,
                              const uint16_t*, int64_t, int, int, const int32_t*, uint16_t*,
                              int64_t, const Buffers&, unsigned*, hipStream_t);

ChunkFn chunk_fn(int d) {
    switch (d / 256) {
        case 2: return run_chunk<2>;
        case 4: return run_chunk<4>;
        case 6: return run_chunk<6>;
        case 8: return run_chunk<8>;
        case 10: return run_chunk<10>;
        case 12: return run_chunk<12>;
        case 14: return run_chunk<14>;
        case 16: return run_chunk<16>;
        default: return nullptr;
    }
}

}  // namespace
}  // namespace scone

extern "C" int scone_fgram_model_layout(int32_t d, int32_t n_heads, int32_t d_ff,
                                        int32_t n_layers, int32_t max_len, int64_t* offsets,
                                        int64_t* n_params, int64_t* total_elems) {
    using namespace scone;
    if (!dims_ok(d, n_heads, d_ff, n_layers, max_len)) return SCONE_EINVAL;
    const std::vector<int64_t> sz = param_sizes(d, d_ff, n_layers, max_len);
    int64_t off = 0;
    for (size_t k = 0; k < sz.size(); ++k) {
        if (offsets) offsets[k] = off;
        off += align_up(sz[k]);
    }
    if (n_params) *n_params = (int64_t)sz.size();
    if (total_elems) *total_elems = off;
    return SCONE_OK;
}

extern "C" int scone_fgram_model_forward(const int32_t* fgrams, const int32_t* lengths,
                                         const int32_t* row_ids, int64_t n, int32_t max_len,
                                         const void* tok_rows, int64_t vocab, const void* params,
                                         int32_t d, int32_t n_heads, int32_t d_ff,
                                         int32_t n_layers, void* rows, int64_t n_rows,
                                         void* stream) {
    using namespace scone;
    if (!dims_ok(d, n_heads, d_ff, n_layers, max_len)) return SCONE_EINVAL;
    if (n < 0 || vocab <= 0 || n_rows < 0 || n > 0x7fffffffLL) return SCONE_EINVAL;
    if (n == 0) return SCONE_OK;
    if (!fgrams || !lengths || !row_ids || !tok_rows || !params || !rows) return SCONE_EINVAL;
    if (((uintptr_t)tok_rows | (uintptr_t)params | (uintptr_t)rows) % 16 != 0)
        return SCONE_EINVAL;
    // Rows are written chunk by chunk while later chunks still read the
    // f-grams, lengths, row ids and parameters: `rows` may share memory with
    // none of them (tok_rows may lie inside it, as documented).
    {
        int64_t p_elems = 0;
        for (int64_t e : param_sizes(d, d_ff, n_layers, max_len)) p_elems += align_up(e);
        const int64_t rb = span_bytes(n_rows, 2 * (int64_t)d);
        if (overlaps(rows, rb, fgrams, span_bytes(n, 4 * (int64_t)max_len)) ||
            overlaps(rows, rb, lengths, span_bytes(n, 4)) ||
            overlaps(rows, rb, row_ids, span_bytes(n, 4)) ||
            overlaps(rows, rb, params, span_bytes(p_elems, 2)))
            return SCONE_EINVAL;
    }
    hipStream_t st = static_cast<hipStream_t>(stream);
    const ChunkFn fn = chunk_fn(d);
    if (!fn) return SCONE_EINVAL;

    // Control block (status, per-length counts and cursors, bucket bases) and
    // the bucket order first; the activations once the bucket sizes are known.
    const size_t ctl_bytes = 256;
    const size_t order_bytes = (size_t)align_up(4 * n);
    uint8_t* ctl = nullptr;
    if (hipMalloc(&ctl, ctl_bytes + order_bytes) != hipSuccess) return SCONE_ENOMEM;
    unsigned* status = reinterpret_cast<unsigned*>(ctl);       // [0]
    unsigned* counts = status + 8;                              // [8..15]
    unsigned* cursor = status + 16;                             // [16..23]
    int64_t* base = reinterpret_cast<int64_t*>(ctl + 128);      // [8]
    int32_t* order = reinterpret_cast<int32_t*>(ctl + ctl_bytes);
    uint8_t* act = nullptr;

    int rc = SCONE_OK;
    auto fail = [&](int code) {
        if (rc == SCONE_OK) rc = code;
    };
    unsigned hc[32] = {0};
    int64_t hbase[8] = {0};
    if (hipMemsetAsync(ctl, 0, ctl_bytes, st) != hipSuccess) fail(SCONE_EHIP);
    const unsigned g_n = (unsigned)((n + kThreads - 1) / kThreads);
    if (rc == SCONE_OK) {
        hipLaunchKernelGGL(k_len_count, dim3(g_n), dim3(kThreads), 0, st, lengths, n, max_len,
                           counts, status);
        if (hipGetLastError() != hipSuccess ||
            hipMemcpyAsync(hc, ctl, 32 * sizeof(unsigned), hipMemcpyDeviceToHost, st) !=
                hipSuccess ||
            hipStreamSynchronize(st) != hipSuccess)
            fail(SCONE_EHIP);
    }
    if (rc == SCONE_OK && (hc[0] & err_bit(SCONE_ELEN))) fail(SCONE_ELEN);
    // One chunk holds at most kChunkTokens tokens of one length.
    int64_t ctok = 0;
    if (rc == SCONE_OK) {
        int64_t acc = 0;
        for (int L = 0; L < 8; ++L) {
            hbase[L] = acc;
            acc += hc[8 + L];
            if (L >= 2) {
                const int64_t t = (int64_t)hc[8 + L] * L;
                const int64_t cap = (kChunkTokens / L) * L;
                ctok = std::max(ctok, std::min(t, cap));
            }
        }
        if (hipMemcpyAsync(base, hbase, sizeof(hbase), hipMemcpyHostToDevice, st) != hipSuccess)
            fail(SCONE_EHIP);
    }
    Buffers B{};
    if (rc == SCONE_OK) {
        const size_t h_bytes = (size_t)align_up(ctok * d) * 4;
        // matrix-product inputs (a, f) are readable up to a whole 256-row tile
        const int64_t ptok = (ctok + 255) / 256 * 256;
        const size_t a_bytes = (size_t)align_up(ptok * d) * 2;
        const size_t qkv_bytes = (size_t)align_up(ctok * 3 * d) * 2;
        const size_t f_bytes = (size_t)align_up(ptok * d_ff) * 2;
        if (hipMalloc(&act, h_bytes + a_bytes + qkv_bytes + f_bytes) != hipSuccess) {
            act = nullptr;
            fail(SCONE_ENOMEM);
        } else {
            B.h = reinterpret_cast<float*>(act);
            B.a = reinterpret_cast<uint16_t*>(act + h_bytes);
            B.qkv = reinterpret_cast<uint16_t*>(act + h_bytes + a_bytes);
            B.f = reinterpret_cast<uint16_t*>(act + h_bytes + a_bytes + qkv_bytes);
        }
    }
    if (rc == SCONE_OK) {
        hipLaunchKernelGGL(k_len_scatter, dim3(g_n), dim3(kThreads), 0, st, lengths, n, max_len,
                           base, cursor, order);
        if (hipGetLastError() != hipSuccess) fail(SCONE_EHIP);
    }
    const Weights w = bind_weights(static_cast<const uint16_t*>(params), d, d_ff, n_layers,
                                   max_len);
    for (int L = 2; L <= max_len && rc == SCONE_OK; ++L) {
        const int64_t cnt = hc[8 + L];
        const int64_t per_chunk = kChunkTokens / L;
        for (int64_t s = 0; s < cnt && rc == SCONE_OK; s += per_chunk) {
            const int64_t nf = cnt - s < per_chunk ? cnt - s : per_chunk;
            if (fn(w, order + hbase[L] + s, nf, L, fgrams, max_len,
                   static_cast<const uint16_t*>(tok_rows), vocab, d_ff, n_heads, row_ids,
                   static_cast<uint16_t*>(rows), n_rows, B, status, st) != hipSuccess)
                fail(SCONE_EHIP);
        }
    }
    unsigned hs = 0;
    if (hipMemcpyAsync(&hs, status, sizeof(unsigned), hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess)
        fail(SCONE_EHIP);
    if (rc == SCONE_OK && hs) rc = code_from_bits(hs);
    (void)hipFree(act);
    (void)hipFree(ctl);
    return rc;
}
