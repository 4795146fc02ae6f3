// bf16 matrix product on the gfx950 matrix cores, with the epilogues the
// f-gram model needs fused in:
//
//   C[m, n] = sum_k A[m, k] * W[n, k] + bias[n]        (A [M, K], W [N, K])
//   kBias:  out_bf16[m, n]  = bf16(C)
//   kGelu:  out_bf16[m, n]  = bf16(GELU(C))             (exact, erf form)
//   kResid: out_f32[m, n]  += C                         (the residual stream)
//
// Both operands are K-contiguous, so every tile row is a run of 16-byte
// loads.  A workgroup of four wavefronts computes a 128 x 128 tile with a
// 64-deep k-slab double-buffered in LDS (one barrier per slab).  Each
// wavefront owns a 64 x 64 quarter as 4 x 4 v_mfma_f32_16x16x32_bf16 tiles.
// W is passed as the instruction's first operand and A as the second, so a
// lane's four accumulators are four consecutive n of one row m: the epilogue
// writes 8 bytes (bf16) or 16 bytes (f32) per lane per tile.
//
// LDS rows are padded from 64 to 72 elements (144 bytes), which spreads the
// sixteen rows a fragment read touches over distinct banks.
#pragma once

#include "scone_internal.h"

namespace scone {
namespace gemm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kBM = 128;  // rows of A (tokens) per tile
constexpr int kBN = 128;  // rows of W (output features) per tile
constexpr int kBK = 64;   // k-slab
constexpr int kLd = kBK + 8;  // padded LDS row, elements

enum Epilogue { kBias = 0, kGelu = 1, kResid = 2 };

__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// Round to nearest, ties to even (inputs are finite).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float gelu_erf(float x) {
    return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f));
}

template <int EPI>
__global__ __launch_bounds__(kThreads) void k_gemm(const uint16_t* __restrict__ A,
                                                   const uint16_t* __restrict__ W,
                                                   const uint16_t* __restrict__ bias,
                                                   void* __restrict__ out, int M, int N, int K,
                                                   int tiles_n) {
    __shared__ __attribute__((aligned(16))) uint16_t sA[2][kBM * kLd];
    __shared__ __attribute__((aligned(16))) uint16_t sW[2][kBN * kLd];

    // Consecutive workgroups land on different XCDs; renumber so that each
    // XCD walks a contiguous run of tiles (n fastest), which keeps the A rows
    // of a tile row in that XCD's L2 while its n-tiles are computed.
    const int nb = gridDim.x;
    const int b = blockIdx.x;
    const int per = nb / 8;
    const int t = (b < per * 8) ? (b % 8) * per + b / 8 : b;
    const int tm = t / tiles_n, tn = t % tiles_n;
    const int m0 = tm * kBM, n0 = tn * kBN;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    // Global -> LDS copy: 256 threads x 16 bytes = 32 rows of 64 elements per pass.
    const int lr = tid >> 3;         // 0..31
    const int lc = (tid & 7) * 8;    // element column within the slab
    const uint16_t* gA[4];
    const uint16_t* gW[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        int ra = m0 + lr + 32 * p;
        ra = ra < M ? ra : M - 1;  // rows past M repeat the last row; never stored
        gA[p] = A + (int64_t)ra * K + lc;
        gW[p] = W + (int64_t)(n0 + lr + 32 * p) * K + lc;
    }

    f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    u32x4 ra[4], rw[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        ra[p] = *reinterpret_cast<const u32x4*>(gA[p]);
        rw[p] = *reinterpret_cast<const u32x4*>(gW[p]);
    }
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        *reinterpret_cast<u32x4*>(&sA[0][(lr + 32 * p) * kLd + lc]) = ra[p];
        *reinterpret_cast<u32x4*>(&sW[0][(lr + 32 * p) * kLd + lc]) = rw[p];
    }
    __syncthreads();

    const int fr = lane & 15;         // fragment row
    const int fk = (lane >> 4) * 8;   // fragment k offset
    const int KT = K / kBK;
    for (int kt = 0; kt < KT; ++kt) {
        const int cur = kt & 1;
        const bool more = kt + 1 < KT;
        if (more) {
            const int off = (kt + 1) * kBK;
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                ra[p] = *reinterpret_cast<const u32x4*>(gA[p] + off);
                rw[p] = *reinterpret_cast<const u32x4*>(gW[p] + off);
            }
        }
#pragma unroll
        for (int ks = 0; ks < kBK; ks += 32) {
            bf16x8 fw[4], fa[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                fw[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                    &sW[cur][(wn * 64 + i * 16 + fr) * kLd + ks + fk]));
                fa[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                    &sA[cur][(wm * 64 + i * 16 + fr) * kLd + ks + fk]));
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[i], fa[j], acc[i][j],
                                                                        0, 0, 0);
        }
        if (more) {
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                *reinterpret_cast<u32x4*>(&sA[cur ^ 1][(lr + 32 * p) * kLd + lc]) = ra[p];
                *reinterpret_cast<u32x4*>(&sW[cur ^ 1][(lr + 32 * p) * kLd + lc]) = rw[p];
            }
        }
        __syncthreads();
    }

    // acc[i][j][r] = C[m, n] with n = n0 + wn*64 + i*16 + (lane/16)*4 + r and
    // m = m0 + wm*64 + j*16 + lane%16.
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int n = n0 + wn * 64 + i * 16 + (lane >> 4) * 4;
        const u32x2 bb = *reinterpret_cast<const u32x2*>(bias + n);
        const float b0 = bf16_to_f32(bb.x & 0xFFFFu), b1 = bf16_to_f32(bb.x >> 16);
        const float b2 = bf16_to_f32(bb.y & 0xFFFFu), b3 = bf16_to_f32(bb.y >> 16);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int m = m0 + wm * 64 + j * 16 + (lane & 15);
            if (m >= M) continue;
            float v0 = acc[i][j][0] + b0, v1 = acc[i][j][1] + b1;
            float v2 = acc[i][j][2] + b2, v3 = acc[i][j][3] + b3;
            if (EPI == kResid) {
                f32x4* p = reinterpret_cast<f32x4*>(static_cast<float*>(out) + (int64_t)m * N + n);
                f32x4 h = *p;
                h[0] += v0; h[1] += v1; h[2] += v2; h[3] += v3;
                *p = h;
            } else {
                if (EPI == kGelu) {
                    v0 = gelu_erf(v0); v1 = gelu_erf(v1); v2 = gelu_erf(v2); v3 = gelu_erf(v3);
                }
                u32x2 o;
                o.x = f32_to_bf16(v0) | (f32_to_bf16(v1) << 16);
                o.y = f32_to_bf16(v2) | (f32_to_bf16(v3) << 16);
                *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(out) + (int64_t)m * N + n) = o;
            }
        }
    }
}

// Shapes: N % 128 == 0, K % 64 == 0, M >= 1; all pointers 16-byte aligned.
template <int EPI>
inline hipError_t launch(const uint16_t* A, const uint16_t* W, const uint16_t* bias, void* out,
                         int M, int N, int K, hipStream_t st) {
    const int tiles_n = N / kBN;
    const int tiles_m = (M + kBM - 1) / kBM;
    hipLaunchKernelGGL(k_gemm<EPI>, dim3((unsigned)(tiles_m * tiles_n)), dim3(kThreads), 0, st,
                       A, W, bias, out, M, N, K, tiles_n);
    return hipGetLastError();
}

}  // namespace gemm
}  // namespace scone
