// bf16 matrix product on the gfx950 matrix cores, with the epilogues the
// f-gram model needs fused in:
//
//   C[m, n] = sum_k A[m, k] * W[n, k] + bias[n]        (A [M, K], W [N, K])
//   kBias:  out_bf16[m, n]  = bf16(C)
//   kGelu:  out_bf16[m, n]  = bf16(GELU(C))             (erf form)
//   kResid: out_f32[m, n]  += C                         (the residual stream)
//
// Both operands are K-contiguous.  A workgroup computes a BM x BN tile over
// 64-deep k-slabs held in a two-stage LDS ring.  Slabs move from global
// memory straight into LDS (global_load_lds_dwordx4: no registers, no LDS
// write instructions); the next slab is in flight while the current one is
// multiplied, and the only synchronisation per slab is a counted wait on the
// wavefront's own copies plus a workgroup barrier.  Fragments are double
// buffered in registers: a slab is two 32-deep halves, and the LDS reads of
// one half are in flight while the matrix cores multiply the other, so the
// products of a slab's second half run after the barrier while the next
// slab's first fragments load.  The reads and copies are slotted one after
// each product (see `step` below) rather than issued as a block.  Each
// wavefront owns a
// (BM / WGM) x (BN / WGN) part of the tile as 16 x 16 v_mfma_f32_16x16x32_bf16
// tiles.  W is the instruction's first operand and A the second, so a lane's
// four accumulators are four consecutive n of one row m: the epilogue writes
// 8 bytes (bf16) or 16 bytes (f32) per lane per tile.
//
// The bf16 epilogues (kBias, kGelu) stage the finished tile in LDS after the
// last slab and store it row by row: a lane's accumulators hold 4 consecutive
// n of one row m, so written straight from registers a row gets 32 bytes per
// store instruction; through LDS each store instruction writes whole 256-byte
// row segments.  Those stores are non-temporal: the outputs (hundreds of MB)
// are read back by the next kernel, never by this one, and streaming them past
// the caches made the q/k/v and fc1 products 6-7% faster at M = 65,536 (the
// narrow direct stores lose with the same hint).  The residual epilogue reads
// its output first and keeps the direct stores.
//
// LDS layout: a slab row is 64 elements = 128 bytes = eight 16-byte chunks,
// stored at slot chunk ^ (row & 7).  A fragment read touches 16 consecutive
// rows at one chunk; with this swizzle the LDS bank-conflict counter reads
// zero and a 16-byte fragment read occupies the LDS for 4 cycles (unswizzled:
// 16; other XOR patterns tried: 8).  One copy instruction fills 1 KB of LDS
// (8 whole rows), each lane fetching the chunk its slot must hold.
#pragma once

#include <type_traits>

#include "scone_internal.h"

namespace scone {
namespace gemm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef __attribute__((address_space(1))) void* gbl_ptr_t;

enum Epilogue { kBias = 0, kGelu = 1, kResid = 2 };

__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// Two floats to two bf16 in one word (a low, b high), rounded to nearest,
// ties to even, by the hardware conversion (v_cvt_pk_bf16_f32): the same
// bits as f32_to_bf16 below for every finite float (checked on gfx950 over
// all 2^32 bit patterns), in one instruction instead of about eight.
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{a, b}), bf16x2));
}

// Round to nearest, ties to even (inputs are finite).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// GELU(x) = x Phi(x) = x (1 + erf(x / sqrt 2)) / 2, with erf from
// Abramowitz and Stegun 7.1.26 (Hastings' rational approximation):
// erf(z) = 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) exp(-z^2),
// t = 1 / (1 + p z), z >= 0, absolute error at most 1.5e-7, odd in z.  The
// outputs are rounded to bf16 (relative step 2^-8), so the approximation is
// invisible in them; it costs one reciprocal and one exp2 on the hardware
// units instead of a full-precision erf.
__device__ __forceinline__ float gelu_erf(float x) {
    const float z = fabsf(x) * 0.70710678118654752f;
    const float t = __builtin_amdgcn_rcpf(1.0f + 0.3275911f * z);
    float q = 1.061405429f;
    q = q * t - 1.453152027f;
    q = q * t + 1.421413741f;
    q = q * t - 0.284496736f;
    q = q * t + 0.254829592f;
    const float e = __builtin_amdgcn_exp2f(-(z * z) * 1.4426950408889634f);  // exp(-z^2)
    const float erf_abs = 1.0f - q * t * e;
    return 0.5f * x * (1.0f + (x < 0.0f ? -erf_abs : erf_abs));
}

// The lane id, computed from the execution mask with an operand the
// compiler cannot see through, so it is not merged with an earlier copy:
// values derived from it are recomputed where they are used instead of being
// held in registers (at 256 registers per lane, held values spill).
__device__ __forceinline__ int fresh_lane() {
    unsigned z = 0;
    asm volatile("" : "+s"(z));
    return (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, z));
}

// s_waitcnt immediates (gfx9 encoding): wait until at most n vector-memory
// operations are outstanding / until no LDS operation is outstanding.
constexpr int waitcnt_vm(int n) {
    return (n & 0xF) | (7 << 4) | (0xF << 8) | (((n >> 4) & 3) << 14);
}
constexpr int kWaitLds = 0xF | (7 << 4) | (0 << 8) | (3 << 14);

constexpr int kBK = 64;        // k-slab depth (elements)
constexpr int kRowBytes = 128;  // one slab row in LDS

template <int EPI, int BM, int BN, int WGM, int WGN, bool kStaged>
__global__ __launch_bounds__(64 * WGM * WGN) void k_gemm(const uint16_t* __restrict__ A,
                                                         const uint16_t* __restrict__ W,
                                                         const uint16_t* __restrict__ bias,
                                                         void* __restrict__ out, int64_t ldc,
                                                         int M, int N, int K, int tiles_n) {
    constexpr int NW = WGM * WGN;
    constexpr int WTM = BM / WGM, WTN = BN / WGN;  // wavefront tile
    constexpr int TM = WTM / 16, TN = WTN / 16;
    constexpr int STAGE = (BM + BN) * kRowBytes;
    constexpr int GA = BM / 8 / NW, GW = BN / 8 / NW;  // 8-row copy groups per wavefront
    static_assert(GA * 8 * NW == BM && GW * 8 * NW == BN, "copy groups must split evenly");
    static_assert(!kStaged || EPI != kResid, "the residual epilogue is not staged");
    constexpr int ERS = WTN * 2 + 16;  // staged row stride: 16 bytes of padding per row
    constexpr int SMEM = kStaged && NW * WTM * ERS > 2 * STAGE ? NW * WTM * ERS : 2 * STAGE;
    __shared__ __attribute__((aligned(1024))) uint8_t smem[SMEM];

    // Consecutive workgroups land on different XCDs; renumber so that each
    // XCD walks a contiguous run of tiles, and order that run in groups of
    // kGroupM tile rows, m fastest inside a group, so that the workgroups an
    // XCD runs at once share A and W slabs in its L2: 32 of them as 8 rows by
    // 4 columns touch 12 slabs per k-step, where a run along n touches 15 on
    // a 12-column product and 18 on a 16-column one (4-column products were
    // 8 by 4 already).
    constexpr int kGroupM = 8;
    const int nb = gridDim.x;
    const int b = blockIdx.x;
    const int per = nb / 8;
    const int t = (b < per * 8) ? (b % 8) * per + b / 8 : b;
    const int tiles_m = (M + BM - 1) / BM;
    const int group = t / (kGroupM * tiles_n);
    const int first = group * kGroupM;
    const int gm = tiles_m - first < kGroupM ? tiles_m - first : kGroupM;
    const int tr = t - group * kGroupM * tiles_n;
    const int tm = first + tr % gm, tn = tr / gm;
    const int m0 = tm * BM, n0 = tn * BN;

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave / WGN, wn = wave % WGN;

    // Copies: wavefront w fills 8-row groups w*GA .. w*GA+GA-1 of the A tile
    // and w*GW .. of the W tile.  Lane l covers row l/8 of a group and slot
    // l%8, which holds chunk (l%8) ^ (row & 7) = (l%8) ^ (l/8).
    const int lrow = lane >> 3, lslot = lane & 7;
    const int chunk = (lslot ^ lrow) * 8;
    const int gA0 = wave * GA, gW0 = wave * GW;
    // A has readable rows up to the next multiple of BM (rows past M hold
    // anything: they only feed output rows that are never stored).
    const uint16_t* pA = A + (int64_t)(m0 + gA0 * 8 + lrow) * K;
    const uint16_t* pW = W + (int64_t)(n0 + gW0 * 8 + lrow) * K;
    const int64_t grp = (int64_t)8 * K;

    auto issue = [&](int slab, int stage) {
        const int ko = slab * kBK;
        uint8_t* sbase = smem + stage * STAGE;
#pragma unroll
        for (int j = 0; j < GA; ++j)
            __builtin_amdgcn_global_load_lds(
                (gbl_ptr_t)(pA + j * grp + ko + chunk),
                (lds_ptr_t)(sbase + (gA0 + j) * 1024), 16, 0, 0);
#pragma unroll
        for (int j = 0; j < GW; ++j)
            __builtin_amdgcn_global_load_lds(
                (gbl_ptr_t)(pW + j * grp + ko + chunk),
                (lds_ptr_t)(sbase + BM * kRowBytes + (gW0 + j) * 1024), 16, 0, 0);
    };

    f32x4 acc[TN][TM];
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int fr = lane & 15;                          // fragment row
    const int swz = lane & 7;                          // fragment row & 7
    const int q0 = lane >> 4;                          // fragment k chunk
    // Fragments of 32-deep half `ks` of the slab in `stage`.
    auto read = [&](int stage, int ks, bf16x8* fw, bf16x8* fa) {
        const uint8_t* sA = smem + stage * STAGE;
        const uint8_t* sW = sA + BM * kRowBytes;
        const int slot = ((ks * 4 + q0) ^ swz) * 16;
#pragma unroll
        for (int i = 0; i < TN; ++i)
            fw[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                sW + (wn * WTN + i * 16 + fr) * kRowBytes + slot));
#pragma unroll
        for (int j = 0; j < TM; ++j)
            fa[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
                sA + (wm * WTM + j * 16 + fr) * kRowBytes + slot));
    };
    auto multiply = [&](const bf16x8* fw, const bf16x8* fa) {
#pragma unroll
        for (int i = 0; i < TN; ++i)
#pragma unroll
            for (int j = 0; j < TM; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[i], fa[j], acc[i][j],
                                                                    0, 0, 0);
    };

    // Scheduling masks of __builtin_amdgcn_sched_group_barrier.
    constexpr int kMfma = 0x008, kVmemRead = 0x020, kDsRead = 0x100;
    constexpr int NR = TN + TM;  // fragment reads per half slab
    constexpr int NP = TN * TM;  // products per half slab
    static_assert(NP >= NR + GA + GW, "the interleave needs a product per read and copy");
    const int KT = K / kBK;
    bf16x8 f0w[TN], f0a[TM], f1w[TN], f1a[TM];  // halves 0 and 1 of a slab
    u32x2 bb[TN];                                // this lane's biases, loaded in the last slab
    issue(0, 0);
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    if (KT > 1) issue(1, 1);
    read(0, 0, f0w, f0a);
    // One slab.  Half 0's products run with half 1's fragment reads slotted
    // one after each product, so the reads overlap the products.  Issued as
    // a block before the products, as the compiler orders them by itself, the
    // reads were followed by a wait for every outstanding LDS read (the count
    // covers all of them, the new ones included) and both wavefronts of a
    // SIMD idled for an LDS round trip per slab.  When a next slab exists:
    // the counted waits and the barrier, then half 1's products with the
    // copies of slab kt + 2 and the next slab's half-0 reads slotted in the
    // same way.  kNext / kIssue are compile-time so that each half is one
    // straight run of code the scheduler can interleave.
    auto step = [&](int kt, auto next_c, auto issue_c) {
        constexpr bool kNext = decltype(next_c)::value;
        constexpr bool kIssue = decltype(issue_c)::value;
        read(kt & 1, 1, f1w, f1a);
        multiply(f0w, f0a);
#pragma unroll
        for (int i = 0; i < NR; ++i) {
            __builtin_amdgcn_sched_group_barrier(kMfma, 1, 0);
            __builtin_amdgcn_sched_group_barrier(kDsRead, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(kMfma, NP - NR, 0);
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (kNext) {
            // Half 1 of slab kt has landed, so this wavefront reads nothing
            // more from stage kt & 1, and its copies of slab kt + 1 are in
            // LDS; after the barrier the same holds for every wavefront:
            // slab kt + 1 is readable and stage kt & 1 may be refilled.
            __builtin_amdgcn_s_waitcnt(kWaitLds);
            __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (kIssue) issue(kt + 2, kt & 1);
            read((kt + 1) & 1, 0, f0w, f0a);
        } else {
            // Last slab: the epilogue's bias loads fly during half 1's
            // products, in the registers half 0's fragments held.
#pragma unroll
            for (int i = 0; i < TN; ++i)
                bb[i] = *reinterpret_cast<const u32x2*>(bias + n0 + wn * WTN + i * 16 +
                                                         (lane >> 4) * 4);
        }
        multiply(f1w, f1a);
        if constexpr (kNext) {
            if constexpr (kIssue) {
#pragma unroll
                for (int i = 0; i < GA + GW; ++i) {
                    __builtin_amdgcn_sched_group_barrier(kMfma, 1, 1);
                    __builtin_amdgcn_sched_group_barrier(kVmemRead, 1, 1);
                }
            }
#pragma unroll
            for (int i = 0; i < NR; ++i) {
                __builtin_amdgcn_sched_group_barrier(kMfma, 1, 1);
                __builtin_amdgcn_sched_group_barrier(kDsRead, 1, 1);
            }
            __builtin_amdgcn_sched_group_barrier(kMfma, NP - NR - (kIssue ? GA + GW : 0), 1);
        }
        __builtin_amdgcn_sched_barrier(0);
    };
    int kt = 0;
    for (; kt + 2 < KT; ++kt) step(kt, std::true_type{}, std::true_type{});
    if (kt + 1 < KT) step(kt++, std::true_type{}, std::false_type{});
    step(kt, std::false_type{}, std::false_type{});

    // The epilogue takes a fresh lane id (see fresh_lane) so that no
    // lane-derived value stays live through the main loop.
    const int elane = fresh_lane();
    // acc[i][j][r] = C[m, n] with n = n0 + wn*WTN + i*16 + (lane/16)*4 + r and
    // m = m0 + wm*WTM + j*16 + lane%16.  Every load the epilogue needs (the
    // biases, and for kResid the residual values of up to four column groups)
    // is issued before its first use, so a wavefront waits once per round
    // instead of once per 16 x 16 tile; rows past M read row M - 1 and are
    // not stored.
    if constexpr (kStaged) {
        // Every wavefront is done reading slabs before any overwrites them.
        __builtin_amdgcn_s_waitcnt(kWaitLds);
        __builtin_amdgcn_s_barrier();
        uint8_t* wb = smem + wave * (WTM * ERS);  // this wavefront's WTM x WTN part
#pragma unroll
        for (int i = 0; i < TN; ++i) {
            const float b0 = bf16_to_f32(bb[i].x & 0xFFFFu), b1 = bf16_to_f32(bb[i].x >> 16);
            const float b2 = bf16_to_f32(bb[i].y & 0xFFFFu), b3 = bf16_to_f32(bb[i].y >> 16);
#pragma unroll
            for (int j = 0; j < TM; ++j) {
                float v0 = acc[i][j][0] + b0, v1 = acc[i][j][1] + b1;
                float v2 = acc[i][j][2] + b2, v3 = acc[i][j][3] + b3;
                if (EPI == kGelu) {
                    v0 = gelu_erf(v0); v1 = gelu_erf(v1); v2 = gelu_erf(v2); v3 = gelu_erf(v3);
                }
                u32x2 o;
                o.x = pack_bf16x2(v0, v1);
                o.y = pack_bf16x2(v2, v3);
                *reinterpret_cast<u32x2*>(wb + (j * 16 + (elane & 15)) * ERS +
                                          (i * 16 + (elane >> 4) * 4) * 2) = o;
            }
        }
        __builtin_amdgcn_s_waitcnt(kWaitLds);
        constexpr int LPR = WTN * 2 / 16;  // lanes per row, 16 bytes each
        constexpr int RPI = 64 / LPR;      // rows per store instruction
        const int rr = elane / LPR, cc = elane % LPR;
        uint16_t* ob = static_cast<uint16_t*>(out);
#pragma unroll
        for (int it = 0; it < WTM / RPI; ++it) {
            const int r = it * RPI + rr;
            const int m = m0 + wm * WTM + r;
            const u32x4 v = *reinterpret_cast<const u32x4*>(wb + r * ERS + cc * 16);
            if (m < M)
                __builtin_nontemporal_store(
                    v, reinterpret_cast<u32x4*>(ob + (int64_t)m * ldc + n0 + wn * WTN + cc * 8));
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < TN; ++i) {
        const int n = n0 + wn * WTN + i * 16 + (elane >> 4) * 4;
        const float b0 = bf16_to_f32(bb[i].x & 0xFFFFu), b1 = bf16_to_f32(bb[i].x >> 16);
        const float b2 = bf16_to_f32(bb[i].y & 0xFFFFu), b3 = bf16_to_f32(bb[i].y >> 16);
        if (EPI == kResid) {
            // G column groups per round: their G * TM residual loads are all
            // in flight before the first add.
            constexpr int G = TN < 4 ? TN : 4;
            if (i % G != 0) continue;
            float* o = static_cast<float*>(out);
            f32x4 h[G][TM];
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
                for (int j = 0; j < TM; ++j) {
                    const int m = m0 + wm * WTM + j * 16 + (elane & 15);
                    h[g][j] = *reinterpret_cast<const f32x4*>(
                        o + (int64_t)(m < M ? m : M - 1) * ldc + n + g * 16);
                }
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const u32x2 bg = bb[i + g];
                const float c0 = bf16_to_f32(bg.x & 0xFFFFu), c1 = bf16_to_f32(bg.x >> 16);
                const float c2 = bf16_to_f32(bg.y & 0xFFFFu), c3 = bf16_to_f32(bg.y >> 16);
#pragma unroll
                for (int j = 0; j < TM; ++j) {
                    const int m = m0 + wm * WTM + j * 16 + (elane & 15);
                    if (m >= M) continue;
                    h[g][j][0] += acc[i + g][j][0] + c0;
                    h[g][j][1] += acc[i + g][j][1] + c1;
                    h[g][j][2] += acc[i + g][j][2] + c2;
                    h[g][j][3] += acc[i + g][j][3] + c3;
                    *reinterpret_cast<f32x4*>(o + (int64_t)m * ldc + n + g * 16) = h[g][j];
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < TM; ++j) {
                const int m = m0 + wm * WTM + j * 16 + (elane & 15);
                if (m >= M) continue;
                float v0 = acc[i][j][0] + b0, v1 = acc[i][j][1] + b1;
                float v2 = acc[i][j][2] + b2, v3 = acc[i][j][3] + b3;
                if (EPI == kGelu) {
                    v0 = gelu_erf(v0); v1 = gelu_erf(v1); v2 = gelu_erf(v2); v3 = gelu_erf(v3);
                }
                u32x2 o;
                o.x = pack_bf16x2(v0, v1);
                o.y = pack_bf16x2(v2, v3);
                *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(out) + (int64_t)m * ldc + n) = o;
            }
        }
    }
}

template <int EPI, int BM, int BN, int WGM, int WGN>
inline hipError_t launch_tiles(const uint16_t* A, const uint16_t* W, const uint16_t* bias,
                               void* out, int64_t ldc, int M, int N, int K, hipStream_t st) {
    const int tiles_n = N / BN;
    const int tiles_m = (M + BM - 1) / BM;
    const dim3 grid((unsigned)(tiles_m * tiles_n)), block(64 * WGM * WGN);
    // The staged store writes 16-byte pieces: rows must start 16-byte aligned.
    if (EPI != kResid && ldc % 8 == 0 && (uintptr_t)out % 16 == 0)
        hipLaunchKernelGGL((k_gemm<EPI, BM, BN, WGM, WGN, EPI != kResid>), grid, block, 0, st, A,
                           W, bias, out, ldc, M, N, K, tiles_n);
    else
        hipLaunchKernelGGL((k_gemm<EPI, BM, BN, WGM, WGN, false>), grid, block, 0, st, A, W,
                           bias, out, ldc, M, N, K, tiles_n);
    return hipGetLastError();
}

// Shapes: N % 128 == 0, K % 64 == 0, M >= 1; all pointers 16-byte aligned;
// A readable up to row roundup(M, 256); output row m starts at out + m * ldc
// elements (ldc >= N, a multiple of 4).  Large products take 256 x 256 tiles
// on eight wavefronts (half the LDS and L2 traffic per flop of 128 x 128);
// N not a multiple of 256, or too few tiles to fill the 256 compute units,
// take 128 x 128 on four.  The eight wavefronts of a 256 x 256 tile own
// 64 x 128 parts (four down, two across): measured faster than 128 x 64
// parts on every product of the f-gram model.
template <int EPI>
inline hipError_t launch(const uint16_t* A, const uint16_t* W, const uint16_t* bias, void* out,
                         int64_t ldc, int M, int N, int K, hipStream_t st) {
    if (N % 256 == 0 && (int64_t)((M + 255) / 256) * (N / 256) >= 256)
        return launch_tiles<EPI, 256, 256, 4, 2>(A, W, bias, out, ldc, M, N, K, st);
    return launch_tiles<EPI, 128, 128, 2, 2>(A, W, bias, out, ldc, M, N, K, st);
}

}  // namespace gemm
}  // namespace scone
