// LUT-decode GEMM on packed Lloyd-Max codes for gfx950 (bf16 MFMA, fp32 accumulate).
//
// Computes Y[n][i] = s_n * r'_i * sum_k L_a[xc[n][k]] * L_w[wc[i][k]]: the rotation cancels in
// the product (Sec. 4.3), so the two code sets are contracted directly in the rotated basis;
// the paper's limitations section names this codebook GEMM as the missing kernel.
//
// Operands: codes are dequantized to the bf16 images of the levels and multiplied in bf16, the
// arithmetic the paper runs its layers in (codes dequantized to BF16, matmul in BF16); on the
// matrix cores the products accumulate in fp32.
//
// Decode: codes are widened to bytes and looked up with v_perm_b32 against byte tables of the
// bf16 levels (low bytes and high bytes of the 2^b levels, 8 entries per register pair), which
// needs no memory access.  Each code of a block tile is decoded exactly once, into a bf16 tile
// in LDS that the matrix cores then read.  bf16 products are exact in fp32, so the result
// differs from an fp64 evaluation with the same bf16 levels only by fp32 accumulation.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "device.h"

namespace orbit {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int LDS_STRIDE = BK + 8;  // halves per tile row (padding against bank conflicts)

// 32 packed codes of one row: 4*BITS bytes, in BITS words (4 words for 2- and 3-bit codes too)
template <int BITS>
using Codes = uint32_t[BITS == 6 ? 6 : 4];

struct ByteTables {
    uint32_t lo[2], hi[2];  // byte e of lo[e/4] (hi[e/4]) is the low (high) byte of table entry e
};

// `lut` holds the levels in label order (entry l is the level of sign-magnitude label l).  Tables
// of at most eight levels hold every label.  The 4-bit table holds labels 0..7 only, the positive
// levels by rank: the codebook is antisymmetric (L[15-c] = -L[c], Sec. 3's symmetric marginal),
// so label 8 + m is the negation of label m, and the decoder looks up the low three bits and
// moves bit 3 into the bf16 sign bit.  The host checks the antisymmetry bit for bit.
template <int BITS>
__device__ __forceinline__ ByteTables make_tables(const uint16_t* lut) {
    constexpr int n = BITS == 4 ? 8 : BITS == 6 ? 0 : 1 << BITS, first = 0;
    ByteTables t;
#pragma unroll
    for (int w = 0; w < 2; ++w) {
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int e = 4 * w + b;
            const uint32_t v = e < n ? lut[first + e] : 0u;
            lo |= (v & 0xFFu) << (8 * b);
            hi |= (v >> 8) << (8 * b);
        }
        t.lo[w] = lo;
        t.hi[w] = hi;
    }
    return t;
}

// Canonical slot order.  The eight codes of each aligned group k0..k7 are written to eight
// consecutive bf16 slots in the order k0 k2 k4 k6 k1 k3 k5 k7.  Both operands use the same order
// for every bit width, so every MFMA still contracts matching k; the order is the one the 4-bit
// decoder produces without any byte shuffling (even and odd nibbles of a code word).

// Four table indices (one per byte of sel, each below 8) -> bf16 low and high bytes.
__device__ __forceinline__ void lookup_bytes(uint32_t sel, const ByteTables& t, uint32_t& lo, uint32_t& hi) {
    lo = __builtin_amdgcn_perm(t.lo[1], t.lo[0], sel);
    hi = __builtin_amdgcn_perm(t.hi[1], t.hi[0], sel);
}

// low/high byte words of four values -> two bf16x2 words (values 0,1 and 2,3)
__device__ __forceinline__ void interleave(uint32_t lo, uint32_t hi, uint32_t& d0, uint32_t& d1) {
    d0 = __builtin_amdgcn_perm(hi, lo, 0x05010400u);  // [lo0 hi0 lo1 hi1]
    d1 = __builtin_amdgcn_perm(hi, lo, 0x07030602u);  // [lo2 hi2 lo3 hi3]
}

// 2- and 3-bit groups: every level is in the table
template <int BITS>
__device__ __forceinline__ void decode8_small(const Codes<BITS>& w, int g, const ByteTables& t, uint32_t (&out)[4]) {
    uint32_t lo, hi;
    uint32_t ce, co;  // codes k0 k2 k4 k6 and k1 k3 k5 k7, one per byte
    if constexpr (BITS == 2) {
        uint32_t xw = w[g >> 1];
        asm volatile("" : "+v"(xw));  // as in decode8: keep the decode at its use
        const uint32_t x = xw >> (16 * (g & 1));             // 16 bits, code j at bits 2j
        const uint32_t e = x & 0x3333u, o = (x >> 2) & 0x3333u;  // nibble i holds k2i (k2i+1)
        ce = __builtin_amdgcn_perm(e >> 4, e, 0x05010400u) & 0x03030303u;
        co = __builtin_amdgcn_perm(o >> 4, o, 0x05010400u) & 0x03030303u;
    } else {
        static_assert(BITS == 3, "bits");
        const int bit = 24 * g;                               // 24 bits, code j at bits 3j
        uint32_t x = bit == 0 ? w[0] : bit == 24 ? (w[0] >> 24) | (w[1] << 8)
                   : bit == 48 ? (w[1] >> 16) | (w[2] << 16) : w[2] >> 8;
        asm volatile("" : "+v"(x));  // as in decode8: keep the decode at its use
        ce = (x & 7u) | (((x >> 6) & 7u) << 8) | (((x >> 12) & 7u) << 16) | (((x >> 18) & 7u) << 24);
        co = ((x >> 3) & 7u) | (((x >> 9) & 7u) << 8) | (((x >> 15) & 7u) << 16) | (((x >> 21) & 7u) << 24);
    }
    lookup_bytes(ce, t, lo, hi);
    interleave(lo, hi, out[0], out[1]);
    lookup_bytes(co, t, lo, hi);
    interleave(lo, hi, out[2], out[3]);
}

// 6-bit groups: 64 levels are too many for byte permutes, so the bf16 levels sit in a 64-entry
// LDS table with a 4-byte stride; every entry has its own bank, so a wave's 64 lookups never
// conflict (equal codes broadcast).
__device__ __forceinline__ void decode8_lds6(const Codes<6>& w, int g, const uint32_t* tab, uint32_t (&out)[4]) {
    // group g covers bits 48g .. 48g+47 of the 192-bit stream (selects, not an indexed load from
    // the register array)
    uint32_t lo = g == 0 ? w[0] : g == 1 ? w[1] : g == 2 ? w[3] : w[4];
    uint32_t hi = g == 0 ? w[1] : g == 1 ? w[2] : g == 2 ? w[4] : w[5];
    asm volatile("" : "+v"(lo), "+v"(hi));  // as in decode8: keep the decode at its use
    const uint64_t x = (((uint64_t)hi << 32) | lo) >> ((g & 1) * 16);
    uint32_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = tab[(uint32_t)(x >> (6 * j)) & 63u];
    out[0] = v[0] | (v[2] << 16);
    out[1] = v[4] | (v[6] << 16);
    out[2] = v[1] | (v[3] << 16);
    out[3] = v[5] | (v[7] << 16);
}

// Group g (codes 8g .. 8g+7) of 32 packed codes (4*BITS bytes, LSB-first) -> four bf16x2 words
// in canonical slot order.
template <int BITS>
__device__ __forceinline__ void decode8(const Codes<BITS>& w, int g, const ByteTables& t, const uint32_t* tab6,
                                        uint32_t (&out)[4]) {
    uint32_t lo, hi;
    if constexpr (BITS == 6) {
        decode8_lds6(w, g, tab6, out);
    } else if constexpr (BITS == 4) {
        // nibble j of x is the label of code k_j: bits 0-2 index the magnitude table, bit 3 (the
        // sign) becomes bit 7 of the high byte, where bf16 keeps its sign.  The empty asm pins the
        // decode here: otherwise the compiler starts it right after the codes' load, which then
        // has to complete a whole K-step early.
        uint32_t x = w[g];
        asm volatile("" : "+v"(x));
        lookup_bytes(x & 0x07070707u, t, lo, hi);                  // k0 k2 k4 k6
        interleave(lo, hi | ((x << 4) & 0x80808080u), out[0], out[1]);
        lookup_bytes((x >> 4) & 0x07070707u, t, lo, hi);           // k1 k3 k5 k7
        interleave(lo, hi | (x & 0x80808080u), out[2], out[3]);
    } else {
        decode8_small<BITS>(w, g, t, out);
    }
}

template <int BITS>
__device__ __forceinline__ void load_codes32(const uint8_t* src, Codes<BITS>& w) {
    if constexpr (BITS == 4) {
        const uint4 v = *(const uint4*)src;
        w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
    } else if constexpr (BITS == 6) {
        // 24 bytes at an 8-byte aligned offset
        const uint2 a = *(const uint2*)src, b = *(const uint2*)(src + 8), c = *(const uint2*)(src + 16);
        w[0] = a.x; w[1] = a.y; w[2] = b.x; w[3] = b.y; w[4] = c.x; w[5] = c.y;
    } else if constexpr (BITS == 2) {
        const uint2 v = *(const uint2*)src;
        w[0] = v.x; w[1] = v.y; w[2] = 0; w[3] = 0;
    } else {
        const uint32_t* s = (const uint32_t*)src;
        w[0] = s[0]; w[1] = s[1]; w[2] = s[2]; w[3] = 0;
    }
}

__device__ __forceinline__ float bf16_to_f32(uint16_t v) { return __uint_as_float((uint32_t)v << 16); }

__device__ __forceinline__ uint32_t f32_to_bf16_rne(float x) {
    const uint32_t u = __float_as_uint(x);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;  // NaN stays NaN
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// GELU(v) = v * Phi(v), Phi the standard normal CDF, with Phi from the complementary error
// function: Phi(v) = 1 - q for v >= 0 and q for v < 0, q = erfc(|v|/sqrt(2)) / 2.  erfc is the
// Chebyshev-fitted form of Numerical Recipes in C (2nd ed., Sec. 6.2, erfcc): for x >= 0,
//     erfc(x) = t exp(-x^2 + P(t)),  t = 1 / (1 + x/2),  P a degree-9 polynomial,
// with fractional error below 1.2e-7 everywhere, so GELU keeps its relative accuracy in the
// negative tail too.  log2(e) is folded into the coefficients (the hardware exponential is base
// 2) and the factor 1/2 of q into the constant term.  One reciprocal, one exp2 and nine fused
// multiply-adds without branches: on a layer's outputs (|Y| up to a few units) the library erff
// takes several ranges whose branches diverge across a wave.
__device__ __forceinline__ float gelu_erfc(float v) {
    constexpr float L2E = 1.4426950408889634f;
    constexpr float c0 = -1.26551223f * L2E - 1.f, c1 = 1.00002368f * L2E, c2 = 0.37409196f * L2E,
                    c3 = 0.09678418f * L2E, c4 = -0.18628806f * L2E, c5 = 0.27886807f * L2E,
                    c6 = -1.13520398f * L2E, c7 = 1.48851587f * L2E, c8 = -0.82215223f * L2E,
                    c9 = 0.17087277f * L2E;
    const float t = __builtin_amdgcn_rcpf(fmaf(0.35355339059327373f, fabsf(v), 1.f));  // x = |v|/sqrt(2)
    float P = fmaf(t, c9, c8);
    P = fmaf(t, P, c7);
    P = fmaf(t, P, c6);
    P = fmaf(t, P, c5);
    P = fmaf(t, P, c4);
    P = fmaf(t, P, c3);
    P = fmaf(t, P, c2);
    P = fmaf(t, P, c1);
    P = fmaf(t, P, c0);
    const float q = t * __builtin_amdgcn_exp2f(fmaf(v * v, -0.5f * L2E, P));
    return v * (v >= 0.f ? 1.f - q : q);
}

// The rest of the layer after the rescaled contraction: bias, then GELU (x * Phi(x)).
__device__ __forceinline__ float epilogue_value(const GemmParams& p, float v, float bias) {
    v += bias;
    if (p.gelu) v = gelu_erfc(v);
    return v;
}

__device__ __forceinline__ void store_one(const GemmParams& p, int64_t row, int64_t col, float v) {
    if (p.out_bf16)
        ((uint16_t*)p.Y)[row * p.ldy + col] = (uint16_t)f32_to_bf16_rne(v);
    else
        ((float*)p.Y)[row * p.ldy + col] = v;
}

// SPLIT: workgroup z of a K-split contracts K-steps z*steps .. (z+1)*steps - 1 (the last split
// fewer) and stores its raw sums to p.ws[z][M][N]; lut_gemm_reduce applies the epilogue.
//
// 128x128 block tiles, K-step 64, four waves of 64x64.  This kernel serves grids too small for the
// 256x256 kernel (often one workgroup per compute unit, so one wave per SIMD), where each
// workgroup's time is its chain of K-steps: it is pipelined like the large kernel.  The block
// tile's codes are decoded once per K-step into a double-buffered bf16 tile in LDS (74 KB); while
// the matrix cores work on step s, each wave decodes step s+1 into the other stage (groups 0-1,
// 2, 3 in slices 0, 1, 2), fragments are read one 16-wide slice ahead, one barrier per step sits
// before the last slice, and the codes of the next five steps are in flight.
constexpr int SMALL_TILE = BM * LDS_STRIDE;  // halves per operand tile

template <int BA, int BW, bool SPLIT>
__global__ __launch_bounds__(256) void lut_gemm_kernel(GemmParams p) {
    extern __shared__ __align__(16) __bf16 slds[];  // [stage][A, B][128][72], then the 6-bit table
    constexpr int STAGE = 2 * SMALL_TILE;
    uint32_t* const tab6 = (uint32_t*)(slds + 2 * STAGE);  // 6-bit activation levels (bf16 in the low half)
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = (int64_t)blockIdx.y * BM, n0 = (int64_t)blockIdx.x * BN;
    const ByteTables ta = make_tables<BA>(p.lut_a);
    const ByteTables tw = make_tables<BW>(p.lut_w);
    if constexpr (BA == 6) {
        if (tid < 64) tab6[tid] = p.lut_a[tid];
        __syncthreads();
    }

    // this thread decodes 32 codes of one A row and 32 codes of one B row per K-step
    const int lr = tid >> 1, lh = tid & 1;
    const int64_t arow = min(m0 + lr, p.M - 1), brow = min(n0 + lr, p.N - 1);
    const int64_t a_row_bytes = (int64_t)p.K * BA / 8, b_row_bytes = (int64_t)p.K * BW / 8;
    // the K-steps this workgroup contracts
    const int kb = SPLIT ? (int)blockIdx.z * p.split_steps : 0;
    const int nk = SPLIT ? min(p.split_steps, p.K / BK - kb) : p.K / BK;
    const uint8_t* asrc = p.xc + arow * a_row_bytes + lh * 4 * BA + (int64_t)kb * (BK * BA / 8);
    const uint8_t* bsrc = p.wc + brow * b_row_bytes + lh * 4 * BW + (int64_t)kb * (BK * BW / 8);

    floatx16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    const int64_t astep = BK * BA / 8, bstep = BK * BW / 8;
    __bf16* const a_dst0 = slds + lr * LDS_STRIDE + lh * 32;  // this thread's decode slots, stage 0
    const __bf16* const a_frag0 = slds + (wm * 64 + (lane & 31)) * LDS_STRIDE + (lane >> 5) * 8;
    const __bf16* const b_frag0 = slds + SMALL_TILE + (wn * 64 + (lane & 31)) * LDS_STRIDE + (lane >> 5) * 8;

    auto decode_group = [&](int stage, int g, const Codes<BA>& ca, const Codes<BW>& cb) {
        uint32_t da[4], db[4];
        decode8<BA>(ca, g, ta, tab6, da);
        decode8<BW>(cb, g, tw, nullptr, db);
        *(uint4*)(a_dst0 + stage + 8 * g) = make_uint4(da[0], da[1], da[2], da[3]);
        *(uint4*)(a_dst0 + stage + SMALL_TILE + 8 * g) = make_uint4(db[0], db[1], db[2], db[3]);
    };

    // a ring of RING code register sets: set u holds the codes of the steps congruent to u, so
    // each load has RING - 1 K-steps to land (a workgroup here is often alone on its compute unit,
    // with nothing else to cover the memory latency)
    constexpr int RING = 6;
    Codes<BA> ca[RING];
    Codes<BW> cb[RING];
    load_codes32<BA>(asrc, ca[0]);
    load_codes32<BW>(bsrc, cb[0]);
#pragma unroll
    for (int g = 0; g < 4; ++g) decode_group(0, g, ca[0], cb[0]);
#pragma unroll
    for (int u = 1; u < RING; ++u) {
        const int64_t su = min(u, nk - 1);
        load_codes32<BA>(asrc + su * astep, ca[u]);
        load_codes32<BW>(bsrc + su * bstep, cb[u]);
    }
    __syncthreads();

    // fragments of one 16-wide k slice of a stage
    bf16x8 a[2][2], b[2][2];
    auto read_frags = [&](int stage, int kk, bf16x8 (&af)[2], bf16x8 (&bf)[2]) {
#pragma unroll
        for (int i = 0; i < 2; ++i) af[i] = *(const bf16x8*)(a_frag0 + stage + i * 32 * LDS_STRIDE + kk * 16);
#pragma unroll
        for (int j = 0; j < 2; ++j) bf[j] = *(const bf16x8*)(b_frag0 + stage + j * 32 * LDS_STRIDE + kk * 16);
    };
    read_frags(0, 0, a[0], b[0]);

    // as the large kernel's K-step: decode step s+1 (codes ca, cb) in slices 0-2, barrier before
    // slice 3, whose MFMAs overlap the next step's first fragments; the codes of step s+RING load
    // into (na, nb), the set step s came from
    auto kstep = [&](int s, const Codes<BA>& ca, const Codes<BW>& cb, Codes<BA>& na, Codes<BW>& nb) {
        // the last steps re-load the final step's codes; they are never used
        const int64_t sl = min(s + RING, nk - 1);
        load_codes32<BA>(asrc + sl * astep, na);
        load_codes32<BW>(bsrc + sl * bstep, nb);
        __builtin_amdgcn_sched_barrier(0);

        const int cur = (s & 1) * STAGE, nxt = STAGE - cur;
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
            const int f = kk & 1;
            if (kk == 3) __syncthreads();
            if (kk < 3) read_frags(cur, kk + 1, a[f ^ 1], b[f ^ 1]);
            else read_frags(nxt, 0, a[f ^ 1], b[f ^ 1]);
            if (kk == 0) {
                decode_group(nxt, 0, ca, cb);
                decode_group(nxt, 1, ca, cb);
            } else if (kk < 3) {
                decode_group(nxt, kk + 1, ca, cb);
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[f][j], a[f][i], acc[i][j], 0, 0, 0);
            // next fragments first, then each MFMA followed by a share of the decode, the decoded
            // rows' LDS writes last
            __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
            if (kk == 0) {
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x002, 15, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x200, 4, 0);
            } else if (kk < 3) {
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x200, 2, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // step s + u decodes set (u + 1) % RING and refills set u; unrolled by RING so that every set
    // index is a constant (registers, none copied)
    int s = 0;
    for (; s + RING - 1 < nk; s += RING) {
#pragma unroll
        for (int u = 0; u < RING; ++u) kstep(s + u, ca[(u + 1) % RING], cb[(u + 1) % RING], ca[u], cb[u]);
    }
#pragma unroll
    for (int u = 0; u < RING - 1; ++u)
        if (s + u < nk) kstep(s + u, ca[(u + 1) % RING], cb[(u + 1) % RING], ca[u], cb[u]);

    // epilogue.  As in the large kernel, the MFMAs computed the transposed tile: element e of
    // accumulator (i, j) belongs to row i*32 + lane%32 and column j*32 + 8*(e/4) + 4*(lane/32) + e%4,
    // so each lane holds runs of four consecutive columns of one row and stores each run as one
    // vector.  Every load comes before the first store (as far as the compiler knows, Y may alias
    // xn, wn or the bias, and a wait placed among the stores would make each store wait for the
    // one before).
    const int64_t col0 = n0 + wn * 64 + 4 * (lane >> 5);
    // With a multiple of 4 columns (and, for Y, rows that allow 4-wide stores) the outputs go
    // through LDS, free after the main loop, so that each store covers 4 rows of contiguous bytes
    // (256 of fp32, 128 of bf16) instead of 32 rows of 16 or 8: each wave writes its 64 x 64
    // sub-tile into a region of its own (68 floats or 72 bf16 per row, padding that keeps the
    // accesses conflict-free) and reads it back by rows.
    constexpr int TS = 68, TSB = 72;
    float* const tl = (float*)slds + wave * (64 * TS);
    uint16_t* const tlb = (uint16_t*)tl;
    const int64_t colg = n0 + wn * 64 + 4 * (lane & 15);
    if constexpr (SPLIT) {
        float* const ws = p.ws + (int64_t)blockIdx.z * p.M * p.N;
        const bool vec = (p.N & 3) == 0;
        if (vec) {
            __syncthreads();   // every wave is done reading the stages
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        *(float4*)(tl + (i * 32 + (lane & 31)) * TS + j * 32 + 8 * q + 4 * (lane >> 5)) =
                            make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
#pragma unroll
            for (int t = 0; t < 16; ++t) {
                const int r = 4 * t + (lane >> 4);
                const int64_t row = m0 + wm * 64 + r;
                const float4 v = *(const float4*)(tl + r * TS + 4 * (lane & 15));
                if (row < p.M && colg < p.N) *(float4*)(ws + row * p.N + colg) = v;
            }
            return;
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int64_t row = m0 + wm * 64 + i * 32 + (lane & 31);
            if (row >= p.M) continue;
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int64_t c = col0 + j * 32 + 8 * q;
                    float* const dst = ws + row * p.N + c;
                    if (vec && c + 3 < p.N) {
                        *(float4*)dst = make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                                    acc[i][j][4 * q + 3]);
                    } else {
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            if (c + r < p.N) dst[r] = acc[i][j][4 * q + r];
                    }
                }
        }
        return;
    }
    float xsv[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int64_t row = m0 + wm * 64 + i * 32 + (lane & 31);
        xsv[i] = row < p.M ? p.xn[row] : 0.f;
    }
    uint2 rwv[2][4], bv[2][4];  // bf16 r' and bias of the lane's columns, four per (j, run)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t c = col0 + j * 32 + 8 * q;
            if (c + 3 < p.N && p.vec4) {
                rwv[j][q] = *(const uint2*)(p.wn + c);
                bv[j][q] = p.bias ? *(const uint2*)(p.bias + c) : make_uint2(0u, 0u);
            } else {
                uint16_t v[4], w[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    v[r] = c + r < p.N ? p.wn[c + r] : (uint16_t)0;
                    w[r] = p.bias && c + r < p.N ? p.bias[c + r] : (uint16_t)0;
                }
                rwv[j][q] = make_uint2(v[0] | ((uint32_t)v[1] << 16), v[2] | ((uint32_t)v[3] << 16));
                bv[j][q] = make_uint2(w[0] | ((uint32_t)w[1] << 16), w[2] | ((uint32_t)w[3] << 16));
            }
        }
    // every output value first, then the stores
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint2 rw = rwv[j][q], bb = bv[j][q];
                const float r4[4] = {__uint_as_float(rw.x << 16), __uint_as_float(rw.x & 0xFFFF0000u),
                                     __uint_as_float(rw.y << 16), __uint_as_float(rw.y & 0xFFFF0000u)};
                const float b4[4] = {__uint_as_float(bb.x << 16), __uint_as_float(bb.x & 0xFFFF0000u),
                                     __uint_as_float(bb.y << 16), __uint_as_float(bb.y & 0xFFFF0000u)};
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    acc[i][j][4 * q + r] = epilogue_value(p, acc[i][j][4 * q + r] * xsv[i] * r4[r], b4[r]);
            }
    if (p.vec4 && (p.N & 3) == 0) {
        __syncthreads();   // every wave is done reading the stages
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int lrow = i * 32 + (lane & 31), lcol = j * 32 + 8 * q + 4 * (lane >> 5);
                    const float v[4] = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
                    if (p.out_bf16)
                        *(uint2*)(tlb + lrow * TSB + lcol) =
                            make_uint2(f32_to_bf16_rne(v[0]) | (f32_to_bf16_rne(v[1]) << 16),
                                       f32_to_bf16_rne(v[2]) | (f32_to_bf16_rne(v[3]) << 16));
                    else
                        *(float4*)(tl + lrow * TS + lcol) = make_float4(v[0], v[1], v[2], v[3]);
                }
#pragma unroll
        for (int t = 0; t < 16; ++t) {
            const int r = 4 * t + (lane >> 4);
            const int64_t row = m0 + wm * 64 + r;
            if (p.out_bf16) {
                const uint2 v = *(const uint2*)(tlb + r * TSB + 4 * (lane & 15));
                if (row < p.M && colg < p.N) *(uint2*)((uint16_t*)p.Y + row * p.ldy + colg) = v;
            } else {
                const float4 v = *(const float4*)(tl + r * TS + 4 * (lane & 15));
                if (row < p.M && colg < p.N) *(float4*)((float*)p.Y + row * p.ldy + colg) = v;
            }
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int64_t row = m0 + wm * 64 + i * 32 + (lane & 31);
        if (row >= p.M) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int64_t c = col0 + j * 32 + 8 * q;
                const float v[4] = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
                const bool full = c + 3 < p.N && p.vec4;
                if (full && p.out_bf16) {
                    *(uint2*)((uint16_t*)p.Y + row * p.ldy + c) =
                        make_uint2(f32_to_bf16_rne(v[0]) | (f32_to_bf16_rne(v[1]) << 16),
                                   f32_to_bf16_rne(v[2]) | (f32_to_bf16_rne(v[3]) << 16));
                } else if (full) {
                    *(float4*)((float*)p.Y + row * p.ldy + c) = make_float4(v[0], v[1], v[2], v[3]);
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (c + r < p.N) store_one(p, row, c + r, v[r]);
                }
            }
    }
}

// ------------------------------------------------------------------------------------------
// Large-problem kernel: 256x256 block tiles, K-step 64, eight waves of 128x64 each.  Every code
// of a block tile is decoded once per K-step into a double-buffered bf16 tile in LDS (147 KB),
// which halves the decodes per flop of the 128x128 kernel.  While the matrix cores work on step
// s, each wave decodes step s+1 into the other stage, a quarter per 16-wide k slice, and the
// codes of steps s+2 and s+3 are in flight.  Block tiles are visited so that the
// workgroups resident on one XCD (round-robin dispatch) share A and B panels in that XCD's L2.
constexpr int BM2 = 256, BN2 = 256, BK2 = 64;
constexpr int LDS2_STRIDE = BK2 + 8;                  // halves per tile row; 144 B keeps 16-byte
                                                      // fragment reads of 16 rows conflict-free
constexpr int LDS2_TILE = BM2 * LDS2_STRIDE;          // halves per operand tile
constexpr int GROUP_M = 8;                            // block rows per L2 group

template <int BA, int BW>
__global__ __launch_bounds__(512, 2) void lut_gemm_big(GemmParams p, int ntm, int ntn, int per_xcd) {
    extern __shared__ __align__(16) __bf16 lds[];  // [stage][A, B][256][72]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 2, wn = wave & 3;

    // XCD-aware tile order: workgroup pid runs on XCD pid % 8; consecutive ids per XCD
    const int pid = blockIdx.x;
    const int nid = (pid & 7) * per_xcd + (pid >> 3);
    const int total = ntm * ntn;
    if (nid >= total) return;
    const int in_group = GROUP_M * ntn;
    const int first_m = (nid / in_group) * GROUP_M;
    const int gsize = min(ntm - first_m, GROUP_M);
    const int tm = first_m + (nid % in_group) % gsize;
    const int tn = (nid % in_group) / gsize;
    const int64_t m0 = (int64_t)tm * BM2, n0 = (int64_t)tn * BN2;

    const ByteTables ta = make_tables<BA>(p.lut_a);
    const ByteTables tw = make_tables<BW>(p.lut_w);
    uint32_t* const tab6 = (uint32_t*)(lds + 2 * 2 * LDS2_TILE);  // 6-bit levels, after the tiles
    if constexpr (BA == 6) {
        if (tid < 64) tab6[tid] = p.lut_a[tid];
        __syncthreads();
    }

    // this thread decodes 32 codes of one A row and 32 codes of one B row per K-step
    const int lr = tid >> 1, lh = tid & 1;
    const int64_t arow = min(m0 + lr, p.M - 1), brow = min(n0 + lr, p.N - 1);
    const uint8_t* asrc = p.xc + arow * ((int64_t)p.K * BA / 8) + lh * 4 * BA;
    const uint8_t* bsrc = p.wc + brow * ((int64_t)p.K * BW / 8) + lh * 4 * BW;

    floatx16 acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    const int nk = p.K / BK2;
    const int64_t astep = BK2 * BA / 8, bstep = BK2 * BW / 8;
    __bf16* const a_dst0 = lds + lr * LDS2_STRIDE + lh * 32;  // this thread's decode slots, stage 0
    const __bf16* const a_frag0 = lds + (wm * 128 + (lane & 31)) * LDS2_STRIDE + (lane >> 5) * 8;
    const __bf16* const b_frag0 = lds + LDS2_TILE + (wn * 64 + (lane & 31)) * LDS2_STRIDE + (lane >> 5) * 8;
    constexpr int STAGE = 2 * LDS2_TILE;

    Codes<BA> wa, xa, ya;
    Codes<BW> wb, xb, yb;
    load_codes32<BA>(asrc, wa);
    load_codes32<BW>(bsrc, wb);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        uint32_t da[4], db[4];
        decode8<BA>(wa, g, ta, tab6, da);
        decode8<BW>(wb, g, tw, nullptr, db);
        *(uint4*)(a_dst0 + 8 * g) = make_uint4(da[0], da[1], da[2], da[3]);
        *(uint4*)(a_dst0 + LDS2_TILE + 8 * g) = make_uint4(db[0], db[1], db[2], db[3]);
    }
    {
        const int64_t s1 = nk > 1 ? 1 : 0, s2 = nk > 2 ? 2 : nk - 1;
        load_codes32<BA>(asrc + s1 * astep, wa);
        load_codes32<BW>(bsrc + s1 * bstep, wb);
        load_codes32<BA>(asrc + s2 * astep, ya);
        load_codes32<BW>(bsrc + s2 * bstep, yb);
    }
    __syncthreads();

    // fragments of one 16-wide k slice of a stage
    bf16x8 a[2][4], b[2][2];
    auto read_frags = [&](int stage, int kk, bf16x8 (&af)[4], bf16x8 (&bf)[2]) {
#pragma unroll
        for (int i = 0; i < 4; ++i) af[i] = *(const bf16x8*)(a_frag0 + stage + i * 32 * LDS2_STRIDE + kk * 16);
#pragma unroll
        for (int j = 0; j < 2; ++j) bf[j] = *(const bf16x8*)(b_frag0 + stage + j * 32 * LDS2_STRIDE + kk * 16);
    };
    auto decode_group = [&](int nxt, int g, const Codes<BA>& ca, const Codes<BW>& cb) {
        uint32_t da[4], db[4];
        decode8<BA>(ca, g, ta, tab6, da);
        decode8<BW>(cb, g, tw, nullptr, db);
        *(uint4*)(a_dst0 + nxt + 8 * g) = make_uint4(da[0], da[1], da[2], da[3]);
        *(uint4*)(a_dst0 + nxt + LDS2_TILE + 8 * g) = make_uint4(db[0], db[1], db[2], db[3]);
    };
    read_frags(0, 0, a[0], b[0]);

    // One K-step in four 16-wide slices.  Slices 0-2 decode the codes of step s+1 (ca, cb) into
    // the other stage while their MFMAs run; then one barrier makes that stage complete and
    // retires every read of this step's stage, so slice 3 can already fetch the next step's
    // first fragments while its MFMAs run.  The codes of step s+3 load into (na, nb), so each
    // load has two K-steps to land.  Three register sets rotate: the loop below is unrolled by
    // three so that they change roles instead of being copied (a copy would wait for the load).
    auto kstep = [&](int s, const Codes<BA>& ca, const Codes<BW>& cb, Codes<BA>& na, Codes<BW>& nb) {
        // the last steps re-load the final step's codes; they are never used
        const int64_t s2 = min(s + 3, nk - 1);
        load_codes32<BA>(asrc + s2 * astep, na);
        load_codes32<BW>(bsrc + s2 * bstep, nb);
        __builtin_amdgcn_sched_barrier(0);

        const int cur = (s & 1) * STAGE, nxt = STAGE - cur;
#pragma unroll
        for (int kk = 0; kk < BK2 / 16; ++kk) {
            const int f = kk & 1;
            if (kk == 3) __syncthreads();
            // next slice's fragments; after the barrier, the next step's first slice (on the final
            // step a refilled stage nobody uses)
            if (kk < 3) read_frags(cur, kk + 1, a[f ^ 1], b[f ^ 1]);
            else read_frags(nxt, 0, a[f ^ 1], b[f ^ 1]);
            // decode groups 0,1 | 2 | 3 | - of the next step in slices 0 | 1 | 2 | 3
            if (kk == 0) {
                decode_group(nxt, 0, ca, cb);
                decode_group(nxt, 1, ca, cb);
            } else if (kk < 3) {
                decode_group(nxt, kk + 1, ca, cb);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[f][j], a[f][i], acc[i][j], 0, 0, 0);
            // issue order inside the slice: next fragments first, then each MFMA followed by a
            // share of the decode, the decoded rows' LDS writes last
            __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
            if (kk == 0) {
#pragma unroll
                for (int m = 0; m < 8; ++m) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x002, 10, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x200, 4, 0);
            } else if (kk < 3) {
#pragma unroll
                for (int m = 0; m < 8; ++m) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x200, 2, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    int s = 0;
    for (; s + 2 < nk; s += 3) {
        kstep(s, wa, wb, xa, xb);
        kstep(s + 1, ya, yb, wa, wb);
        kstep(s + 2, xa, xb, ya, yb);
    }
    if (s < nk) kstep(s, wa, wb, xa, xb);
    if (s + 1 < nk) kstep(s + 1, ya, yb, wa, wb);

    // epilogue.  The MFMAs computed the transposed tile, so element e of accumulator (i, j)
    // belongs to row i*32 + lane%32 and column j*32 + 8*(e/4) + 4*(lane/32) + e%4: each lane
    // holds runs of four consecutive columns of one row and stores them as one vector (16 bytes
    // of fp32 or 8 of bf16).
    const int64_t col0 = n0 + wn * 64 + 4 * (lane >> 5);
    uint2 rwv[2][4];  // bf16 r' of the lane's columns, four per (j, run)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t c = col0 + j * 32 + 8 * q;
            if (c + 3 < p.N && p.vec4) {
                rwv[j][q] = *(const uint2*)(p.wn + c);
            } else {
                uint16_t v[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = c + r < p.N ? p.wn[c + r] : (uint16_t)0;
                rwv[j][q] = make_uint2(v[0] | ((uint32_t)v[1] << 16), v[2] | ((uint32_t)v[3] << 16));
            }
        }
    const bool plain = !p.bias && !p.gelu && !p.out_bf16;
    // bf16 bias of the lane's columns, loaded once for its four rows (zero without a bias)
    uint2 bv[2][4];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t c = col0 + j * 32 + 8 * q;
            if (p.bias && c + 3 < p.N && p.vec4) {
                bv[j][q] = *(const uint2*)(p.bias + c);
            } else {
                uint16_t v[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = p.bias && c + r < p.N ? p.bias[c + r] : (uint16_t)0;
                bv[j][q] = make_uint2(v[0] | ((uint32_t)v[1] << 16), v[2] | ((uint32_t)v[3] << 16));
            }
        }
    // the lane's four row norms before the first store (Y may alias xn as far as the compiler
    // knows, so a load after a store would wait for it)
    float xsv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t row = m0 + wm * 128 + i * 32 + (lane & 31);
        xsv[i] = row < p.M ? p.xn[row] : 0.f;
    }
    // Rows that allow 4-wide stores (and a multiple of 4 columns): the finished outputs go through
    // LDS (free after the main loop) so that each store covers 4 rows of contiguous bytes (256 of
    // fp32, 128 of bf16) instead of 32 rows of 16 or 8 bytes.  Each wave owns a region of 64 rows
    // (68 floats or 72 bf16 per row, padding that keeps the accesses conflict-free) and turns its
    // 128 x 64 sub-tile around in two halves; a wave's LDS accesses run in order, so the halves
    // reuse the region without a barrier.
    if (p.vec4 && (p.N & 3) == 0) {
        __syncthreads();   // every wave is done reading the stages
        constexpr int TS = 68, TSB = 72;
        float* const tl = (float*)lds + wave * (64 * TS);
        uint16_t* const tlb = (uint16_t*)tl;
        const int64_t colg = n0 + wn * 64 + 4 * (lane & 15);
#pragma unroll
        for (int half = 0; half < 2; ++half) {
#pragma unroll
            for (int ii = 0; ii < 2; ++ii) {
                const int i = 2 * half + ii;
                const float xs = xsv[i];
                const int lrow = ii * 32 + (lane & 31);
#pragma unroll
                for (int j = 0; j < 2; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const uint2 rw = rwv[j][q];
                        float v[4] = {acc[i][j][4 * q + 0] * xs * __uint_as_float(rw.x << 16),
                                      acc[i][j][4 * q + 1] * xs * __uint_as_float(rw.x & 0xFFFF0000u),
                                      acc[i][j][4 * q + 2] * xs * __uint_as_float(rw.y << 16),
                                      acc[i][j][4 * q + 3] * xs * __uint_as_float(rw.y & 0xFFFF0000u)};
                        const int lcol = j * 32 + 8 * q + 4 * (lane >> 5);
                        if (!plain) {
                            const uint2 b = bv[j][q];
                            v[0] = epilogue_value(p, v[0], __uint_as_float(b.x << 16));
                            v[1] = epilogue_value(p, v[1], __uint_as_float(b.x & 0xFFFF0000u));
                            v[2] = epilogue_value(p, v[2], __uint_as_float(b.y << 16));
                            v[3] = epilogue_value(p, v[3], __uint_as_float(b.y & 0xFFFF0000u));
                        }
                        if (p.out_bf16)
                            *(uint2*)(tlb + lrow * TSB + lcol) =
                                make_uint2(f32_to_bf16_rne(v[0]) | (f32_to_bf16_rne(v[1]) << 16),
                                           f32_to_bf16_rne(v[2]) | (f32_to_bf16_rne(v[3]) << 16));
                        else
                            *(float4*)(tl + lrow * TS + lcol) = make_float4(v[0], v[1], v[2], v[3]);
                    }
            }
#pragma unroll
            for (int t = 0; t < 16; ++t) {
                const int r = 4 * t + (lane >> 4);
                const int64_t row = m0 + wm * 128 + 64 * half + r;
                if (p.out_bf16) {
                    const uint2 v = *(const uint2*)(tlb + r * TSB + 4 * (lane & 15));
                    if (row < p.M && colg < p.N) *(uint2*)((uint16_t*)p.Y + row * p.ldy + colg) = v;
                } else {
                    const float4 v = *(const float4*)(tl + r * TS + 4 * (lane & 15));
                    if (row < p.M && colg < p.N) *(float4*)((float*)p.Y + row * p.ldy + colg) = v;
                }
            }
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t row = m0 + wm * 128 + i * 32 + (lane & 31);
        if (row >= p.M) continue;
        const float xs = xsv[i];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int64_t c = col0 + j * 32 + 8 * q;
                const uint2 rw = rwv[j][q];
                float v[4] = {acc[i][j][4 * q + 0] * xs * __uint_as_float(rw.x << 16),
                              acc[i][j][4 * q + 1] * xs * __uint_as_float(rw.x & 0xFFFF0000u),
                              acc[i][j][4 * q + 2] * xs * __uint_as_float(rw.y << 16),
                              acc[i][j][4 * q + 3] * xs * __uint_as_float(rw.y & 0xFFFF0000u)};
                const bool full = c + 3 < p.N && p.vec4;
                if (plain && full) {
                    *(float4*)((float*)p.Y + row * p.ldy + c) = make_float4(v[0], v[1], v[2], v[3]);
                    continue;
                }
                if (!plain) {
                    const uint2 b = bv[j][q];
                    v[0] = epilogue_value(p, v[0], __uint_as_float(b.x << 16));
                    v[1] = epilogue_value(p, v[1], __uint_as_float(b.x & 0xFFFF0000u));
                    v[2] = epilogue_value(p, v[2], __uint_as_float(b.y << 16));
                    v[3] = epilogue_value(p, v[3], __uint_as_float(b.y & 0xFFFF0000u));
                }
                if (full && p.out_bf16) {
                    *(uint2*)((uint16_t*)p.Y + row * p.ldy + c) =
                        make_uint2(f32_to_bf16_rne(v[0]) | (f32_to_bf16_rne(v[1]) << 16),
                                   f32_to_bf16_rne(v[2]) | (f32_to_bf16_rne(v[3]) << 16));
                } else if (full) {
                    *(float4*)((float*)p.Y + row * p.ldy + c) = make_float4(v[0], v[1], v[2], v[3]);
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (c + r < p.N) store_one(p, row, c + r, v[r]);
                }
            }
        }
    }
}

template <int BA, int BW>
hipError_t launch_big(const GemmParams& p, hipStream_t stream) {
    static std::atomic<uint64_t> attr{0};
    const size_t smem = (size_t)2 * 2 * LDS2_TILE * sizeof(__bf16) + (BA == 6 ? 64 * sizeof(uint32_t) : 0);
    const hipError_t e = raise_lds_limit((const void*)lut_gemm_big<BA, BW>, (int)smem, attr);
    if (e != hipSuccess) return e;
    const int ntm = (int)((p.M + BM2 - 1) / BM2), ntn = (int)((p.N + BN2 - 1) / BN2);
    const int per_xcd = (ntm * ntn + 7) / 8;
    hipLaunchKernelGGL((lut_gemm_big<BA, BW>), dim3(per_xcd * 8), dim3(512), smem, stream, p, ntm, ntn, per_xcd);
    return hipGetLastError();
}

// The K-splits' sums in split order (deterministic), rescaled and through the layer epilogue:
// one thread per four consecutive outputs of a row.
__global__ __launch_bounds__(256) void lut_gemm_reduce(GemmParams p, int splits) {
    const int64_t nq = (p.N + 3) / 4;
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= p.M * nq) return;
    const int64_t row = t / nq, c0 = (t - row * nq) * 4;
    const float xs = p.xn[row];
    if (p.vec4 && (p.N & 3) == 0) {
        // whole runs of four, 16-byte aligned in the workspace and in Y: vector loads and stores
        const int64_t plane = p.M * p.N;
        const float* src = p.ws + row * p.N + c0;
        float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int z = 0; z < splits; ++z) {
            const float4 b = *(const float4*)(src + z * plane);
            a.x += b.x;
            a.y += b.y;
            a.z += b.z;
            a.w += b.w;
        }
        const uint2 rw = *(const uint2*)(p.wn + c0);
        const uint2 bb = p.bias ? *(const uint2*)(p.bias + c0) : make_uint2(0u, 0u);
        float v[4] = {a.x * xs * __uint_as_float(rw.x << 16), a.y * xs * __uint_as_float(rw.x & 0xFFFF0000u),
                      a.z * xs * __uint_as_float(rw.y << 16), a.w * xs * __uint_as_float(rw.y & 0xFFFF0000u)};
        v[0] = epilogue_value(p, v[0], __uint_as_float(bb.x << 16));
        v[1] = epilogue_value(p, v[1], __uint_as_float(bb.x & 0xFFFF0000u));
        v[2] = epilogue_value(p, v[2], __uint_as_float(bb.y << 16));
        v[3] = epilogue_value(p, v[3], __uint_as_float(bb.y & 0xFFFF0000u));
        if (p.out_bf16)
            *(uint2*)((uint16_t*)p.Y + row * p.ldy + c0) =
                make_uint2(f32_to_bf16_rne(v[0]) | (f32_to_bf16_rne(v[1]) << 16),
                           f32_to_bf16_rne(v[2]) | (f32_to_bf16_rne(v[3]) << 16));
        else
            *(float4*)((float*)p.Y + row * p.ldy + c0) = make_float4(v[0], v[1], v[2], v[3]);
        return;
    }
    const int nc = (int)min((int64_t)4, p.N - c0);
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    for (int z = 0; z < splits; ++z) {
        const float* src = p.ws + (int64_t)z * p.M * p.N + row * p.N + c0;
#pragma unroll
        for (int r = 0; r < 4; ++r)
            if (r < nc) v[r] += src[r];
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        if (r >= nc) continue;
        const int64_t col = c0 + r;
        const float out = epilogue_value(p, v[r] * xs * bf16_to_f32(p.wn[col]), p.bias ? bf16_to_f32(p.bias[col]) : 0.f);
        store_one(p, row, col, out);
    }
}

template <int BA, int BW>
hipError_t launch_small(const GemmParams& p, hipStream_t stream) {
    dim3 grid((unsigned)((p.N + BN - 1) / BN), (unsigned)((p.M + BM - 1) / BM));
    const size_t smem = (size_t)2 * 2 * SMALL_TILE * sizeof(__bf16) + (BA == 6 ? 64 * sizeof(uint32_t) : 0);
    static std::atomic<uint64_t> attr_split{0}, attr_whole{0};
    if (p.ws && p.splits > 1) {
        const hipError_t ea = raise_lds_limit((const void*)lut_gemm_kernel<BA, BW, true>, (int)smem, attr_split);
        if (ea != hipSuccess) return ea;
        grid.z = (unsigned)p.splits;
        hipLaunchKernelGGL((lut_gemm_kernel<BA, BW, true>), grid, dim3(256), smem, stream, p);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int64_t threads = p.M * ((p.N + 3) / 4);
        hipLaunchKernelGGL(lut_gemm_reduce, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream, p, p.splits);
        return hipGetLastError();
    }
    const hipError_t ew = raise_lds_limit((const void*)lut_gemm_kernel<BA, BW, false>, (int)smem, attr_whole);
    if (ew != hipSuccess) return ew;
    hipLaunchKernelGGL((lut_gemm_kernel<BA, BW, false>), grid, dim3(256), smem, stream, p);
    return hipGetLastError();
}

// Rows m0 .. M-1 of the layer as a layer of their own (operands and output shifted by m0 rows).
inline GemmParams rows_from(const GemmParams& p, int64_t m0, int ba) {
    GemmParams q = p;
    q.xc = p.xc + m0 * ((int64_t)p.K * ba / 8);
    q.xn = p.xn + m0;
    q.Y = (char*)p.Y + m0 * p.ldy * (p.out_bf16 ? 2 : 4);
    q.M = p.M - m0;
    return q;
}

template <int BA, int BW>
hipError_t launch_one(const GemmParams& p, hipStream_t stream, int cus) {
    const int64_t m_big = lut_gemm_big_rows(p.M, p.N, cus);
    if (m_big == 0) return launch_small<BA, BW>(p, stream);
    if (m_big == p.M) return launch_big<BA, BW>(p, stream);
    GemmParams head = p;
    head.M = m_big;
    hipError_t e = launch_big<BA, BW>(head, stream);
    if (e != hipSuccess) return e;
    return launch_small<BA, BW>(rows_from(p, m_big, BA), stream);
}

}  // namespace

int64_t lut_gemm_big_rows(int64_t M, int64_t N, int cus) {
    // the large kernel from one 256x256 tile per compute unit up (measured: at 432 tiles on 256
    // compute units it beats the 128x128 kernel by a quarter, despite its half-empty second round)
    const int64_t ntm = (M + BM2 - 1) / BM2, ntn = (N + BN2 - 1) / BN2, tiles = ntm * ntn;
    if (tiles < (int64_t)cus) return 0;
    // Wave quantization: the large kernel runs one tile per compute unit at a time, so a last round
    // that is only partly full costs as long as a full one (c4's down-projection: 2600 tiles, an
    // eleventh round of 40).  When that pays, the large kernel takes the tile rows that fill its
    // full rounds and the 128x128 kernel the rest.  A round of those does a quarter of a large
    // tile's work per workgroup but, with one workgroup per compute unit, is latency-bound and
    // takes 0.6-0.8 of a large round (c4's down-projection: 4.61 -> 4.53 ms; the up-projection,
    // whose last round is 42% full, is left alone).
    const int64_t rows_big = (tiles / cus) * cus / ntn;
    if (rows_big > 0 && rows_big < ntm) {
        const int64_t m0 = rows_big * BM2;
        const int64_t small_wgs = ((M - m0 + BM - 1) / BM) * ((N + BN - 1) / BN);
        const double whole = (double)((tiles + cus - 1) / cus);
        const double split = (double)((rows_big * ntn + cus - 1) / cus) + 0.6 * (double)((small_wgs + cus - 1) / cus);
        if (split + 0.1 < whole) return m0;
    }
    return M;
}

int lut_gemm_small_splits(int64_t M, int64_t N, int64_t K, int cus, int* split_steps) {
    const int nk = (int)(K / BK);
    *split_steps = nk;
    // The 128x128 workgroups are each one K-step chain that is latency-bound.  The count of splits
    // minimises an estimate of the busiest compute unit's time, in K-steps: k co-resident
    // workgroups of `steps` K-steps take w(k) * steps (measured on 256 compute units: 1, 1.66 and
    // 2.58 for k = 1, 2, 3, then about 0.86 k), plus the partial sums' round trip through the
    // workspace at about 7 MB per K-step's time.  At least 4 K-steps per split, at most 64 splits.
    const int64_t wgs = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
    auto busiest = [&](int splits, int steps) {
        const int64_t k = (wgs * splits + cus - 1) / cus;
        return (k == 1 ? 1.0 : k == 2 ? 1.66 : k == 3 ? 2.58 : 0.86 * (double)k) * steps;
    };
    int best_splits = 1, best_steps = nk;
    double best = busiest(1, nk);
    for (int s = 2; s <= std::min(64, nk / 4); ++s) {
        const int steps = (nk + s - 1) / s, splits = (nk + steps - 1) / steps;
        const double cost = busiest(splits, steps) + (double)splits * (double)M * (double)N * 8.0 / 7.0e6;
        if (cost < best) {
            best = cost;
            best_splits = splits;
            best_steps = steps;
        }
    }
    *split_steps = best_steps;
    return best_splits;
}

hipError_t launch_lut_gemm(const GemmParams& p, int ba, int bw, int cus, hipStream_t stream) {
    switch (ba * 8 + bw) {
        case 2 * 8 + 2: return launch_one<2, 2>(p, stream, cus);
        case 2 * 8 + 3: return launch_one<2, 3>(p, stream, cus);
        case 2 * 8 + 4: return launch_one<2, 4>(p, stream, cus);
        case 3 * 8 + 2: return launch_one<3, 2>(p, stream, cus);
        case 3 * 8 + 3: return launch_one<3, 3>(p, stream, cus);
        case 3 * 8 + 4: return launch_one<3, 4>(p, stream, cus);
        case 6 * 8 + 2: return launch_one<6, 2>(p, stream, cus);
        case 6 * 8 + 3: return launch_one<6, 3>(p, stream, cus);
        case 6 * 8 + 4: return launch_one<6, 4>(p, stream, cus);
        case 4 * 8 + 2: return launch_one<4, 2>(p, stream, cus);
        case 4 * 8 + 3: return launch_one<4, 3>(p, stream, cus);
        default: return launch_one<4, 4>(p, stream, cus);
    }
}

}  // namespace orbit
