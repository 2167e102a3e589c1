// Fused RPBH rotate -> normalize -> Lloyd-Max encode -> pack for the common case of the
// activation quantizer and the offline weight pass: a permutation plan with Hadamard blocks of
// h = 128 .. 1024 and rows of K = 1024 .. 16384 inputs (a multiple of 128 and of h), on gfx950.
//
// One workgroup holds one row at a time and walks rows persistently (row w, w + G, ...).  Every
// lane transforms 16 post-permutation positions, so a 128-block belongs to eight consecutive lanes
// and a row to K/16 lanes; holding 16 values instead of 32 keeps the register count low enough for
// about twice the resident waves of a 32-value layout, which is what hides the latency of the
// staging loads and the permutation gather.
//
// Per iteration (row g):
//   gather    16 ds_read_u16 through loop-invariant per-lane byte offsets (the permutation) from
//             the row staged in LDS; one v_perm pairs two halves per bf16 pair;
//   stage     the next row streams from HBM straight into the other half of a double-buffered
//             staging area (global_load_lds_dwordx4, no registers, non-temporal), so one barrier
//             per iteration suffices;
//   H_4       the first two butterfly stages of each quad of positions, with the Rademacher signs
//             of Eq. (9) folded in, as six v_dot2_f32_bf16 (bf16 pairs against per-lane sign pairs
//             with neg_lo / neg_hi modifiers; the radix-4 form uses the first stage's result as the
//             accumulator of the second): 1.5 ops per element for two stages, exact products;
//   norm      half a v_dot2 per element (each pair against itself), summed over the 8 lanes of a
//             block by DPP and over the row's blocks through LDS (the one barrier), deterministic;
//   H_16..H_128  two more in-register stages and three across the block's eight lanes as fused
//             v_fmac_f32_dpp (lane pairs along 1, 2 and 7: quad_perm and row_half_mirror; the
//             output permutation this basis implies is undone by where each lane stores its codes);
//   encode    the uniform-cell table of the codebook (4 ops per code), as in the general kernel;
//   pack      v_cvt_pk_u8_f32 byte inserts and a few shift-ors, one 2*BITS-byte store per lane.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "device.h"

namespace orbit {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));

constexpr int kLaneVals = 16;   // positions per lane
// Staging layout: a row is K/8 chunks of 16 bytes, loaded 64 at a time (one wave) straight into
// LDS.  The two buffers interleave those 1 KB blocks: chunk c of buffer b sits at byte
// 2048 (c / 64) + 1024 b + 16 (c % 64) of the staging area, so the second buffer is the first one
// 1024 bytes further (an immediate offset of the LDS instructions).
constexpr int kBufGap = 1024;
// Cache-policy bits of the staging loads: non-temporal (each row is read once)
constexpr int kNonTemporal = 2;

// Butterfly between lanes 16 (SPAN = 16) or 32 (SPAN = 32) apart on two registers at once, with
// v_permlane16_swap / v_permlane32_swap (VALU, no LDS).  The swap trades the upper SPAN lanes of
// each 2*SPAN group of `a` for the lower SPAN lanes of `b`, so each lane then holds a pair
// (x_lo, x_hi) of one register; it forms x_lo + x_hi and x_hi - x_lo, and a second swap puts both
// back where they belong: a lower lane ends with x_lo + x_hi, an upper one with x_hi - x_lo, as a
// fused multiply-add own + (-1 on upper lanes) partner would give.
template <int SPAN>
__device__ __forceinline__ void swap_butterfly(float& a, float& b) {
    static_assert(SPAN == 16 || SPAN == 32, "span");
    uint32_t lo, hi;
    if constexpr (SPAN == 32) {
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false, false);
        lo = r[0];
        hi = r[1];
    } else {
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
        lo = r[0];
        hi = r[1];
    }
    const float s = __uint_as_float(lo) + __uint_as_float(hi), d = __uint_as_float(hi) - __uint_as_float(lo);
    if constexpr (SPAN == 32) {
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(s), __float_as_uint(d), false, false);
        a = __uint_as_float(r[0]);
        b = __uint_as_float(r[1]);
    } else {
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(s), __float_as_uint(d), false, false);
        a = __uint_as_float(r[0]);
        b = __uint_as_float(r[1]);
    }
}

template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}

// z[r] <- z[r] + sgn * (z[r] of the partner lane), 16 registers, fused DPP FMACs.  The compiler
// cannot fuse mov_dpp into the tied-operand fmac, so it is written out; the leading s_nop covers
// the two wait states a DPP read needs after a VALU write of its source.
#define ORBIT_ROW_DPP16(Z, SGN, PERM)                                                             \
    asm volatile("s_nop 1\n"                                                                      \
                 "v_fmac_f32_dpp %0, %0, %16 " PERM " row_mask:0xf bank_mask:0xf\n"               \
                 "v_fmac_f32_dpp %1, %1, %16 " PERM " row_mask:0xf bank_mask:0xf\n"               \
                 "v_fmac_f32_dpp %2, %2, %16 " PERM " row_mask:0xf bank_mask:0xf\n"               \
                 "v_fmac_f32_dpp %3, %3, %16 " PERM " row_mask:0xf bank_mask:0xf\n"               \
                 "v_fmac_f32_dpp %4, %4, %16 " PERM " row_mask:0xf bank_mask:0xf\n"               \
                 "v_fmac_f32_dpp %5, %5, %16 " PERM " row_mask:0xf bank_mask:0xf\n"               \
                 "v_fmac_f32_dpp %6, %6, %16 " PERM " row_mask:0xf bank_mask:0xf\n"               \
                 "v_fmac_f32_dpp %7, %7, %16 " PERM " row_mask:0xf bank_mask:0xf\n"               \
                 "v_fmac_f32_dpp %8, %8, %16 " PERM " row_mask:0xf bank_mask:0xf\n"               \
                 "v_fmac_f32_dpp %9, %9, %16 " PERM " row_mask:0xf bank_mask:0xf\n"               \
                 "v_fmac_f32_dpp %10, %10, %16 " PERM " row_mask:0xf bank_mask:0xf\n"             \
                 "v_fmac_f32_dpp %11, %11, %16 " PERM " row_mask:0xf bank_mask:0xf\n"             \
                 "v_fmac_f32_dpp %12, %12, %16 " PERM " row_mask:0xf bank_mask:0xf\n"             \
                 "v_fmac_f32_dpp %13, %13, %16 " PERM " row_mask:0xf bank_mask:0xf\n"             \
                 "v_fmac_f32_dpp %14, %14, %16 " PERM " row_mask:0xf bank_mask:0xf\n"             \
                 "v_fmac_f32_dpp %15, %15, %16 " PERM " row_mask:0xf bank_mask:0xf\n"             \
                 : "+v"(Z[0]), "+v"(Z[1]), "+v"(Z[2]), "+v"(Z[3]), "+v"(Z[4]), "+v"(Z[5]),           \
                   "+v"(Z[6]), "+v"(Z[7]), "+v"(Z[8]), "+v"(Z[9]), "+v"(Z[10]), "+v"(Z[11]),         \
                   "+v"(Z[12]), "+v"(Z[13]), "+v"(Z[14]), "+v"(Z[15])                                \
                 : "v"(SGN))

// The first two butterfly stages of the lane's four quads, signs included.  Pair i of the lane
// holds positions 2i (low half) and 2i+1 (high half) as bf16; S[i] holds their Rademacher signs
// as the bf16 pair (s_2i, s_2i+1).  For quad u (pairs 2u, 2u+1, positions y0..y3):
//     a = s0 y0 + s1 y1,  b = s0 y0 - s1 y1                       (neg_hi on S)
//     z0 = a + s2 y2 + s3 y3,  z1 = b + s2 y2 - s3 y3,  z2 = a - s2 y2 - s3 y3,  z3 = b - s2 y2 + s3 y3
// which is H_4 (Sylvester order) of the signed quad; every product is exact (bf16 times +-1).
// n[u] collects y0^2 + y1^2 + y2^2 + y3^2.  A DOT result needs wait states before a VALU op
// reads it and the compiler's hazard tracking does not look inside asm, so every read here comes
// at least five instructions after its producer, and the block ends with s_nop 4 for the reads
// that follow it.
#define ORBIT_ROW_H4(Z, N, P, S)                                                                  \
    asm volatile(                                                                                 \
        "v_dot2_f32_bf16 %20, %21, %29, 0\n"                                                      \
        "v_dot2_f32_bf16 %0, %21, %29, 0 neg_hi:[0,1,0]\n"                                        \
        "v_dot2_f32_bf16 %4, %23, %31, 0\n"                                                       \
        "v_dot2_f32_bf16 %5, %23, %31, 0 neg_hi:[0,1,0]\n"                                        \
        "v_dot2_f32_bf16 %8, %25, %33, 0\n"                                                       \
        "v_dot2_f32_bf16 %9, %25, %33, 0 neg_hi:[0,1,0]\n"                                        \
        "v_dot2_f32_bf16 %12, %27, %35, 0\n"                                                      \
        "v_dot2_f32_bf16 %13, %27, %35, 0 neg_hi:[0,1,0]\n"                                       \
        "v_dot2_f32_bf16 %16, %21, %21, 0\n"                                                      \
        "v_dot2_f32_bf16 %17, %23, %23, 0\n"                                                      \
        "v_dot2_f32_bf16 %18, %25, %25, 0\n"                                                      \
        "v_dot2_f32_bf16 %19, %27, %27, 0\n"                                                      \
        "v_dot2_f32_bf16 %1, %22, %30, %0 neg_hi:[0,1,0]\n"                                       \
        "v_dot2_f32_bf16 %2, %22, %30, %20 neg_lo:[0,1,0] neg_hi:[0,1,0]\n"                       \
        "v_dot2_f32_bf16 %3, %22, %30, %0 neg_lo:[0,1,0]\n"                                       \
        "v_dot2_f32_bf16 %0, %22, %30, %20\n"                                                     \
        "v_dot2_f32_bf16 %6, %24, %32, %4 neg_lo:[0,1,0] neg_hi:[0,1,0]\n"                        \
        "v_dot2_f32_bf16 %7, %24, %32, %5 neg_lo:[0,1,0]\n"                                       \
        "v_dot2_f32_bf16 %4, %24, %32, %4\n"                                                      \
        "v_dot2_f32_bf16 %5, %24, %32, %5 neg_hi:[0,1,0]\n"                                       \
        "v_dot2_f32_bf16 %10, %26, %34, %8 neg_lo:[0,1,0] neg_hi:[0,1,0]\n"                       \
        "v_dot2_f32_bf16 %11, %26, %34, %9 neg_lo:[0,1,0]\n"                                      \
        "v_dot2_f32_bf16 %8, %26, %34, %8\n"                                                      \
        "v_dot2_f32_bf16 %9, %26, %34, %9 neg_hi:[0,1,0]\n"                                       \
        "v_dot2_f32_bf16 %14, %28, %36, %12 neg_lo:[0,1,0] neg_hi:[0,1,0]\n"                      \
        "v_dot2_f32_bf16 %15, %28, %36, %13 neg_lo:[0,1,0]\n"                                     \
        "v_dot2_f32_bf16 %12, %28, %36, %12\n"                                                    \
        "v_dot2_f32_bf16 %13, %28, %36, %13 neg_hi:[0,1,0]\n"                                     \
        "v_dot2_f32_bf16 %16, %22, %22, %16\n"                                                    \
        "v_dot2_f32_bf16 %17, %24, %24, %17\n"                                                    \
        "v_dot2_f32_bf16 %18, %26, %26, %18\n"                                                    \
        "v_dot2_f32_bf16 %19, %28, %28, %19\n"                                                    \
        "s_nop 4"                                                                                 \
        : "=&v"(Z[0]), "=&v"(Z[1]), "=&v"(Z[2]), "=&v"(Z[3]), "=&v"(Z[4]), "=&v"(Z[5]),             \
          "=&v"(Z[6]), "=&v"(Z[7]), "=&v"(Z[8]), "=&v"(Z[9]), "=&v"(Z[10]), "=&v"(Z[11]),           \
          "=&v"(Z[12]), "=&v"(Z[13]), "=&v"(Z[14]), "=&v"(Z[15]), "=&v"(N[0]), "=&v"(N[1]),         \
          "=&v"(N[2]), "=&v"(N[3]), "=&v"(tmp_a)                                                   \
        : "v"(P[0]), "v"(P[1]), "v"(P[2]), "v"(P[3]), "v"(P[4]), "v"(P[5]), "v"(P[6]), "v"(P[7]), \
          "v"(S[0]), "v"(S[1]), "v"(S[2]), "v"(S[3]), "v"(S[4]), "v"(S[5]), "v"(S[6]), "v"(S[7]))

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float x) {
    uint32_t b = __float_as_uint(x);
    b += 0x7FFFu + ((b >> 16) & 1u);
    return (uint16_t)(b >> 16);
}

template <int K>
__device__ __forceinline__ uint32_t code_byte(float y, uint32_t into) {
    return __builtin_amdgcn_cvt_pk_u8_f32(y, K, into);
}

// 16 codes, given as values y whose nearest integer is the level index, stored as sign-magnitude
// labels packed LSB-first into 2*BITS bytes: w[0] (2 bits), w[0..1] (4 bits), w[0] and the low
// half of w[1] (3 bits), w[0..2] (6 bits).  The labels are formed on words of byte or packed
// fields (one bitwise pass per word).
template <int BITS>
__device__ __forceinline__ void pack16(const float (&y)[16], uint32_t (&w)[3]) {
    if constexpr (BITS == 4) {
        // bytes of A = codes 8i, 8i+2, 8i+4, 8i+6 and of B = codes 8i+1, 8i+3, ...: A | B << 4
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const float* v = y + 8 * i;
            uint32_t A = code_byte<0>(v[0], 0u), B = code_byte<0>(v[1], 0u);
            A = code_byte<1>(v[2], A);
            B = code_byte<1>(v[3], B);
            A = code_byte<2>(v[4], A);
            B = code_byte<2>(v[5], B);
            A = code_byte<3>(v[6], A);
            B = code_byte<3>(v[7], B);
            w[i] = sign_magnitude_labels<0x88888888u, 3, 0xFFFFFFFFu>(A | (B << 4));
        }
        w[2] = 0u;
    } else if constexpr (BITS == 2) {
        // byte j of D_k holds code 4j + k: D_0 | D_1 << 2 | D_2 << 4 | D_3 << 6
        uint32_t D[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            uint32_t d = code_byte<0>(y[k], 0u);
            d = code_byte<1>(y[4 + k], d);
            d = code_byte<2>(y[8 + k], d);
            D[k] = code_byte<3>(y[12 + k], d);
        }
        w[0] = sign_magnitude_labels<0xAAAAAAAAu, 1, 0xFFFFFFFFu>(D[0] | (D[1] << 2) | (D[2] << 4) | (D[3] << 6));
        w[1] = w[2] = 0u;
    } else if constexpr (BITS == 3) {
        // 8 codes = 24 bits: codes 2j, 2j+1 share byte j of P (6 bits), then the gaps close
        uint32_t g[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const float* v = y + 8 * i;
            uint32_t A = code_byte<0>(v[0], 0u), B = code_byte<0>(v[1], 0u);
            A = code_byte<1>(v[2], A);
            B = code_byte<1>(v[3], B);
            A = code_byte<2>(v[4], A);
            B = code_byte<2>(v[5], B);
            A = code_byte<3>(v[6], A);
            B = code_byte<3>(v[7], B);
            const uint32_t P = sign_magnitude_labels<0x24242424u, 2, 0x3F3F3F3Fu>(A | (B << 3));
            g[i] = (P & 0x3Fu) | ((P >> 2) & 0xFC0u) | ((P >> 4) & 0x3F000u) | ((P >> 6) & 0xFC0000u);
        }
        w[0] = g[0] | (g[1] << 24);  // bytes 0..3
        w[1] = g[1] >> 8;            // bytes 4..5
        w[2] = 0u;
    } else {
        static_assert(BITS == 6, "bits");
        // 4 codes = 24 bits: the bytes of A are codes 4i .. 4i+3, then the gaps close
        uint32_t g[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float* v = y + 4 * i;
            uint32_t A = code_byte<0>(v[0], 0u);
            A = code_byte<1>(v[1], A);
            A = code_byte<2>(v[2], A);
            A = sign_magnitude_labels<0x20202020u, 5, 0x3F3F3F3Fu>(code_byte<3>(v[3], A));
            g[i] = (A & 0x3Fu) | ((A >> 2) & 0xFC0u) | ((A >> 4) & 0x3F000u) | ((A >> 6) & 0xFC0000u);
        }
        w[0] = g[0] | (g[1] << 24);
        w[1] = (g[1] >> 8) | (g[2] << 16);
        w[2] = (g[2] >> 16) | (g[3] << 8);
    }
}

// 2*BITS bytes of packed codes at a 2*BITS-byte aligned offset, stored non-temporal (the codes
// are written once and not read again by this kernel; the hint keeps them from displacing the
// streaming rows in the caches)
template <int BITS>
__device__ __forceinline__ void store16(uint8_t* dst, const uint32_t (&w)[3]) {
    if constexpr (BITS == 4) {
        u32x2 v;
        v.x = w[0];
        v.y = w[1];
        __builtin_nontemporal_store(v, (u32x2*)dst);
    } else if constexpr (BITS == 2) {
        __builtin_nontemporal_store(w[0], (uint32_t*)dst);
    } else if constexpr (BITS == 6) {
        uint32_t* d = (uint32_t*)dst;
        __builtin_nontemporal_store(w[0], d);
        __builtin_nontemporal_store(w[1], d + 1);
        __builtin_nontemporal_store(w[2], d + 2);
    } else {
        uint16_t* d = (uint16_t*)dst;   // 6 bytes at an even offset
        __builtin_nontemporal_store((uint16_t)w[0], d);
        __builtin_nontemporal_store((uint16_t)(w[0] >> 16), d + 1);
        __builtin_nontemporal_store((uint16_t)w[1], d + 2);
    }
}

template <int BITS, bool NORM_BF16, int OUTER>
__global__ __launch_bounds__(1024) void rpbh_quantize_row_kernel(QuantParams p) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int tid = threadIdx.x;
    const int lanes = p.K / kLaneVals;     // lanes holding positions (a multiple of 8: whole blocks)
    const bool active = tid < lanes;
    const int blk = tid >> 3, q = tid & 7;
    const int nb = p.nb;
    float* const part = (float*)(smem + p.part_off);

    // Stages across lanes.  An h-block (h = 128 * 2^OUTER) spans L = h/16 consecutive, aligned lanes
    // and its Hadamard stages pair lane j with j ^ v along a basis of the lane-index bits:
    //   h = 128:   v = 1, 2 (quad_perm), 7 (row_half_mirror)                          dual {5, 6, 4}
    //   h >= 256:  v = 1, 2, 7, 15 (row_mirror), then 16 and 32 (lane swaps) as far as the block
    //              spans                                                               dual {5, 6, 12, 8, 16, 32}
    // Butterflies along a basis v_k whose lower / upper roles follow the dual basis s_k (parity of
    // s_k & v_m is 1 iff k = m) compute the Sylvester transform with permuted outputs: lane j ends
    // with the 16 outputs of lane position M(j), the XOR of the s_k whose parity with j is odd, so
    // it stores its codes there.  Each stage leaves the upper partner's value negated; sigma, the
    // parity of j & (XOR of the s_k), collects those signs and goes into the encoder scale.
    auto odd = [](int v) { return (__popc(v) & 1) != 0; };
    constexpr int LB = 8 << OUTER;                         // lanes per h-block
    const int j = tid & (LB - 1);
    constexpr int d1 = 5, d2 = 6, d3 = OUTER == 0 ? 4 : 12, d4 = 8;
    const float sg1 = odd(j & d1) ? -1.f : 1.f, sg2 = odd(j & d2) ? -1.f : 1.f, sg3 = odd(j & d3) ? -1.f : 1.f;
    const float sg4 = odd(j & d4) ? -1.f : 1.f;
    int mj = (odd(j & d1) ? d1 : 0) ^ (odd(j & d2) ? d2 : 0) ^ (odd(j & d3) ? d3 : 0);
    if (OUTER >= 1 && odd(j & d4)) mj ^= d4;
    mj |= j & ~15;                                         // bits 4, 5: the standard basis
    constexpr int SX = OUTER == 0 ? 5 ^ 6 ^ 4 : (5 ^ 6 ^ 12 ^ 8) | (OUTER >= 2 ? 16 : 0) | (OUTER >= 3 ? 32 : 0);
    const float sigma = odd(j & SX) ? -1.f : 1.f;
    const int mpos = (tid & ~(LB - 1)) + mj;               // output position, in 16-code units
    const int lane = tid & 63;

    // encoder table -> LDS
    for (int i = tid; i < p.ncell; i += blockDim.x) ((float*)smem)[i] = p.enc[i];

    // gather offsets (buffer 0; buffer 1 is 16 bytes further) and sign pairs of the lane's 16
    // positions: meta[j] = 2 perm[j] with bit 31 set where sign[j] = -1
    uint32_t addr[kLaneVals];
    uint32_t S[8];
    {
        const int pos = active ? tid * kLaneVals : 0;
        const uint4* src = (const uint4*)(p.meta + pos);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint4 v = src[i];
            const uint32_t m[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t e = (m[k] & 0x7FFFFFFFu) >> 1;  // source element perm[j]
                const uint32_t c = e >> 3;                      // its chunk
                addr[4 * i + k] = p.row_off + 2048u * (c >> 6) + 16u * (c & 63u) + 2u * (e & 7u);
            }
#pragma unroll
            for (int k = 0; k < 4; k += 2)
                S[2 * i + k / 2] = ((m[k] >> 31) ? 0xBF80u : 0x3F80u) | (((m[k + 1] >> 31) ? 0xBF80u : 0x3F80u) << 16);
        }
    }

    // staging: wave w brings chunks 64 w + 64 v .. 64 w + 64 v + 63 of a row for v = 0, T/64, ...
    // (T threads), straight from HBM into LDS (global_load_lds_dwordx4: lane i of the wave writes
    // the LDS base + 16 i); a row issued after one barrier has landed by the next
    const int G = gridDim.x;
    const int M = (int)p.M;   // below 2^31 (checked by the caller)
    const int nchunks = p.K / 8, wave = tid >> 6, waves = blockDim.x >> 6;
    // A row is K/512 blocks of 64 chunks and a workgroup has at least K/1024 waves, so each wave
    // brings at most two blocks: `wave` and `wave + waves`.  The row's address is uniform, the lane's
    // part of a block is 16 * lane bytes further.
    const int nblk = (nchunks + 63) / 64;
    const uint32_t lane_off = 16u * (uint32_t)(tid & 63);
    const bool lane_in_last = (nchunks & 63) == 0 || (tid & 63) < (nchunks & 63);
    auto load_row = [&](int row, int buf) {
        if (row >= M) return;
        const char* base = (const char*)p.X + (int64_t)row * p.ldx * 2;
#pragma unroll
        for (int v = 0; v < 2; ++v) {
            const int b = wave + v * waves;
            if (b >= nblk) break;
            __attribute__((address_space(3))) void* dst = (__attribute__((address_space(3))) void*)(
                (__attribute__((address_space(3))) unsigned char*)smem + p.row_off + 2048u * b + kBufGap * buf);
            if (b < nblk - 1 || lane_in_last)
                __builtin_amdgcn_global_load_lds((const void*)(base + 1024 * b + lane_off), dst, 16, 0, kNonTemporal);
        }
    };

    // The first row, then the second in flight before the loop (the loop keeps one row in flight
    // for a whole iteration: issued right after a barrier, waited for at the next one).
    int g = blockIdx.x;
    if (g < M) load_row(g, 0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    load_row(g + G, 1);

    const float cm = p.enc_center + 8388608.0f;
    // f = C + 2^23 + round(t - C) has the bit pattern 0x4B000000 + cell, so the cell's LDS byte
    // address is 4 * bits(f) + (table - 4 * 0x4B000000) (mod 2^32): one shift-add
    const uint32_t tab = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)smem - 0x2C000000u;
    const int64_t code_row = (int64_t)p.K * BITS / 8;

    // One row from staging buffer BUF (a compile-time constant, so the buffer offset is the LDS
    // instructions' immediate): the loop below alternates the two.  Row g + G is already in flight
    // into the other buffer.
    auto iteration = [&](auto buf_tag) {
        constexpr int BUF = decltype(buf_tag)::value;
        // gather: pair i = positions 2i (low half), 2i+1 (high half).  All sixteen reads are issued
        // before the first is used (one LDS round trip per row, not two).
        uint16_t gv[kLaneVals];
#pragma unroll
        for (int r = 0; r < kLaneVals; ++r) gv[r] = *(const uint16_t*)(smem + addr[r] + kBufGap * BUF);
        __builtin_amdgcn_sched_barrier(0);
        uint32_t P[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            u16x2 v;
            v.x = gv[2 * i];
            v.y = gv[2 * i + 1];
            P[i] = __builtin_bit_cast(uint32_t, v);
        }

        float z[kLaneVals], n[4], tmp_a;
        ORBIT_ROW_H4(z, n, P, S);
        // z[4u + v] is output v of quad u; two more stages inside the lane (distance 4 and 8)
#pragma unroll
        for (int st = 4; st < 16; st <<= 1) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                if (r & st) continue;
                const float x0 = z[r], x1 = z[r + st];
                z[r] = x0 + x1;
                z[r + st] = x0 - x1;
            }
        }
        ORBIT_ROW_DPP16(z, sg1, "quad_perm:[1,0,3,2]");
        ORBIT_ROW_DPP16(z, sg2, "quad_perm:[2,3,0,1]");
        ORBIT_ROW_DPP16(z, sg3, "row_half_mirror");
        if constexpr (OUTER >= 1) ORBIT_ROW_DPP16(z, sg4, "row_mirror");
        // lanes 16 apart inside 32, then 32 apart: register pairs through lane swaps
        if constexpr (OUTER >= 2) {
#pragma unroll
            for (int r = 0; r < kLaneVals; r += 2) swap_butterfly<16>(z[r], z[r + 1]);
        }
        if constexpr (OUTER >= 3) {
#pragma unroll
            for (int r = 0; r < kLaneVals; r += 2) swap_butterfly<32>(z[r], z[r + 1]);
        }

        // block sums of squares: the eight lanes of a block, in a fixed order
        float ss = (n[0] + n[1]) + (n[2] + n[3]);
        ss += dpp_mov<0xB1>(ss);   // quad_perm [1,0,3,2]
        ss += dpp_mov<0x4E>(ss);   // quad_perm [2,3,0,1]
        ss += dpp_mov<0x141>(ss);  // row_half_mirror
        float* const pt = part + BUF * nb;
        if (active && q == 0) pt[blk] = ss;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // row g + G's staging loads
        __syncthreads();
        // every wave has gathered row g: row g + 2G goes into its buffer, with the encode below and
        // the next row's gather and transform to complete in
        load_row(g + 2 * G, BUF);
        // row total: every wave sums the block partials in the same fixed order
        float acc = lane < nb ? pt[lane] : 0.f;   // nb <= 128 block partials
        if (lane + 64 < nb) acc += pt[lane + 64];
        acc += dpp_mov<0xB1>(acc);
        acc += dpp_mov<0x4E>(acc);
        acc += dpp_mov<0x141>(acc);
        acc += dpp_mov<0x140>(acc);   // row_mirror
        const float tot = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(acc), 0)) +
                          __int_as_float(__builtin_amdgcn_readlane(__float_as_int(acc), 16)) +
                          __int_as_float(__builtin_amdgcn_readlane(__float_as_int(acc), 32)) +
                          __int_as_float(__builtin_amdgcn_readlane(__float_as_int(acc), 48));
        const float s = __builtin_amdgcn_sqrtf(tot);   // v_sqrt_f32 (1 ulp)
        if (tid == 0) {
            if constexpr (NORM_BF16)
                ((uint16_t*)p.norm)[g] = f32_to_bf16_rne(s);
            else
                ((float*)p.norm)[g] = s;
        }
        // u = z / (s + eps), z unnormalised by sqrt(h); t = u / w + C is the cell coordinate and
        // round(0.5 (t - C) + bias[cell]) the code.  Adding 2^23 rounds t to the cell index in the
        // low mantissa bits (|u| <= 1 keeps it inside the table for every finite row); lanes
        // holding no positions take a zero scale, the middle cell.
        const float a = active ? sigma * p.enc_inv_w * __builtin_amdgcn_rcpf(fmaxf(s + p.eps, 1e-30f) * p.sqrt_h) : 0.f;
        const float ah = 0.5f * a;
        float y[kLaneVals];
#pragma unroll
        for (int r = 0; r < kLaneVals; ++r) {
            const uint32_t ad = __float_as_uint(fmaf(z[r], a, cm)) * 4u + tab;
            y[r] = fmaf(z[r], ah, *(const __attribute__((address_space(3))) float*)(uintptr_t)ad);
        }
        uint32_t w[3];
        pack16<BITS>(y, w);
        if (active) store16<BITS>(p.codes + (int64_t)g * code_row + (int64_t)mpos * (2 * BITS), w);
        (void)tmp_a;
    };
    for (;;) {
        if (g >= M) break;
        iteration(std::integral_constant<int, 0>{});
        g += G;
        if (g >= M) break;
        iteration(std::integral_constant<int, 1>{});
        g += G;
    }
}

template <int BITS, bool NB, int OUTER>
hipError_t set_row_smem_limit() {
    static std::atomic<uint64_t> done{0};
    return raise_lds_limit((const void*)rpbh_quantize_row_kernel<BITS, NB, OUTER>, 160 * 1024, done);
}

}  // namespace

bool rpbh_quantize_row_fits(int K, int h, bool gather) {
    return gather && h >= 128 && h <= 1024 && K % 128 == 0 && K % h == 0 && K >= 1024 && K <= 16384;
}

hipError_t launch_rpbh_quantize_row(QuantParams p, int bits, bool norm_bf16, int cus, hipStream_t stream) {
    const int threads = (p.K / kLaneVals + 63) / 64 * 64;
    auto align16 = [](uint32_t b) { return (b + 15u) & ~15u; };
    p.part_off = align16((uint32_t)p.ncell * 4u);
    p.row_off = p.part_off + align16((uint32_t)p.nb * 8u);
    // two interleaved row buffers of whole 1 KB blocks (64 chunks)
    const size_t smem = (size_t)p.row_off + 2048u * (size_t)((p.K / 8 + 63) / 64);
    if (smem > 160u * 1024u) return hipErrorInvalidValue;
    // persistent: exactly as many workgroups as are resident at once (a grid larger than that would
    // start its last workgroups only when earlier ones had finished all their rows)
#define ORBIT_ROW_LAUNCH(B, NB, OU)                                                                 \
    do {                                                                                            \
        const hipError_t e = set_row_smem_limit<B, NB, OU>();                                       \
        if (e != hipSuccess) return e;                                                              \
        const int64_t want = (int64_t)cus * resident_blocks((const void*)rpbh_quantize_row_kernel<B, NB, OU>, threads, smem); \
        const int grid = (int)(p.M < want ? p.M : want);                                            \
        hipLaunchKernelGGL((rpbh_quantize_row_kernel<B, NB, OU>), dim3(grid), dim3(threads), smem, stream, p); \
    } while (0)
#define ORBIT_ROW_OUTER(B, NB)                                                                      \
    do {                                                                                            \
        if (p.outer == 0) ORBIT_ROW_LAUNCH(B, NB, 0);                                               \
        else if (p.outer == 1) ORBIT_ROW_LAUNCH(B, NB, 1);                                          \
        else if (p.outer == 2) ORBIT_ROW_LAUNCH(B, NB, 2);                                          \
        else ORBIT_ROW_LAUNCH(B, NB, 3);                                                            \
    } while (0)
#define ORBIT_ROW_BITS(NB)                                                                          \
    do {                                                                                            \
        if (bits == 2) ORBIT_ROW_OUTER(2, NB);                                                      \
        else if (bits == 3) ORBIT_ROW_OUTER(3, NB);                                                 \
        else if (bits == 6) ORBIT_ROW_OUTER(6, NB);                                                 \
        else ORBIT_ROW_OUTER(4, NB);                                                                \
    } while (0)
    if (norm_bf16) ORBIT_ROW_BITS(true);
    else ORBIT_ROW_BITS(false);
#undef ORBIT_ROW_BITS
#undef ORBIT_ROW_OUTER
#undef ORBIT_ROW_LAUNCH
    return hipGetLastError();
}

}  // namespace orbit
