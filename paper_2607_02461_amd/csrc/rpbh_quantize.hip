// Fused RPBH rotate -> normalize -> Lloyd-Max encode -> pack, for gfx950.
//
// One kernel serves the online activation quantizer (Sec. 4.3, Eqs. (7)-(8)) and the offline
// weight pass (Sec. 4.2, Eqs. (4)-(6)); they differ only in the type of the stored norm.
//
// Work mapping (h = 128).  A persistent workgroup owns R rows per iteration and loops over row
// groups.  Rows are staged in LDS with 16-byte coalesced loads, twice: as loaded and with every
// bf16 sign bit flipped.  The next group is loaded into registers right after the current
// group's gathers and written over the staging buffers at the end of the iteration, so the HBM
// reads overlap the butterflies, the norm reduction and the encoder, and the gather offsets stay
// loop-invariant registers.  Every 128-block of a row belongs to one quad of lanes; lane q of the
// quad holds the 32 consecutive post-permutation positions q*32 .. q*32+31.  (With an identity
// permutation there is no staging: each lane loads its 64 contiguous bytes straight from HBM.)
//
// Per element the hot loop costs:
//   gather       one LDS u16 read through a per-lane table of byte offsets (the permutation),
//                each pointing into the copy the position's Rademacher sign selects;
//   sign         the flipped copy: half an XOR per element while staging;
//   widening and the first butterfly stage together: one v_dot2_f32_bf16 of a gathered bf16
//                pair (y0, y1) with (1, 1) or (1, -1) gives y0 + y1 or y0 - y1 exactly in fp32;
//   row norm     half a v_dot2 (the pair against itself; the rotation is orthogonal, so the sum of
//                squares of the gathered inputs is the squared norm of the rotated row);
//   butterflies  four more in-register stages and two stages across the quad, each one fused
//                v_fmac_f32_dpp computing own + sign*partner.  That leaves the upper lane of each
//                pair holding the negated output; the sign is fixed per lane,
//                sigma = (-1)^popcount(q), and is folded into the per-row encoder scale;
//   encode       fma(z, a, C + 2^23) rounds the coordinate to its cell of a table in LDS whose cells
//                are narrower than the smallest gap between thresholds, the index sitting in the
//                low mantissa bits; with the cell's bias b, y = fma(z, a/2, b) lies within 0.25 of
//                the code away from the cell's threshold (if it has one) and crosses code + 0.5
//                exactly at it;
//   pack         v_cvt_pk_u8_f32 rounds y to the code and inserts it as one byte of a word;
//                a few shift-ors close the gaps, and 32 codes leave as one 4*b-byte vector store.
// Blocks larger than 128 (h = 128 * 2^m, up to 4096): Sylvester H_h = (H_{2^m} (x) I_128)(I_{2^m} (x)
// H_128), so after the 128-point transform the remaining m stages pair equal offsets of the 128-blocks
// of an h-block.  The quads of an h-block are consecutive and aligned, so those stages pair lanes
// of an aligned group of h/32.  Inside a 16-lane row they run on DPP alone, like the quad stages:
// the four stages of a 16-lane group pair lanes along 1, 2, 7 and 15 (quad_perm, row_half_mirror,
// row_mirror), a basis of the lane index bits; the output permutation this basis implies is undone
// by where each lane stores its codes (see the lane set-up in the kernel).  Lanes 16 and 32 apart
// pair through ds_swizzle and ds_bpermute, and for h = 4096 an exchange through LDS joins two waves.
// Each stage again leaves the upper lane's value negated, which the per-lane encoder sign absorbs.
// The row's squared norm is reduced deterministically: quad DPP sums, per-block partials in LDS,
// then one wave per row.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device.h"

namespace orbit {

namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));


template <int CTRL>
__device__ __forceinline__ float quad_perm(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}
constexpr int kQuadXor1 = 0xB1;  // quad_perm [1,0,3,2]

// z[r] <- z[r] + sgn * z[r] of lane (lane ^ XOR), for XOR in {16, 32}
// (eight registers at a time, so that the exchanges in flight need few temporaries)
template <int XOR>
__device__ __forceinline__ void lane_xor_stage(float (&z)[32], float sgn, int lane) {
#pragma unroll
    for (int c = 0; c < 32; c += 8) {
#pragma unroll
        for (int r = c; r < c + 8; ++r) {
            int v;
            if constexpr (XOR < 32)
                v = __builtin_amdgcn_ds_swizzle(__float_as_int(z[r]), 0x1F | (XOR << 10));  // lane ^ XOR in 32
            else
                v = __builtin_amdgcn_ds_bpermute((lane ^ 32) << 2, __float_as_int(z[r]));
            z[r] = fmaf(__int_as_float(v), sgn, z[r]);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
}
constexpr int kQuadXor2 = 0x4E;  // quad_perm [2,3,0,1]

// z[r] <- z[r] + sgn * z[r] of the partner lane, for 16 registers, as fused DPP FMACs.  The compiler
// cannot fuse mov_dpp into the tied-operand fmac, so this is written out; the leading s_nop covers
// the two wait states a DPP read needs after a VALU write of its source.
#define ORBIT_DPP_FMAC16(Z, B, SGN, PERM)                                                          \
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
                 : "+v"(Z[B + 0]), "+v"(Z[B + 1]), "+v"(Z[B + 2]), "+v"(Z[B + 3]), "+v"(Z[B + 4]),    \
                   "+v"(Z[B + 5]), "+v"(Z[B + 6]), "+v"(Z[B + 7]), "+v"(Z[B + 8]), "+v"(Z[B + 9]),    \
                   "+v"(Z[B + 10]), "+v"(Z[B + 11]), "+v"(Z[B + 12]), "+v"(Z[B + 13]),              \
                   "+v"(Z[B + 14]), "+v"(Z[B + 15])                                                  \
                 : "v"(SGN))

// Sum over the 64 lanes of a wave, the same value in every lane, in a fixed order: quad, half-row
// and row sums by DPP, then the four row sums read out lane by lane.
__device__ __forceinline__ float wave_total(float v) {
    v += quad_perm<kQuadXor1>(v);
    v += quad_perm<kQuadXor2>(v);
    v += quad_perm<0x141>(v);  // row_half_mirror: lane l of 8 <- lane 7 - l
    v += quad_perm<0x140>(v);  // row_mirror: lane l of 16 <- lane 15 - l
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0)) +
           __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16)) +
           __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32)) +
           __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float x) {
    uint32_t b = __float_as_uint(x);
    b += 0x7FFFu + ((b >> 16) & 1u);
    return (uint16_t)(b >> 16);
}

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

// First butterfly stage from a bf16 pair (y0, y1): y0 + y1 and y0 - y1 as the three-operand
// v_dot2_f32_bf16 against (1, 1) held in an SGPR, with neg_hi giving (1, -1).  (The accumulating
// two-operand form the compiler picks would need its destination zeroed first.)  A DOT result
// needs wait states before another VALU op may read it, and the compiler's hazard tracking does
// not look inside asm, so the pair ends with an s_nop covering them.  The sum is early-clobber
// (it is written before the pair is read again); the difference may take the pair's register.
__device__ __forceinline__ void stage1(uint32_t P, uint32_t one_one, float& sum, float& diff) {
    asm("v_dot2_f32_bf16 %0, %2, %3, 0\n"
        "v_dot2_f32_bf16 %1, %2, %3, 0 neg_hi:[0,1,0]\n"
        "s_nop 3"
        : "=&v"(sum), "=v"(diff)
        : "v"(P), "s"(one_one));
}

template <int BITS>
__device__ __forceinline__ void store_packed(uint8_t* dst, const uint32_t (&w)[6]) {
    if constexpr (BITS == 4) {
        *(uint4*)dst = make_uint4(w[0], w[1], w[2], w[3]);
    } else if constexpr (BITS == 6) {
        // 24 bytes at an 8-byte aligned offset
        *(uint2*)dst = make_uint2(w[0], w[1]);
        *(uint2*)(dst + 8) = make_uint2(w[2], w[3]);
        *(uint2*)(dst + 16) = make_uint2(w[4], w[5]);
    } else if constexpr (BITS == 2) {
        *(uint2*)dst = make_uint2(w[0], w[1]);
    } else {
        uint32_t* d = (uint32_t*)dst;
        d[0] = w[0];
        d[1] = w[1];
        d[2] = w[2];
    }
}

// y -> round-to-nearest-even(y) saturated to [0, 255], inserted as byte K of `into`
template <int K>
__device__ __forceinline__ uint32_t code_byte(float y, uint32_t into) {
    return __builtin_amdgcn_cvt_pk_u8_f32(y, K, into);
}

// Packs 32 codes, given as values y whose nearest integer is the level index, as sign-magnitude
// labels LSB-first into 4*BITS bytes.  v_cvt_pk_u8_f32 converts a value and inserts it as one byte
// of a word in a single op; the codes are spread over bytes so that a few shifts and ORs close the
// gaps between them, and the labels are formed on words of byte or packed fields.
template <int BITS>
__device__ __forceinline__ void pack_codes(const float (&y)[32], uint32_t (&w)[6]) {
    if constexpr (BITS == 6) {
        // 4 codes = 24 bits: the bytes of A are codes 4i .. 4i+3, then the gaps close; eight
        // 24-bit groups fill six words
        uint32_t g[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float* v = y + 4 * i;
            uint32_t A = code_byte<0>(v[0], 0u);
            A = code_byte<1>(v[1], A);
            A = code_byte<2>(v[2], A);
            A = sign_magnitude_labels<0x20202020u, 5, 0x3F3F3F3Fu>(code_byte<3>(v[3], A));
            g[i] = (A & 0x3Fu) | ((A >> 2) & 0xFC0u) | ((A >> 4) & 0x3F000u) | ((A >> 6) & 0xFC0000u);
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            w[3 * h + 0] = g[4 * h] | (g[4 * h + 1] << 24);
            w[3 * h + 1] = (g[4 * h + 1] >> 8) | (g[4 * h + 2] << 16);
            w[3 * h + 2] = (g[4 * h + 2] >> 16) | (g[4 * h + 3] << 8);
        }
        return;
    } else if constexpr (BITS == 4) {
        // bytes of A = codes 8i, 8i+2, 8i+4, 8i+6 and of B = codes 8i+1, 8i+3, ...: A | B << 4
#pragma unroll
        for (int i = 0; i < 4; ++i) {
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
        return;
    } else if constexpr (BITS == 2) {
        // byte j of D_k holds code 16i + 4j + k: D_0 | D_1 << 2 | D_2 << 4 | D_3 << 6
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const float* v = y + 16 * i;
            uint32_t D[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                uint32_t d = code_byte<0>(v[k], 0u);
                d = code_byte<1>(v[4 + k], d);
                d = code_byte<2>(v[8 + k], d);
                D[k] = code_byte<3>(v[12 + k], d);
            }
            w[i] = sign_magnitude_labels<0xAAAAAAAAu, 1, 0xFFFFFFFFu>(D[0] | (D[1] << 2) | (D[2] << 4) | (D[3] << 6));
        }
        w[2] = w[3] = w[4] = w[5] = 0u;
    } else {
        static_assert(BITS == 3, "bits");
        // 8 codes = 24 bits: codes 2j, 2j+1 share byte j of P (6 bits), then the gaps close
        uint32_t g[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
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
        w[0] = g[0] | (g[1] << 24);
        w[1] = (g[1] >> 8) | (g[2] << 16);
        w[2] = (g[2] >> 16) | (g[3] << 8);
        w[3] = w[4] = w[5] = 0u;
    }
}

template <int BITS, bool NORM_BF16, bool OUTER, bool GATHER>
struct Quantizer {
    const QuantParams& p;
    unsigned char* smem;
    int tid, T, q, rg, blk;
    bool active;         // lane owns a (row slot, block) of the group
    uint32_t addr[32];   // staged gather: byte offset of each gathered element inside the staged group
    uint32_t mask[16];   // direct loads: bf16 sign bits of this lane's 16 element pairs
    uint32_t xoff;       // direct loads: byte offset of this lane's 64 bytes from the group's first row
    float sigma;
    float sgn1, sgn2, sgn3, sgn4;  // +1 / -1: lower / upper partner in the in-row butterfly stages
    int chunk;           // position (in 32-code units) of this lane's outputs in the row
    int cpr;             // 16-byte chunks per row

    __device__ __forceinline__ int rows_of(int g) const { return (int)min((int64_t)p.R, p.M - (int64_t)g * p.R); }

    // Staging: the R rows of a group sit back to back in LDS, so 16-byte chunk c of the group lands
    // at byte 16*c of the row buffer, and negated at byte 16*c of its copy.  In global memory
    // chunk c of row r lies 16*c + r*row_gap bytes past the group's first row.  With h = 128 the
    // four offsets of a lane are loop-invariant registers (goff).  The stages across 128-blocks
    // leave no room for them (they spilled, and each reload waited on the in-flight prefetch), so
    // there they are recomputed per iteration; the chunk index goes through an empty asm so that
    // the compiler cannot hoist them back out of the loop.
    uint32_t goff[OUTER ? 1 : 4];

    __device__ __forceinline__ uint32_t chunk_offset(int k) const {
        uint32_t off;
        if constexpr (OUTER) {
            uint32_t c = (uint32_t)(tid + k * T);
            asm volatile("" : "+v"(c));
            // 24-bit products (full rate): c < 2^11, row_magic < 2^20, row_gap < 2^24
            off = c * 16u + __umul24(__umul24(c, p.row_magic) >> p.row_shift, p.row_gap);
        } else {
            off = goff[k];
        }
        // (a register of its own: built in the load's destination, which the compiler cannot
        // prove free of the previous iteration's load, it would cost a full wait per load)
        asm volatile("" : "+v"(off));
        return off;
    }

    __device__ __forceinline__ void load_group(int g, u32x4 (&pf)[4]) const {
        const int lim = rows_of(g) * cpr;
        const char* base = (const char*)p.X + (int64_t)g * p.R * p.ldx * 2;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint32_t off = chunk_offset(k);
            if (tid + k * T < lim) pf[k] = __builtin_nontemporal_load((const u32x4*)(base + off));
        }
    }

    // writes the group to LDS as it is and with every bf16 sign flipped: the gather of a position
    // whose Rademacher sign is -1 reads the flipped copy, so the signs cost no work in the loop
    __device__ __forceinline__ void store_group(int g, const u32x4 (&pf)[4]) const {
        const int lim = rows_of(g) * cpr;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            int c = tid + k * T;
            asm volatile("" : "+v"(c));
            if (c < lim) {
                unsigned char* dst = smem + p.row_off + 16 * c;
                *(u32x4*)dst = pf[k];
                *(u32x4*)(dst + p.neg_off) = pf[k] ^ 0x80008000u;
            }
        }
    }

    // Identity permutation: the 32 positions a lane transforms are 64 consecutive bytes of its row,
    // read straight into registers (lanes without a block of a valid row keep what they hold).
    __device__ __forceinline__ void load_direct(int g, u32x4 (&v)[4]) const {
        const char* base = (const char*)p.X + (int64_t)g * p.R * p.ldx * 2;
        uint32_t off = xoff;
        asm volatile("" : "+v"(off));
        if (active && rg < rows_of(g)) {
            const u32x4* src = (const u32x4*)(base + off);
#pragma unroll
            for (int k = 0; k < 4; ++k) v[k] = __builtin_nontemporal_load(src + k);
        }
    }

    // One row group.  Every lane runs the arithmetic (lanes without a block of a valid row work on
    // harmless data); only the stores are guarded, so the hot path has no divergence.  `pf` carries
    // the direct loads of this group in and those of the next group out; `it` counts iterations.
    __device__ __forceinline__ void iteration(int g, int it, u32x4 (&pf)[4]) {
        const int next = g + gridDim.x;
        const int nb = p.nb;
        const int nrows = rows_of(g);
        const int64_t row0 = (int64_t)g * p.R;
        const bool owner = active && rg < nrows;
        // Block partials.  With direct loads the iteration has a single barrier, so the partials
        // alternate between two buffers: a wave writes the next group's partials only after the
        // barrier that every wave passes once it has finished reading this group's.
        float* part = (float*)(smem + p.part_off) + (GATHER ? 0 : (it & 1) * p.R * nb);

        // element pairs: element 2i in the low half, 2i+1 in the high half of P[i]
        uint32_t P[16];
        if constexpr (GATHER) {
            // (built as a two-lane vector, the pair becomes one v_perm of the two loads with no
            // masking of the zero-extended halves)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                u16x2 v;
                v.x = *(const uint16_t*)(smem + addr[2 * i]);
                v.y = *(const uint16_t*)(smem + addr[2 * i + 1]);
                P[i] = __builtin_bit_cast(uint32_t, v);
            }
        } else {
#pragma unroll
            for (int i = 0; i < 16; ++i) P[i] = pf[i >> 2][i & 3] ^ mask[i];
        }
        if (next < p.ngroups) {
            if constexpr (GATHER)
                load_group(next, pf);
            else
                load_direct(next, pf);
        }

        float z[32];
        float ss = 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            stage1(P[i], p.one_one, z[2 * i], z[2 * i + 1]);
            ss = dot2(P[i], P[i], ss);
        }
#pragma unroll
        for (int s = 2; s < 32; s <<= 1) {
#pragma unroll
            for (int r = 0; r < 32; ++r) {
                if (r & s) continue;
                const float a = z[r], b = z[r + s];
                z[r] = a + b;
                z[r + s] = a - b;
            }
        }
        // (for h = 128 the roles follow the quad index directly, recomputed here rather than held)
        const float sg1 = OUTER ? sgn1 : ((q & 1) ? -1.f : 1.f);
        const float sg2 = OUTER ? sgn2 : ((q & 2) ? -1.f : 1.f);
        ORBIT_DPP_FMAC16(z, 0, sg1, "quad_perm:[1,0,3,2]");
        ORBIT_DPP_FMAC16(z, 16, sg1, "quad_perm:[1,0,3,2]");
        ORBIT_DPP_FMAC16(z, 0, sg2, "quad_perm:[2,3,0,1]");
        ORBIT_DPP_FMAC16(z, 16, sg2, "quad_perm:[2,3,0,1]");
        if constexpr (OUTER) {
            // stages across the 128-blocks of an h-block: inside a 16-lane row along 7 and 15
            // (DPP mirrors), then lanes 16 and 32 apart
            const int lane = tid & 63, task = tid >> 2;
            if (p.outer > 0) {
                ORBIT_DPP_FMAC16(z, 0, sgn3, "row_half_mirror");
                ORBIT_DPP_FMAC16(z, 16, sgn3, "row_half_mirror");
            }
            if (p.outer > 1) {
                ORBIT_DPP_FMAC16(z, 0, sgn4, "row_mirror");
                ORBIT_DPP_FMAC16(z, 16, sgn4, "row_mirror");
            }
            if (p.outer > 2) lane_xor_stage<16>(z, (task & 4) ? -1.f : 1.f, lane);
            if (p.outer > 3) lane_xor_stage<32>(z, (task & 8) ? -1.f : 1.f, lane);
        }
        ss += quad_perm<kQuadXor1>(ss);
        ss += quad_perm<kQuadXor2>(ss);
        if (owner && q == 0) {
            // rg * nb + blk is the lane's task, tid / 4: recomputed here (the empty asm keeps it
            // from being hoisted), since a register held across the loop spilled with h > 128 and
            // its reload waited for the in-flight prefetch
            int task = tid >> 2;
            asm volatile("" : "+v"(task));
            part[task] = ss;
        }
        __syncthreads();

        if constexpr (OUTER) {
            if (p.outer > 4) {
                // h = 4096: the last stage pairs lanes 64 apart, in two waves.  The staging buffer
                // is free once every wave has passed the barrier above (all gathers are done); it
                // holds half of the lanes' values at a time.
                float* xb = (float*)(smem + p.row_off);
                const float sgn = (tid & 64) ? -1.f : 1.f;
#pragma unroll
                for (int hf = 0; hf < 2; ++hf) {
                    if (hf) __syncthreads();
                    float4* dst = (float4*)(xb + tid * 16);
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        dst[i] = make_float4(z[16 * hf + 4 * i], z[16 * hf + 4 * i + 1], z[16 * hf + 4 * i + 2],
                                             z[16 * hf + 4 * i + 3]);
                    __syncthreads();
                    const float4* src = (const float4*)(xb + (tid ^ 64) * 16);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float4 v = src[i];
                        z[16 * hf + 4 * i] = fmaf(v.x, sgn, z[16 * hf + 4 * i]);
                        z[16 * hf + 4 * i + 1] = fmaf(v.y, sgn, z[16 * hf + 4 * i + 1]);
                        z[16 * hf + 4 * i + 2] = fmaf(v.z, sgn, z[16 * hf + 4 * i + 2]);
                        z[16 * hf + 4 * i + 3] = fmaf(v.w, sgn, z[16 * hf + 4 * i + 3]);
                    }
                }
                __syncthreads();  // every read of the exchange is done before the buffer is refilled
            }
        }

        // Row totals: each wave reduces the block partials of the rows its lanes hold (the same
        // fixed-order sum in every wave), so no second barrier is needed.  The lane holding block 0
        // of a row stores its norm.
        const int lane = tid & 63;
        const int r_first = __builtin_amdgcn_readfirstlane(rg);
        const int r_last = __builtin_amdgcn_readlane(rg, 63);
        float s = 0.f;
        for (int r = r_first; r <= r_last && r < nrows; ++r) {
            float acc = 0.f;
            for (int i = lane; i < nb; i += 64) acc += part[r * nb + i];
            const float tot = __builtin_amdgcn_sqrtf(wave_total(acc));  // v_sqrt_f32 (1 ulp; no scaling fixups)
            if (rg == r) s = tot;
        }
        if (owner && blk == 0 && q == 0) {
            if constexpr (NORM_BF16)
                ((uint16_t*)p.norm)[row0 + rg] = f32_to_bf16_rne(s);
            else
                ((float*)p.norm)[row0 + rg] = s;
        }

        // u = z / (s + eps) with z = z_unnormalised / sqrt(h); t = u / w + C is the cell coordinate
        // and round(0.5 (t - C) + bias[cell]) the code.  Adding 2^23 rounds t to the cell index in
        // the low mantissa bits, so the index costs no conversion.  The index stays inside the
        // table for every finite row (|u| <= 1; the floor keeps the scale finite for any eps >= 0),
        // and lanes that store nothing take a zero scale.  A row holding Inf or NaN has
        // unspecified codes (its lookups may read outside the table, which returns zero).
        const float a = owner ? sigma * p.enc_inv_w * __builtin_amdgcn_rcpf(fmaxf(s + p.eps, 1e-30f) * p.sqrt_h) : 0.f;  // 1-ulp rcp
        const float ah = 0.5f * a;
        const float cm = p.enc_center + 8388608.0f;
        // f = C + 2^23 + round(t - C) has the bit pattern 0x4B000000 + cell, so the cell's LDS byte
        // address is 4 * bits(f) + (table - 4 * 0x4B000000) (mod 2^32): one shift-add
        const uint32_t tab = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)smem - 0x2C000000u;
        float y[32];
#pragma unroll
        for (int r = 0; r < 32; ++r) {
            const uint32_t addr = __float_as_uint(fmaf(z[r], a, cm)) * 4u + tab;
            y[r] = fmaf(z[r], ah, *(const __attribute__((address_space(3))) float*)(uintptr_t)addr);
        }
        uint32_t w[6];
        pack_codes<BITS>(y, w);
        if (owner)
            store_packed<BITS>(p.codes + (row0 + rg) * ((int64_t)p.K * BITS / 8) + (int64_t)(OUTER ? chunk : blk * 4 + q) * 4 * BITS, w);
        if constexpr (GATHER) {
            if (next < p.ngroups) {
                store_group(next, pf);
                __syncthreads();
            }
        }
    }
};

// GATHER: the permutation is applied by staging each row group in LDS and gathering from it; without
// it (identity permutation: Block-RHT and full-dimension rotations) lanes load their data directly.
template <int BITS, bool NORM_BF16, bool OUTER, bool GATHER>
__global__ __launch_bounds__(512, 4) void rpbh_quantize_kernel(QuantParams p) {
    extern __shared__ __align__(16) unsigned char smem[];
    Quantizer<BITS, NORM_BF16, OUTER, GATHER> Q{p, smem};
    Q.tid = threadIdx.x;
    Q.T = blockDim.x;
    const int task = Q.tid >> 2;
    Q.q = Q.tid & 3;
    Q.active = task < p.R * p.nb;
    // lanes past the last block keep the row index their task would have (so a wave's rows are
    // contiguous); every access they could make through it is guarded by `active`
    Q.rg = task / p.nb;
    Q.blk = task - Q.rg * p.nb;
    Q.cpr = p.K >> 3;
    {
        // Butterflies inside a 16-lane row pair lane j with j ^ v for v = 1, 2 (quad_perm), 7
        // (row_half_mirror) and 15 (row_mirror), as many as the h-block spans: 2 for h = 128, 3
        // for 256, 4 from 512 up.  Stages along a basis v_k whose lower / upper roles follow the
        // dual basis s_k (parity of s_k & v_m is 1 iff k = m) compute the Sylvester transform with
        // its outputs permuted: lane j ends with the output at position M(j), the XOR of the s_k
        // for which s_k & j has odd parity, so it stores its codes there.  As in every stage the
        // upper partner's value comes out negated; sigma collects those signs.
        const int nd = OUTER ? (p.outer == 1 ? 3 : p.outer >= 2 ? 4 : 2) : 2;
        const int s1 = nd == 2 ? 1 : 5, s2 = nd == 2 ? 2 : 6, s3 = nd == 3 ? 4 : 12, s4 = 8;
        const int jj = Q.tid & ((1 << nd) - 1);
        auto odd = [](int v) { return (__popc(v) & 1) != 0; };
        Q.sgn1 = odd(jj & s1) ? -1.f : 1.f;
        Q.sgn2 = odd(jj & s2) ? -1.f : 1.f;
        Q.sgn3 = odd(jj & s3) ? -1.f : 1.f;
        Q.sgn4 = odd(jj & s4) ? -1.f : 1.f;
        int m = (odd(jj & s1) ? s1 : 0) ^ (odd(jj & s2) ? s2 : 0);
        if (nd > 2 && odd(jj & s3)) m ^= s3;
        if (nd > 3 && odd(jj & s4)) m ^= s4;
        Q.chunk = ((Q.blk * 4 + Q.q) & ~((1 << nd) - 1)) | m;
        const int sx = s1 ^ s2 ^ (nd > 2 ? s3 : 0) ^ (nd > 3 ? s4 : 0);
        Q.sigma = odd(jj & sx) ? -1.f : 1.f;
        if constexpr (OUTER) {
            // one more negation per stage across rows and waves (lanes 16, 32, 64 apart) in which
            // this lane is the upper partner
            for (int j = 2; j < p.outer; ++j)
                if ((task >> j) & 1) Q.sigma = -Q.sigma;
        }
    }
    // encoder table -> LDS
    float* tab = (float*)smem;
    for (int i = Q.tid; i < p.ncell; i += Q.T) tab[i] = p.enc[i];

    u32x4 pf[4] = {};
    if constexpr (GATHER) {
        if constexpr (!OUTER) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int c = Q.tid + k * Q.T, r = c / Q.cpr;
                Q.goff[k] = (uint32_t)(r * p.ldx * 2 + (c - r * Q.cpr) * 16);
            }
        }
        const uint4* src = (const uint4*)(p.meta + Q.blk * 128 + Q.q * 32);
        const uint32_t rowoff = p.row_off + (uint32_t)(Q.rg * p.K * 2);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint4 v = src[i];
            const uint32_t m[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int k = 0; k < 4; ++k)
                Q.addr[4 * i + k] = Q.active ? rowoff + (m[k] & 0x7FFFFFFFu) + ((m[k] >> 31) ? p.neg_off : 0u) : p.row_off;
        }
        if (blockIdx.x < p.ngroups) {
            Q.load_group(blockIdx.x, pf);
            Q.store_group(blockIdx.x, pf);
        }
    } else {
        // with the identity permutation the sign mask of source pair i is that of position pair i
        const int pos = Q.active ? Q.blk * 128 + Q.q * 32 : 0;
        const uint4* src = (const uint4*)(p.smask + pos / 2);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint4 v = src[i];
            Q.mask[4 * i] = v.x;
            Q.mask[4 * i + 1] = v.y;
            Q.mask[4 * i + 2] = v.z;
            Q.mask[4 * i + 3] = v.w;
        }
        Q.xoff = (uint32_t)(Q.rg * p.ldx * 2 + pos * 2);
        if (blockIdx.x < p.ngroups) Q.load_direct(blockIdx.x, pf);
    }
    __syncthreads();
    int it = 0;
    for (int g = blockIdx.x; g < p.ngroups; g += gridDim.x) Q.iteration(g, it++, pf);
}

template <int BITS, bool NB, bool OUTER, bool GATHER>
hipError_t set_smem_limit() {
    static std::atomic<uint64_t> done{0};
    return raise_lds_limit((const void*)rpbh_quantize_kernel<BITS, NB, OUTER, GATHER>, 160 * 1024, done);
}

}  // namespace

int quant_rows_per_group(int K) {
    const int nb = K / 128;
    return nb >= 128 ? 1 : 128 / nb;
}

hipError_t launch_rpbh_quantize(QuantParams p, int bits, bool norm_bf16, bool gather, int cus, hipStream_t stream) {
    const int threads = ((p.R * p.nb * 4 + 63) / 64) * 64;
    // LDS: encoder table, two sets of block partials (the direct-load path alternates them), then
    // the staged rows and their negated copy (the gather path), or the exchange buffer of the
    // last h = 4096 stage (64 bytes per thread)
    auto align16 = [](uint32_t b) { return (b + 15u) & ~15u; };
    p.part_off = align16((uint32_t)p.ncell * 4u);
    p.row_off = p.part_off + align16((uint32_t)(p.R * p.nb) * 8u);
    const uint32_t rows = (uint32_t)(p.R * p.K) * 2u;
    p.neg_off = rows;
    const uint32_t row_bytes = gather ? 2u * rows : 0u;
    const uint32_t xchg = p.outer > 4 ? (uint32_t)threads * 64u : 0u;
    const size_t smem = (size_t)p.row_off + (row_bytes > xchg ? row_bytes : xchg);
    if (smem > 160u * 1024u) return hipErrorInvalidValue;
    // persistent: as many workgroups as fit a compute unit by LDS, at most two
    const int per_cu = smem * 2 <= 160u * 1024u ? 2 : 1;
    const int grid = (int)(p.ngroups < (int64_t)cus * per_cu ? p.ngroups : (int64_t)cus * per_cu);
#define ORBIT_LAUNCH(B, NB, OU, GA)                                                                \
    do {                                                                                           \
        const hipError_t e = set_smem_limit<B, NB, OU, GA>();                                      \
        if (e != hipSuccess) return e;                                                             \
        hipLaunchKernelGGL((rpbh_quantize_kernel<B, NB, OU, GA>), dim3(grid), dim3(threads), smem, stream, p); \
    } while (0)
#define ORBIT_LAUNCH_BITS(NB, OU, GA)                                                              \
    do {                                                                                           \
        if (bits == 2) ORBIT_LAUNCH(2, NB, OU, GA);                                                \
        else if (bits == 3) ORBIT_LAUNCH(3, NB, OU, GA);                                           \
        else if (bits == 6) ORBIT_LAUNCH(6, NB, OU, GA);                                           \
        else ORBIT_LAUNCH(4, NB, OU, GA);                                                          \
    } while (0)
#define ORBIT_LAUNCH_OUTER(NB, GA)                                                                 \
    do {                                                                                           \
        if (p.outer > 0) ORBIT_LAUNCH_BITS(NB, true, GA);                                          \
        else ORBIT_LAUNCH_BITS(NB, false, GA);                                                     \
    } while (0)
    if (norm_bf16) {
        if (gather) ORBIT_LAUNCH_OUTER(true, true);
        else ORBIT_LAUNCH_OUTER(true, false);
    } else {
        if (gather) ORBIT_LAUNCH_OUTER(false, true);
        else ORBIT_LAUNCH_OUTER(false, false);
    }
#undef ORBIT_LAUNCH_OUTER
#undef ORBIT_LAUNCH_BITS
#undef ORBIT_LAUNCH
    return hipGetLastError();
}

}  // namespace orbit
