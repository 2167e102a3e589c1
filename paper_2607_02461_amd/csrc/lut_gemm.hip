// LUT-decode GEMM on packed Lloyd-Max codes for gfx950 (fp16 MFMA, fp32 accumulate).
//
// Computes Y[n][i] = s_n * r'_i * sum_k L_a[xc[n][k]] * L_w[wc[i][k]]: the rotation cancels in
// the product (Sec. 4.3), so the two code sets are contracted directly in the rotated basis;
// the paper's limitations section names this codebook GEMM as the missing kernel.
//
// Decode: codes are widened to bytes and looked up with v_perm_b32 against byte tables of the
// fp16 levels (low bytes and high bytes of the 2^b levels, 8 entries per register pair), which
// needs no memory access.  Each code of a block tile is decoded exactly once, into an fp16 tile
// in LDS that the matrix cores then read.  fp16 products are exact in fp32, so the result
// differs from an fp64 evaluation with the same fp16 levels only by fp32 accumulation.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device.h"

namespace orbit {

namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int LDS_STRIDE = BK + 8;  // halves per tile row (padding against bank conflicts)

struct ByteTables {
    uint32_t lo[4], hi[4];  // byte e of lo[e/4] (hi[e/4]) is the low (high) byte of level e
};

__device__ __forceinline__ ByteTables make_tables(const uint16_t* lut, int n) {
    ByteTables t;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int e = 4 * w + b;
            const uint32_t v = e < n ? lut[e] : 0u;
            lo |= (v & 0xFFu) << (8 * b);
            hi |= (v >> 8) << (8 * b);
        }
        t.lo[w] = lo;
        t.hi[w] = hi;
    }
    return t;
}

// Four codes (one per byte of c4) -> four fp16 values as two fp16x2 words.
template <int BITS>
__device__ __forceinline__ void lookup4(uint32_t c4, const ByteTables& t, uint32_t& d0, uint32_t& d1) {
    uint32_t lo, hi;
    if constexpr (BITS <= 3) {
        lo = __builtin_amdgcn_perm(t.lo[1], t.lo[0], c4);
        hi = __builtin_amdgcn_perm(t.hi[1], t.hi[0], c4);
    } else {
        const uint32_t sel = c4 & 0x07070707u;
        const uint32_t mask = ((c4 >> 3) & 0x01010101u) * 0xFFu;
        const uint32_t lo0 = __builtin_amdgcn_perm(t.lo[1], t.lo[0], sel);
        const uint32_t lo1 = __builtin_amdgcn_perm(t.lo[3], t.lo[2], sel);
        const uint32_t hi0 = __builtin_amdgcn_perm(t.hi[1], t.hi[0], sel);
        const uint32_t hi1 = __builtin_amdgcn_perm(t.hi[3], t.hi[2], sel);
        lo = (mask & lo1) | (~mask & lo0);
        hi = (mask & hi1) | (~mask & hi0);
    }
    d0 = __builtin_amdgcn_perm(hi, lo, 0x05010400u);  // [lo0 hi0 lo1 hi1]
    d1 = __builtin_amdgcn_perm(hi, lo, 0x07030602u);  // [lo2 hi2 lo3 hi3]
}

// 32 packed codes (4*BITS bytes, LSB-first) -> 32 fp16 values in out[16] (fp16x2 words).
template <int BITS>
__device__ __forceinline__ void decode32(const uint32_t* w, const ByteTables& t, uint32_t (&out)[16]) {
    if constexpr (BITS == 4) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t even = w[i] & 0x0F0F0F0Fu;
            const uint32_t odd = (w[i] >> 4) & 0x0F0F0F0Fu;
            const uint32_t c0 = __builtin_amdgcn_perm(odd, even, 0x05010400u);  // codes 8i .. 8i+3
            const uint32_t c1 = __builtin_amdgcn_perm(odd, even, 0x07030602u);  // codes 8i+4 .. 8i+7
            lookup4<4>(c0, t, out[4 * i], out[4 * i + 1]);
            lookup4<4>(c1, t, out[4 * i + 2], out[4 * i + 3]);
        }
    } else if constexpr (BITS == 2) {
#pragma unroll
        for (int g = 0; g < 8; ++g) {
            const uint32_t x = w[g >> 2] >> (8 * (g & 3));
            const uint32_t c4 = (x & 3u) | (((x >> 2) & 3u) << 8) | (((x >> 4) & 3u) << 16) | (((x >> 6) & 3u) << 24);
            lookup4<2>(c4, t, out[2 * g], out[2 * g + 1]);
        }
    } else {
        static_assert(BITS == 3, "bits");
        const uint64_t lo64 = (uint64_t)w[0] | ((uint64_t)w[1] << 32);
        const uint64_t hi64 = (uint64_t)w[1] | ((uint64_t)w[2] << 32);
#pragma unroll
        for (int g = 0; g < 8; ++g) {
            const int bit = 12 * g;
            const uint32_t x = bit < 32 ? (uint32_t)(lo64 >> bit) : (uint32_t)(hi64 >> (bit - 32));
            const uint32_t c4 = (x & 7u) | (((x >> 3) & 7u) << 8) | (((x >> 6) & 7u) << 16) | (((x >> 9) & 7u) << 24);
            lookup4<3>(c4, t, out[2 * g], out[2 * g + 1]);
        }
    }
}

template <int BITS>
__device__ __forceinline__ void load_codes32(const uint8_t* src, uint32_t (&w)[4]) {
    if constexpr (BITS == 4) {
        const uint4 v = *(const uint4*)src;
        w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
    } else if constexpr (BITS == 2) {
        const uint2 v = *(const uint2*)src;
        w[0] = v.x; w[1] = v.y; w[2] = 0; w[3] = 0;
    } else {
        const uint32_t* s = (const uint32_t*)src;
        w[0] = s[0]; w[1] = s[1]; w[2] = s[2]; w[3] = 0;
    }
}

__device__ __forceinline__ float bf16_to_f32(uint16_t v) { return __uint_as_float((uint32_t)v << 16); }

template <int BA, int BW>
__global__ __launch_bounds__(256) void lut_gemm_kernel(GemmParams p) {
    __shared__ __align__(16) _Float16 As[BM * LDS_STRIDE];
    __shared__ __align__(16) _Float16 Bs[BN * LDS_STRIDE];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = (int64_t)blockIdx.y * BM, n0 = (int64_t)blockIdx.x * BN;
    const ByteTables ta = make_tables(p.lut_a, 1 << BA);
    const ByteTables tw = make_tables(p.lut_w, 1 << BW);

    // this thread decodes 32 codes of one A row and 32 codes of one B row per K-step
    const int lr = tid >> 1, lh = tid & 1;
    const int64_t arow = min(m0 + lr, p.M - 1), brow = min(n0 + lr, p.N - 1);
    const int64_t a_row_bytes = (int64_t)p.K * BA / 8, b_row_bytes = (int64_t)p.K * BW / 8;
    const uint8_t* asrc = p.xc + arow * a_row_bytes + lh * 4 * BA;
    const uint8_t* bsrc = p.wc + brow * b_row_bytes + lh * 4 * BW;

    floatx16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    for (int k0 = 0; k0 < p.K; k0 += BK) {
        uint32_t wa[4], wb[4], da[16], db[16];
        load_codes32<BA>(asrc + (int64_t)k0 * BA / 8, wa);
        load_codes32<BW>(bsrc + (int64_t)k0 * BW / 8, wb);
        decode32<BA>(wa, ta, da);
        decode32<BW>(wb, tw, db);
        uint4* adst = (uint4*)(As + lr * LDS_STRIDE + lh * 32);
        uint4* bdst = (uint4*)(Bs + lr * LDS_STRIDE + lh * 32);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            adst[i] = make_uint4(da[4 * i], da[4 * i + 1], da[4 * i + 2], da[4 * i + 3]);
            bdst[i] = make_uint4(db[4 * i], db[4 * i + 1], db[4 * i + 2], db[4 * i + 3]);
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
            half8 a[2], b[2];
#pragma unroll
            for (int i = 0; i < 2; ++i)
                a[i] = *(const half8*)(As + (wm * 64 + i * 32 + (lane & 31)) * LDS_STRIDE + kk * 16 + (lane >> 5) * 8);
#pragma unroll
            for (int j = 0; j < 2; ++j)
                b[j] = *(const half8*)(Bs + (wn * 64 + j * 32 + (lane & 31)) * LDS_STRIDE + kk * 16 + (lane >> 5) * 8);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
    }

    // epilogue: acc element e of a 32x32 tile sits at row 8*(e/4) + 4*(lane/32) + e%4, col lane%32
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t col = n0 + wn * 64 + j * 32 + (lane & 31);
            if (col >= p.N) continue;
            const float rw = bf16_to_f32(p.wn[col]);
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int64_t row = m0 + wm * 64 + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
                if (row < p.M) p.Y[row * p.ldy + col] = acc[i][j][e] * p.xn[row] * rw;
            }
        }
    }
}

}  // namespace

hipError_t launch_lut_gemm(const GemmParams& p, int ba, int bw, hipStream_t stream) {
    dim3 grid((unsigned)((p.N + BN - 1) / BN), (unsigned)((p.M + BM - 1) / BM));
#define ORBIT_GEMM(A, W) hipLaunchKernelGGL((lut_gemm_kernel<A, W>), grid, dim3(256), 0, stream, p)
    switch (ba * 8 + bw) {
        case 2 * 8 + 2: ORBIT_GEMM(2, 2); break;
        case 2 * 8 + 3: ORBIT_GEMM(2, 3); break;
        case 2 * 8 + 4: ORBIT_GEMM(2, 4); break;
        case 3 * 8 + 2: ORBIT_GEMM(3, 2); break;
        case 3 * 8 + 3: ORBIT_GEMM(3, 3); break;
        case 3 * 8 + 4: ORBIT_GEMM(3, 4); break;
        case 4 * 8 + 2: ORBIT_GEMM(4, 2); break;
        case 4 * 8 + 3: ORBIT_GEMM(4, 3); break;
        default: ORBIT_GEMM(4, 4); break;
    }
#undef ORBIT_GEMM
    return hipGetLastError();
}

}  // namespace orbit
