// INT4 round-to-nearest weight-only layer of the AdaLN modulation projections, for gfx950.
//
// The experimental setup (Sec. 5) keeps the adaptive-layer-norm modulation projections at INT4
// weight round-to-nearest, and the supplementary material fixes group size 64 with BF16
// activations: those layers are not rotated, because their timestep-dependent scale-and-shift
// cannot be folded into neighbouring weights and their input is one conditioning token per step.
//
// Offline: each group of 64 consecutive inputs of a weight row gets the FP16 scale
// fp16(absmax / 7) (the FP32 quotient rounded to nearest even, saturating at the largest finite
// FP16) and codes clamp(RNE(w / scale), -8, 7), the quotient in FP32; codes are stored as q + 8
// in LSB-first nibbles.
//
// Online: Y = X (q * scale)^T (+ bias) for a handful of BF16 rows of X.  The layer streams its
// weights once, so it is bound by HBM and, a few microseconds long per projection, by how much
// of it is in flight: groups of 16 lanes own two output rows, each lane issues the loads of up
// to four 32-code chunks per row before computing, and the activations sit in LDS, staged once
// by each persistent workgroup.  A code nibble u becomes the BF16 value 128 + u by OR-ing it into
// the mantissa of 128 (0x4300 | u is exact: 128..143 are BF16 integers), two per register at
// bits 0 and 16, so one v_dot2_f32_bf16 takes two codes against two activations with exact
// products; per chunk the accumulator starts at -136 * sum(x), which removes the 128 + 8 offset.
// The activations of a chunk are paired to match: element j of each 8 with element j + 4.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "device.h"

namespace orbit {

namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kRtnGroup = 64;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

// One thread per group of 64 weights: 128 bytes in, 32 bytes of codes and one FP16 scale out.
__global__ __launch_bounds__(256) void adaln_int4_quantize_kernel(const uint16_t* __restrict__ W, int64_t N, int K,
                                                                  int64_t ldw, uint8_t* __restrict__ q,
                                                                  uint16_t* __restrict__ scales) {
    const int groups = K / kRtnGroup;
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= N * groups) return;
    const int64_t n = gid / groups;
    const int g = (int)(gid - n * groups);
    const uint4* src = (const uint4*)(W + n * ldw + (int64_t)g * kRtnGroup);
    uint32_t w[32];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const uint4 v = src[i];
        w[4 * i] = v.x;
        w[4 * i + 1] = v.y;
        w[4 * i + 2] = v.z;
        w[4 * i + 3] = v.w;
    }
    float amax = 0.f;
#pragma unroll
    for (int j = 0; j < 32; ++j) amax = fmaxf(amax, fmaxf(fabsf(bf16_lo(w[j])), fabsf(bf16_hi(w[j]))));
    const _Float16 sh = (_Float16)fminf(amax / 7.0f, 65504.0f);  // IEEE fp32 quotient, then RNE to fp16
    const float s = (float)sh;
    uint32_t out[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        uint32_t word = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const uint32_t src_w = w[4 * t + (e >> 1)];
            const float v = (e & 1) ? bf16_hi(src_w) : bf16_lo(src_w);
            float r = s > 0.f ? rintf(v / s) : 0.f;  // IEEE quotient, round half to even
            r = fminf(fmaxf(r, -8.f), 7.f);
            word |= (uint32_t)((int)r + 8) << (4 * e);
        }
        out[t] = word;
    }
    uint4* dst = (uint4*)(q + n * (int64_t)(K / 2) + (int64_t)g * (kRtnGroup / 2));
    dst[0] = make_uint4(out[0], out[1], out[2], out[3]);
    dst[1] = make_uint4(out[4], out[5], out[6], out[7]);
    scales[n * groups + g] = __builtin_bit_cast(uint16_t, sh);
}

template <int CTRL>
__device__ __forceinline__ float dpp_add(float v) {
    return v + __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}

// Rows of Y per 16-lane group, groups per workgroup (a block of 32 rows), and chunks (32 codes)
// whose loads a lane issues before it computes any of them.
constexpr int kRtnRows = 2;
constexpr int kRtnLanes = 16;
constexpr int kRtnGroupsPerWg = 16;
constexpr int kRtnBatch = 4;
constexpr int kRtnBlockRows = kRtnRows * kRtnGroupsPerWg;

// Persistent: a workgroup stages its tokens once, then walks row blocks blockIdx.x, +gridDim.x, ...
template <int MT>
__global__ __launch_bounds__(256) void adaln_int4_linear_kernel(RtnLinearParams p) {
    // activations of the workgroup's MT tokens, paired per 8 as (x0,x4) (x1,x5) (x2,x6) (x3,x7),
    // then one fp32 sum per chunk of 32
    extern __shared__ __align__(16) uint32_t xlds[];
    const int nchunk = p.K / 32;
    float* const csum = (float*)(xlds + MT * (p.K / 2));
    const int m0 = blockIdx.y * MT;
    const uint32_t magic = 0x43004300u, one_one = 0x3F803F80u;

    for (int i = threadIdx.x; i < MT * (p.K / 8); i += blockDim.x) {
        const int m = i / (p.K / 8), t = i - m * (p.K / 8);
        const uint4 v = *(const uint4*)(p.X + (int64_t)min(m0 + m, (int)p.M - 1) * p.ldx + (int64_t)t * 8);
        *(uint4*)(xlds + m * (p.K / 2) + t * 4) =
            make_uint4(__builtin_amdgcn_perm(v.z, v.x, 0x05040100u), __builtin_amdgcn_perm(v.z, v.x, 0x07060302u),
                       __builtin_amdgcn_perm(v.w, v.y, 0x05040100u), __builtin_amdgcn_perm(v.w, v.y, 0x07060302u));
    }
    __syncthreads();
    for (int i = threadIdx.x; i < MT * nchunk; i += blockDim.x) {
        const uint32_t* w = xlds + (i / nchunk) * (p.K / 2) + (i % nchunk) * 16;
        float sum = 0.f;
#pragma unroll
        for (int k = 0; k < 16; ++k) sum = dot2(w[k], one_one, sum);
        csum[i] = sum;
    }
    __syncthreads();

    const int lane = threadIdx.x & (kRtnLanes - 1), grp = threadIdx.x / kRtnLanes;
    const int64_t qrow = p.K / 2, srow = p.K / kRtnGroup;
    const int64_t nblocks = (p.N + kRtnBlockRows - 1) / kRtnBlockRows;
    for (int64_t blk = blockIdx.x; blk < nblocks; blk += gridDim.x) {
        const int64_t n0 = blk * kRtnBlockRows + grp * kRtnRows;
        int64_t nrow[kRtnRows];
#pragma unroll
        for (int r = 0; r < kRtnRows; ++r) nrow[r] = min(n0 + r, p.N - 1);  // the ragged end re-reads the last row
        float tot[kRtnRows][MT];
#pragma unroll
        for (int r = 0; r < kRtnRows; ++r)
#pragma unroll
            for (int m = 0; m < MT; ++m) tot[r][m] = 0.f;

        for (int c0 = 0; c0 < nchunk; c0 += kRtnLanes * kRtnBatch) {
            // every load of the batch first; chunks past the end re-read the last one with scale 0
            uint4 cw[kRtnBatch][kRtnRows];
            float sc[kRtnBatch][kRtnRows];
            int cidx[kRtnBatch];
#pragma unroll
            for (int b = 0; b < kRtnBatch; ++b) {
                const int c = c0 + lane + kRtnLanes * b;
                cidx[b] = min(c, nchunk - 1);
                if (c0 + kRtnLanes * b >= nchunk) continue;  // the whole slot is past the end (uniform)
#pragma unroll
                for (int r = 0; r < kRtnRows; ++r) {
                    cw[b][r] = *(const uint4*)(p.q + nrow[r] * qrow + (int64_t)cidx[b] * 16);
                    const float sv = (float)__builtin_bit_cast(_Float16, p.scales[nrow[r] * srow + (cidx[b] >> 1)]);
                    sc[b][r] = c < nchunk ? sv : 0.f;
                }
            }
#pragma unroll
            for (int b = 0; b < kRtnBatch; ++b) {
                if (c0 + kRtnLanes * b >= nchunk) break;  // uniform: no chunk of this slot exists
                uint32_t xp[MT][16];
                float xs[MT];
#pragma unroll
                for (int m = 0; m < MT; ++m) {
                    const uint4* src = (const uint4*)(xlds + m * (p.K / 2) + cidx[b] * 16);
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const uint4 v = src[k];
                        xp[m][4 * k] = v.x;
                        xp[m][4 * k + 1] = v.y;
                        xp[m][4 * k + 2] = v.z;
                        xp[m][4 * k + 3] = v.w;
                    }
                    xs[m] = csum[m * nchunk + cidx[b]];
                }
#pragma unroll
                for (int r = 0; r < kRtnRows; ++r) {
                    const uint32_t words[4] = {cw[b][r].x, cw[b][r].y, cw[b][r].z, cw[b][r].w};
                    uint32_t u[16];  // (128 + u_j, 128 + u_{j+4}) of each 8 codes, as BF16 pairs
#pragma unroll
                    for (int t = 0; t < 4; ++t)
#pragma unroll
                        for (int jj = 0; jj < 4; ++jj) u[4 * t + jj] = ((words[t] >> (4 * jj)) & 0x000F000Fu) | magic;
#pragma unroll
                    for (int m = 0; m < MT; ++m) {
                        float acc = -136.f * xs[m];
#pragma unroll
                        for (int k = 0; k < 16; ++k) acc = dot2(u[k], xp[m][k], acc);
                        tot[r][m] = fmaf(sc[b][r], acc, tot[r][m]);
                    }
                }
            }
        }

        // fixed-order sum over the 16 lanes of the group (one DPP row): pairs, quads, 8, 16
#pragma unroll
        for (int r = 0; r < kRtnRows; ++r) {
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                float v = tot[r][m];
                v = dpp_add<0xB1>(v);   // quad_perm [1,0,3,2]
                v = dpp_add<0x4E>(v);   // quad_perm [2,3,0,1]
                v = dpp_add<0x141>(v);  // row_half_mirror
                v = dpp_add<0x140>(v);  // row_mirror
                const int64_t n = n0 + r;
                if (lane == 0 && n < p.N && m0 + m < p.M) {
                    if (p.bias) v += __uint_as_float((uint32_t)p.bias[n] << 16);
                    p.Y[(int64_t)(m0 + m) * p.ldy + n] = v;
                }
            }
        }
    }
}

}  // namespace

hipError_t launch_adaln_int4_quantize(const uint16_t* W, int64_t N, int K, int64_t ldw, uint8_t* q, uint16_t* scales,
                                      hipStream_t stream) {
    const int64_t total = N * (K / kRtnGroup);
    const int64_t blocks = (total + 255) / 256;
    hipLaunchKernelGGL(adaln_int4_quantize_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, W, N, K, ldw, q,
                       scales);
    return hipGetLastError();
}

hipError_t launch_adaln_int4_linear(const RtnLinearParams& p, int cus, hipStream_t stream) {
    // up to four resident workgroups per compute unit walk the row blocks
    const int64_t nblocks = (p.N + kRtnBlockRows - 1) / kRtnBlockRows;
    const unsigned gx = (unsigned)std::min<int64_t>(nblocks, (int64_t)4 * cus);
    const int mt = p.M == 1 ? 1 : 2;
    const size_t lds = (size_t)mt * (p.K / 2) * sizeof(uint32_t) + (size_t)mt * (p.K / 32) * sizeof(float);
    if (mt == 1) {
        hipLaunchKernelGGL(adaln_int4_linear_kernel<1>, dim3(gx, 1), dim3(256), lds, stream, p);
    } else {
        static std::atomic<uint64_t> attr{0};
        const hipError_t e = raise_lds_limit((const void*)adaln_int4_linear_kernel<2>, 80 * 1024, attr);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(adaln_int4_linear_kernel<2>, dim3(gx, (unsigned)((p.M + 1) / 2)), dim3(256), lds, stream, p);
    }
    return hipGetLastError();
}

}  // namespace orbit
