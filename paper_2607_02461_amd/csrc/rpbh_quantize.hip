// Fused RPBH rotate -> normalize -> Lloyd-Max encode -> pack, for gfx950.
//
// One kernel serves the online activation quantizer (Sec. 4.3, Eqs. (7)-(8)) and the offline
// weight pass (Sec. 4.2, Eqs. (4)-(6)); they differ only in the type of the stored norm.
//
// Work mapping (h = 128): a workgroup owns R rows at a time.  Each row is staged in LDS as raw
// bf16 with 16-byte coalesced loads.  Every 128-block of a row belongs to one quad of lanes;
// lane q of the quad holds the 32 consecutive post-permutation positions q*32 .. q*32+31 of the
// block in registers.  The permutation gather reads LDS through a per-lane table that also
// carries the Rademacher sign, so gather, sign and bf16->fp32 widening cost one LDS read and
// one VALU op per element.  The Walsh-Hadamard butterflies over the five register bits of the
// position run in registers; the two remaining stages cross lanes of the quad with DPP
// quad permutations.  Those two stages compute own + sign*partner, which leaves the upper
// lane of each pair holding the negated butterfly output; that sign is fixed per lane
// (sigma = (-1)^popcount(q)) and is folded into the per-row scale used by the encoder.
// The row's squared norm is reduced deterministically (quad DPP, then a per-row pass over
// the block partials in LDS), after which each lane encodes its 32 coordinates against the
// fp32 thresholds and writes them packed: 32 codes are 4*b bytes, one vector store per lane.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device.h"

namespace orbit {

namespace {

template <int CTRL>
__device__ __forceinline__ float quad_perm(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kQuadXor1 = 0xB1;  // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;  // quad_perm [2,3,0,1]

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float x) {
    uint32_t b = __float_as_uint(x);
    b += 0x7FFFu + ((b >> 16) & 1u);
    return (uint16_t)(b >> 16);
}

template <int BITS>
__device__ __forceinline__ void store_codes(uint8_t* dst, const int (&code)[32]) {
    if constexpr (BITS == 4) {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            uint32_t v = 0;
#pragma unroll
            for (int t = 0; t < 8; ++t) v |= (uint32_t)code[8 * i + t] << (4 * t);
            w[i] = v;
        }
        *(uint4*)dst = make_uint4(w[0], w[1], w[2], w[3]);
    } else if constexpr (BITS == 2) {
        uint32_t w[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            uint32_t v = 0;
#pragma unroll
            for (int t = 0; t < 16; ++t) v |= (uint32_t)code[16 * i + t] << (2 * t);
            w[i] = v;
        }
        *(uint2*)dst = make_uint2(w[0], w[1]);
    } else {
        static_assert(BITS == 3, "bits");
        uint32_t w[3] = {0u, 0u, 0u};
#pragma unroll
        for (int r = 0; r < 32; ++r) {
            const int pos = 3 * r, wi = pos >> 5, sh = pos & 31;
            w[wi] |= (uint32_t)code[r] << sh;
            if (sh > 29) w[wi + 1] |= (uint32_t)code[r] >> (32 - sh);
        }
        uint32_t* d = (uint32_t*)dst;
        d[0] = w[0];
        d[1] = w[1];
        d[2] = w[2];
    }
}

template <int BITS, bool NORM_BF16>
__global__ __launch_bounds__(512) void rpbh_quantize_kernel(QuantParams p) {
    extern __shared__ __align__(16) unsigned char smem[];
    constexpr int NTHR = (1 << BITS) - 1;
    const int K = p.K, nb = p.nb, R = p.R;
    uint16_t* rows = (uint16_t*)smem;                       // R x K bf16
    float* part = (float*)(smem + (size_t)R * K * 2);       // R x nb block partial sums
    float* rowss = part + R * nb;                           // R row sums
    const int tid = threadIdx.x, T = blockDim.x;
    const int task = tid >> 2, q = tid & 3;
    const int rg = task / nb, blk = task - rg * nb;
    const bool active = task < R * nb;

    uint32_t meta[32];
    if (active) {
        const uint4* src = (const uint4*)(p.meta + blk * 128 + q * 32);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            uint4 v = src[i];
            meta[4 * i] = v.x;
            meta[4 * i + 1] = v.y;
            meta[4 * i + 2] = v.z;
            meta[4 * i + 3] = v.w;
        }
    }
    const float sgn1 = (q & 1) ? -1.f : 1.f;
    const float sgn2 = (q & 2) ? -1.f : 1.f;
    const float sigma = sgn1 * sgn2;
    const int chunks = K >> 3;  // 16-byte chunks per row
    const int64_t code_row_bytes = (int64_t)K * BITS / 8;

    for (int g = blockIdx.x; g < p.ngroups; g += gridDim.x) {
        const int64_t row0 = (int64_t)g * R;
        const int nrows = (int)min((int64_t)R, p.M - row0);
        for (int c = tid; c < nrows * chunks; c += T) {
            const int r = c / chunks, o = c - r * chunks;
            const uint4 v = *(const uint4*)(p.X + (row0 + r) * p.ldx + (int64_t)o * 8);
            *(uint4*)(rows + (size_t)r * K + (size_t)o * 8) = v;
        }
        __syncthreads();

        const bool live = active && rg < nrows;
        float z[32];
        if (live) {
            const unsigned char* myrow = (const unsigned char*)(rows + (size_t)rg * K);
#pragma unroll
            for (int r = 0; r < 32; ++r) {
                const uint32_t m = meta[r];
                const uint32_t b = *(const uint16_t*)(myrow + (m & 0xFFFFu));
                z[r] = __uint_as_float((b << 16) ^ (m & 0x80000000u));
            }
#pragma unroll
            for (int s = 1; s < 32; s <<= 1) {
#pragma unroll
                for (int r = 0; r < 32; ++r) {
                    if (r & s) continue;
                    const float a = z[r], b = z[r + s];
                    z[r] = a + b;
                    z[r + s] = a - b;
                }
            }
#pragma unroll
            for (int r = 0; r < 32; ++r) z[r] = fmaf(quad_perm<kQuadXor1>(z[r]), sgn1, z[r]);
#pragma unroll
            for (int r = 0; r < 32; ++r) z[r] = fmaf(quad_perm<kQuadXor2>(z[r]), sgn2, z[r]);
            float ss = 0.f;
#pragma unroll
            for (int r = 0; r < 32; ++r) ss = fmaf(z[r], z[r], ss);
            ss += quad_perm<kQuadXor1>(ss);
            ss += quad_perm<kQuadXor2>(ss);
            if (q == 0) part[rg * nb + blk] = ss;
        }
        __syncthreads();

        const int wave = tid >> 6, lane = tid & 63, nwaves = T >> 6;
        for (int r = wave; r < nrows; r += nwaves) {
            float acc = 0.f;
            for (int i = lane; i < nb; i += 64) acc += part[r * nb + i];
            acc = wave_sum(acc);
            if (lane == 0) {
                rowss[r] = acc;
                const float s = sqrtf(acc * (1.0f / 128.0f));
                if constexpr (NORM_BF16)
                    ((uint16_t*)p.norm)[row0 + r] = f32_to_bf16_rne(s);
                else
                    ((float*)p.norm)[row0 + r] = s;
            }
        }
        __syncthreads();

        if (live) {
            const float s = sqrtf(rowss[rg] * (1.0f / 128.0f));
            // u = z / (s + eps) with z = z_unnormalised / sqrt(128); sigma undoes the lane sign
            const float scale = sigma / ((s + p.eps) * 11.313708498984761f);
            int code[32];
#pragma unroll
            for (int r = 0; r < 32; ++r) {
                const float u = z[r] * scale;
                int c = 0;
#pragma unroll
                for (int j = 0; j < NTHR; ++j) c += (u >= p.thr[j]) ? 1 : 0;
                code[r] = c;
            }
            uint8_t* dst = p.codes + (row0 + rg) * code_row_bytes + (int64_t)(blk * 4 + q) * 4 * BITS;
            store_codes<BITS>(dst, code);
        }
        __syncthreads();
    }
}

}  // namespace

size_t quant_smem_bytes(int K, int R) {
    const int nb = K / 128;
    return (size_t)R * K * 2 + (size_t)R * nb * 4 + (size_t)R * 4;
}

int quant_rows_per_group(int K) {
    const int nb = K / 128;
    return nb >= 128 ? 1 : 128 / nb;
}

hipError_t launch_rpbh_quantize(const QuantParams& p, int bits, bool norm_bf16, int grid, hipStream_t stream) {
    const int threads = ((p.R * p.nb * 4 + 63) / 64) * 64;
    const size_t smem = quant_smem_bytes(p.K, p.R);
#define ORBIT_LAUNCH(B, NB)                                                                   \
    hipLaunchKernelGGL((rpbh_quantize_kernel<B, NB>), dim3(grid), dim3(threads), smem, stream, p)
    if (norm_bf16) {
        if (bits == 2) ORBIT_LAUNCH(2, true);
        else if (bits == 3) ORBIT_LAUNCH(3, true);
        else ORBIT_LAUNCH(4, true);
    } else {
        if (bits == 2) ORBIT_LAUNCH(2, false);
        else if (bits == 3) ORBIT_LAUNCH(3, false);
        else ORBIT_LAUNCH(4, false);
    }
#undef ORBIT_LAUNCH
    return hipGetLastError();
}

}  // namespace orbit
