// Kernel parameter blocks and launchers shared by the device entry points and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <mutex>

namespace orbit {

// A kernel's dynamic-LDS limit is a per-device attribute: raise it once on the current device
// (bit `device` of `done` records that; device ordinals are below 64).
inline hipError_t raise_lds_limit(const void* kernel, int bytes, std::atomic<uint64_t>& done) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const uint64_t bit = 1ull << (dev & 63);
    if (done.load(std::memory_order_acquire) & bit) return hipSuccess;
    e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e == hipSuccess) done.fetch_or(bit, std::memory_order_acq_rel);
    return e;
}

// Workgroups of `kernel` resident on one compute unit at `threads` threads and `smem` bytes of
// dynamic LDS (registers, LDS and wave slots together), looked up once per shape.
inline int resident_blocks(const void* kernel, int threads, size_t smem) {
    struct Entry {
        const void* k;
        int t;
        size_t s;
        int n;
    };
    static std::mutex mu;
    static Entry cache[64];
    static int used = 0;
    std::lock_guard<std::mutex> lk(mu);
    for (int i = 0; i < used; ++i)
        if (cache[i].k == kernel && cache[i].t == threads && cache[i].s == smem) return cache[i].n;
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, threads, smem) != hipSuccess || n < 1) n = 1;
    if (used < 64) cache[used++] = Entry{kernel, threads, smem, n};
    return n;
}

// Fused RPBH quantizer (activations: fp32 norms; weights: bf16 norms).
struct QuantParams {
    const uint16_t* X;     // bf16 [M][ldx]
    int64_t ldx;           // elements
    int64_t M;
    const uint32_t* meta;  // [K]: 2*perm[j], the byte offset of the gathered element in a staged row,
                           // with bit 31 set where sign[j] = -1
    const uint32_t* smask; // [K/2]: bf16 sign bits of position pairs (the identity-permutation path)
    uint8_t* codes;        // [M][K*bits/8]
    void* norm;            // fp32 or bf16 [M]
    int K, nb, R;          // input dim, K/128 blocks, rows staged per workgroup iteration
    int ngroups;           // ceil(M / R)
    float eps;
    const float* enc;      // encoder table: per-cell bias (see the codebook's encoder table)
    int ncell;
    float enc_inv_w;       // cells per unit of the normalized coordinate
    float enc_center;      // C: the (integer) cell of u = 0
    uint32_t one_one;      // bf16 pair (1.0, 1.0), 0x3F803F80
    int outer;             // log2(h / 128): Hadamard stages across 128-blocks (0 for h = 128)
    float sqrt_h;          // sqrt(h), the FWHT's normalization
    // staging: the row of 16-byte chunk c of a group is (c * row_magic) >> row_shift (exact for
    // every chunk a workgroup stages), and the chunk sits row_gap = 2*(ldx - K) bytes per row
    // further than in a contiguous group
    uint32_t row_magic, row_shift, row_gap;
    // LDS layout in bytes (set by the launcher): encoder table at 0, block partials at part_off,
    // staged rows at row_off and their negated copy neg_off bytes further
    uint32_t part_off, row_off, neg_off;
};

// Stored code labels.  A b-bit code of level index c (levels ascending) is stored as the
// sign-magnitude label: c - 2^(b-1) for the upper half (positive levels) and 2^b - 1 - c for the
// lower half, so the top bit is the level's sign and the low b-1 bits rank its magnitude.  On a
// word of packed fields whose top bits are TOP, SHIFT = b - 1 apart from each field's bit 0, and
// whose bits are MASK: t - (t >> SHIFT) is 2^(b-1) - 1 in fields with the top bit set (no borrow
// leaves a field), so ~x ^ that is c - 2^(b-1) there and 2^b - 1 - c elsewhere.
template <uint32_t TOP, int SHIFT, uint32_t MASK>
__device__ __forceinline__ uint32_t sign_magnitude_labels(uint32_t x) {
    const uint32_t t = x & TOP;
    return (~x ^ (t - (t >> SHIFT))) & MASK;
}

int quant_rows_per_group(int K);
// The one-row-per-workgroup quantizer (16 positions per lane) covers permutation plans with
// h = 128 .. 1024 and K a multiple of 128 and of h from 1024 to 16384; the general kernel covers
// the rest.  Its persistent grid holds as many workgroups as are resident at once.
bool rpbh_quantize_row_fits(int K, int h, bool gather);
hipError_t launch_rpbh_quantize_row(QuantParams p, int bits, bool norm_bf16, int cus, hipStream_t stream);
// gather: apply the permutation through the LDS-staged gather (false only for the identity).
// Launches a persistent grid of at most two workgroups per compute unit.
hipError_t launch_rpbh_quantize(QuantParams p, int bits, bool norm_bf16, bool gather, int cus, hipStream_t stream);

// LUT-decode GEMM: Y = diag(sx) La[Xc] (Lw[Wc])^T diag(rw).
struct GemmParams {
    const uint8_t* xc;     // [M][K*ba/8]
    const float* xn;       // [M]
    const uint8_t* wc;     // [N][K*bw/8]
    const uint16_t* wn;    // bf16 [N]
    void* Y;               // fp32 or bf16 [M][ldy]
    int64_t M, N, ldy;
    int K;
    int vec4;              // Y, ldy, wn and bias allow 4-wide row stores and loads
    const uint16_t* bias;  // bf16 [N] or null, added after the rescaling
    int gelu;              // apply x * Phi(x) (erfc to 1.2e-7 fractional error) after the bias
    int out_bf16;          // store Y as bf16 (round to nearest even) instead of fp32
    uint16_t lut_a[64];    // bf16 levels (2^ba used)
    uint16_t lut_w[16];    // bf16 levels (2^bw used)
    // K-split of the 128x128 kernel's rows (caller workspace): fp32 partial sums [splits][M][N]
    // of the rows it runs, each split split_steps K-steps of 64; ws = null runs unsplit
    float* ws;
    int splits, split_steps;
};

hipError_t launch_lut_gemm(const GemmParams& p, int ba, int bw, int cus, hipStream_t stream);
// Rows [0, m_big) of an M x N layer run on the 256x256 kernel, the rest on the 128x128 kernel
int64_t lut_gemm_big_rows(int64_t M, int64_t N, int cus);
// K-splits of the 128x128 kernel on M x N outputs when a workspace is given (1: none), and the
// K-steps per split (the last split may have fewer)
int lut_gemm_small_splits(int64_t M, int64_t N, int64_t K, int cus, int* split_steps);

// INT4 round-to-nearest (group 64) weight-only layer of the AdaLN modulation projections.
struct RtnLinearParams {
    const uint16_t* X;       // bf16 [M][ldx]
    int64_t M, ldx;
    const uint8_t* q;        // [N][K/2]: code + 8 per nibble, LSB-first
    const uint16_t* scales;  // fp16 [N][K/64]
    int64_t N;
    int K;
    const uint16_t* bias;    // bf16 [N] or null
    float* Y;                // fp32 [M][ldy]
    int64_t ldy;
};

hipError_t launch_adaln_int4_quantize(const uint16_t* W, int64_t N, int K, int64_t ldw, uint8_t* q, uint16_t* scales,
                                      hipStream_t stream);
hipError_t launch_adaln_int4_linear(const RtnLinearParams& p, int cus, hipStream_t stream);

}  // namespace orbit
