// Device entry points of the C ABI: argument checks, per-device plan tables, kernel launches.
#include <hip/hip_runtime.h>

#include <cmath>
#include <algorithm>
#include <cstring>
#include <vector>

#include "device.h"
#include "internal.h"

using namespace orbit;

namespace {

constexpr int kQuantH = 128;       // the fused quantizer's in-register transform (larger h adds stages)
constexpr int64_t kQuantMaxK = 16384;
constexpr int kQuantMaxH = 4096;  // block sizes 128 .. 4096 (the FWHT's stages across blocks)
constexpr int kQuantMaxCells = 8192;  // encoder table cells (LDS budget; 6-bit tables reach ~4300 at K = 16384)

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

orbit_status hip_fail(hipError_t e, const char* what) {
    return fail(ORBIT_EHIP, "%s: %s (%s)", what, hipGetErrorString(e), hipGetErrorName(e));
}

struct DeviceInfo {
    int cus = 0;
};
DeviceInfo g_dev[kMaxDevices];
std::mutex g_dev_mu;

orbit_status current_device(int* dev, DeviceInfo* info) {
    hipError_t e = hipGetDevice(dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (*dev < 0 || *dev >= kMaxDevices) return fail(ORBIT_EUNSUPPORTED, "device ordinal %d out of range", *dev);
    std::lock_guard<std::mutex> lk(g_dev_mu);
    if (g_dev[*dev].cus == 0) {
        int cus = 0;
        e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, *dev);
        if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
        g_dev[*dev].cus = cus > 0 ? cus : 1;
    }
    *info = g_dev[*dev];
    return ORBIT_OK;
}

// The plan's tables on device `dev`: K gather offsets (2*perm[j], the byte offset of the element
// that moves to position j, with bit 31 set where sign[j] = -1) followed by K/2 sign masks over
// positions (bit 15 / bit 31 of word i carry sign[2i] / sign[2i+1]), which the identity-permutation
// path applies to the pairs it loads.  Built and copied once per device, at set-up (handle creation
// or an explicit upload), never from a device call.
orbit_status plan_upload_dev(orbit_plan p, int dev) {
    std::lock_guard<std::mutex> lk(p->mu);
    if (p->dev_meta[dev]) return ORBIT_OK;
    const int64_t d = p->d;
    std::vector<uint32_t> meta;
    try {
        meta.assign((size_t)(d + (d + 1) / 2), 0u);
    } catch (...) {
        return fail(ORBIT_ENOMEM, "plan upload: out of host memory");
    }
    for (int64_t j = 0; j < d; ++j) {
        meta[j] = (uint32_t)p->perm[j] * 2u | (p->sign[j] < 0 ? 0x80000000u : 0u);
        if (p->sign[j] < 0) meta[d + j / 2] |= (j & 1) ? 0x80000000u : 0x8000u;
    }
    void* dp = nullptr;
    hipError_t e = hipMalloc(&dp, meta.size() * sizeof(uint32_t));
    if (e != hipSuccess)
        return e == hipErrorOutOfMemory ? fail(ORBIT_ENOMEM, "plan upload: hipMalloc failed") : hip_fail(e, "hipMalloc");
    e = hipMemcpy(dp, meta.data(), meta.size() * sizeof(uint32_t), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(dp);
        return hip_fail(e, "plan upload: hipMemcpy");
    }
    p->dev_meta[dev] = (uint32_t*)dp;
    return ORBIT_OK;
}

// The codebook's encoder table on device `dev`, copied once per device at set-up.
orbit_status codebook_upload_dev(orbit_codebook c, int dev) {
    std::lock_guard<std::mutex> lk(c->mu);
    if (c->dev_enc[dev]) return ORBIT_OK;
    const size_t bytes = c->enc.bias.size() * sizeof(float);
    void* d = nullptr;
    hipError_t e = hipMalloc(&d, bytes);
    if (e != hipSuccess)
        return e == hipErrorOutOfMemory ? fail(ORBIT_ENOMEM, "codebook upload: hipMalloc failed") : hip_fail(e, "hipMalloc");
    e = hipMemcpy(d, c->enc.bias.data(), bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(d);
        return hip_fail(e, "codebook upload: hipMemcpy");
    }
    c->dev_enc[dev] = (float*)d;
    return ORBIT_OK;
}

// Scratch of the allocation-free layer (orbit_qlinear_noalloc): the K-split's fp32 partial sums
// live in this file-scope device array instead of a caller workspace.  Every device that loads the
// library holds its own copy until the process ends, and every call on a device shares it.  In host
// code `scratch` names a host-side stand-in, not device memory: kernels get the address resolved
// below, per device, and never the name itself.
constexpr size_t kScratchBytes = (size_t)32 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
void* g_scratch[kMaxDevices] = {};
std::mutex g_scratch_mu;

// The device address of `scratch` on device `dev` (the current device), looked up once per device.
orbit_status scratch_on(int dev, void** out) {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress((void**)&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        g_scratch[dev] = ptr;
    }
    *out = g_scratch[dev];
    return ORBIT_OK;
}

// The current device, or -1 when no HIP device is visible (handles then stay host-only).
orbit_status device_for_upload(int* dev) {
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess || n <= 0) {
        (void)hipGetLastError();  // leave no sticky error behind on a machine without a GPU
        *dev = -1;
        return ORBIT_OK;
    }
    hipError_t e = hipGetDevice(dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (*dev < 0 || *dev >= kMaxDevices) return fail(ORBIT_EUNSUPPORTED, "device ordinal %d out of range", *dev);
    return ORBIT_OK;
}

// Tables of a handle on the device of a call: present since set-up, or the call is refused (a
// device call only enqueues work; it never allocates or copies synchronously).
orbit_status plan_meta(orbit_plan p, int dev, const uint32_t** out) {
    std::lock_guard<std::mutex> lk(p->mu);
    if (!p->dev_meta[dev])
        return fail(ORBIT_EINVAL, "the plan has no tables on device %d: create it with that device current, or call "
                                  "rpbh_plan_upload there first", dev);
    *out = p->dev_meta[dev];
    return ORBIT_OK;
}

orbit_status codebook_enc(orbit_codebook c, int dev, const float** out) {
    std::lock_guard<std::mutex> lk(c->mu);
    if (!c->dev_enc[dev])
        return fail(ORBIT_EINVAL, "the codebook has no encoder table on device %d: create it with that device "
                                  "current, or call lloydmax_codebook_upload there first", dev);
    *out = c->dev_enc[dev];
    return ORBIT_OK;
}

orbit_status quantize_rows(const char* who, orbit_plan p, orbit_codebook cb, const uint16_t* X, int64_t M, int64_t K,
                           int64_t ldx, float eps, uint8_t* codes, void* norm, bool norm_bf16, void* stream) {
    clear_error();
    if (!p || !cb) return fail(ORBIT_EINVAL, "%s: plan or codebook is NULL", who);
    if (M < 0) return fail(ORBIT_EINVAL, "%s: negative row count %lld", who, (long long)M);
    if (K != p->d || K != cb->d)
        return fail(ORBIT_EINVAL, "%s: K=%lld but plan.d=%lld and codebook.d=%lld", who, (long long)K, (long long)p->d,
                    (long long)cb->d);
    if (!(eps >= 0.0f) || !std::isfinite(eps)) return fail(ORBIT_EINVAL, "%s: eps must be finite and >= 0", who);
    if (ldx < K || ldx % 8 != 0) return fail(ORBIT_EINVAL, "%s: ld=%lld must be >= K and a multiple of 8", who, (long long)ldx);
    if (p->h < kQuantH || p->h > kQuantMaxH)
        return fail(ORBIT_EUNSUPPORTED, "%s: block size h=%d not implemented (powers of two 128..%d are)", who, p->h,
                    kQuantMaxH);
    if (cb->bits < 2 || cb->bits > 6 || cb->bits == 5)
        return fail(ORBIT_EUNSUPPORTED, "%s: %d-bit codes not implemented (2, 3, 4 and 6 are)", who, cb->bits);
    if (K > kQuantMaxK) return fail(ORBIT_EUNSUPPORTED, "%s: K=%lld above %lld", who, (long long)K, (long long)kQuantMaxK);
    if ((int64_t)quant_rows_per_group((int)K) * ldx * 2 >= ((int64_t)1 << 31) || (ldx - K) * 2 >= ((int64_t)1 << 24))
        return fail(ORBIT_EUNSUPPORTED, "%s: row stride %lld too large", who, (long long)ldx);
    if (M > INT32_MAX) return fail(ORBIT_EUNSUPPORTED, "%s: M=%lld above 2^31-1 rows", who, (long long)M);
    if (cb->enc.ncell > kQuantMaxCells)
        return fail(ORBIT_EUNSUPPORTED, "%s: encoder table of %d cells exceeds %d", who, cb->enc.ncell, kQuantMaxCells);
    if (M == 0) return ORBIT_OK;
    if (!X || !codes || !norm) return fail(ORBIT_EINVAL, "%s: null device pointer", who);
    if (!aligned(X, 16) || !aligned(codes, 16) || !aligned(norm, norm_bf16 ? 2 : 4))
        return fail(ORBIT_EINVAL, "%s: misaligned pointer (input and codes need 16 bytes)", who);
    int dev;
    DeviceInfo info;
    orbit_status st = current_device(&dev, &info);
    if (st != ORBIT_OK) return st;
    const uint32_t* meta = nullptr;
    st = plan_meta(p, dev, &meta);
    if (st != ORBIT_OK) return st;
    const float* enc = nullptr;
    st = codebook_enc(cb, dev, &enc);
    if (st != ORBIT_OK) return st;

    QuantParams q{};
    q.X = X;
    q.ldx = ldx;
    q.M = M;
    q.meta = meta;
    q.smask = meta + K;
    q.codes = codes;
    q.norm = norm;
    q.K = (int)K;
    q.nb = (int)(K / kQuantH);
    // rows per group: the most a workgroup holds, or fewer when that leaves compute units idle
    // (a few hundred rows: one row per workgroup spreads them over the device)
    q.R = (int)std::min<int64_t>(quant_rows_per_group((int)K), (M + info.cus - 1) / info.cus);
    q.ngroups = (int)((M + q.R - 1) / q.R);
    q.eps = eps;
    q.enc = enc;
    q.ncell = cb->enc.ncell;
    q.enc_inv_w = cb->enc.inv_w;
    q.enc_center = cb->enc.center;
    q.one_one = 0x3F803F80u;
    q.outer = 0;
    while ((kQuantH << q.outer) < p->h) ++q.outer;
    q.sqrt_h = (float)std::sqrt((double)p->h);
    // row of a staged chunk: an exact multiply-shift division by the chunks per row d for every
    // chunk index a workgroup stages (4 per thread, at most 512 threads: below 2^11).  With
    // s = 11 + ceil(log2 d) and m = ceil(2^s / d), m d - 2^s < d <= 2^(s - 11), so
    // floor(c m / 2^s) = floor(c / d) for c < 2^11 (Granlund and Montgomery, PLDI 1994); c m stays
    // below 2^24 for the kernel's 24-bit multiply.
    {
        const uint32_t cpr = (uint32_t)(K / 8);
        uint32_t lg = 0;
        while ((1u << lg) < cpr) ++lg;
        q.row_shift = 11 + lg;
        q.row_magic = (uint32_t)(((1ull << q.row_shift) + cpr - 1) / cpr);
        q.row_gap = (uint32_t)((ldx - K) * 2);
    }
    hipError_t e = rpbh_quantize_row_fits((int)K, p->h, !p->identity)
                       ? launch_rpbh_quantize_row(q, cb->bits, norm_bf16, info.cus, (hipStream_t)stream)
                       : launch_rpbh_quantize(q, cb->bits, norm_bf16, !p->identity, info.cus, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, who);
    return ORBIT_OK;
}

// Frees a handle's per-device tables (each on its own device).
template <typename T>
void free_per_device(T* (&ptrs)[kMaxDevices]) {
    for (int dev = 0; dev < kMaxDevices; ++dev) {
        if (ptrs[dev]) {
            int cur = 0;
            (void)hipGetDevice(&cur);
            (void)hipSetDevice(dev);
            (void)hipFree(ptrs[dev]);
            (void)hipSetDevice(cur);
            ptrs[dev] = nullptr;
        }
    }
}

}  // namespace

orbit_status orbit::upload_on_create(orbit_plan p, orbit_codebook c) {
    int dev;
    orbit_status st = device_for_upload(&dev);
    if (st != ORBIT_OK || dev < 0) return st;
    // per-device set-up of the allocation-free layer's scratch address as well
    void* sp = nullptr;
    st = scratch_on(dev, &sp);
    if (st != ORBIT_OK) return st;
    return p ? plan_upload_dev(p, dev) : codebook_upload_dev(c, dev);
}

extern "C" {

orbit_status rpbh_plan_upload(orbit_plan p) {
    clear_error();
    if (!p) return fail(ORBIT_EINVAL, "rpbh_plan_upload: plan is NULL");
    int dev;
    DeviceInfo info;
    orbit_status st = current_device(&dev, &info);
    if (st != ORBIT_OK) return st;
    void* sp = nullptr;
    st = scratch_on(dev, &sp);
    if (st != ORBIT_OK) return st;
    return plan_upload_dev(p, dev);
}

orbit_status lloydmax_codebook_upload(orbit_codebook c) {
    clear_error();
    if (!c) return fail(ORBIT_EINVAL, "lloydmax_codebook_upload: codebook is NULL");
    int dev;
    DeviceInfo info;
    orbit_status st = current_device(&dev, &info);
    if (st != ORBIT_OK) return st;
    void* sp = nullptr;
    st = scratch_on(dev, &sp);
    if (st != ORBIT_OK) return st;
    return codebook_upload_dev(c, dev);
}

void rpbh_plan_destroy(orbit_plan p) {
    if (!p) return;
    free_per_device(p->dev_meta);
    delete p;
}

void lloydmax_codebook_destroy(orbit_codebook c) {
    if (!c) return;
    free_per_device(c->dev_enc);
    delete c;
}

orbit_status quantize_weights_offline(orbit_plan p, orbit_codebook cb_w, const uint16_t* W, int64_t N, int64_t K,
                                      int64_t ldw, float eps, uint8_t* w_codes, uint16_t* w_norm, void* stream) {
    return quantize_rows("quantize_weights_offline", p, cb_w, W, N, K, ldw, eps, w_codes, w_norm, true, stream);
}

orbit_status rpbh_quantize_act(orbit_plan p, orbit_codebook cb_a, const uint16_t* X, int64_t M, int64_t K, int64_t ldx,
                               float eps, uint8_t* x_codes, float* x_norm, void* stream) {
    return quantize_rows("rpbh_quantize_act", p, cb_a, X, M, K, ldx, eps, x_codes, x_norm, false, stream);
}

orbit_status orbit_qlinear_ws(orbit_codebook cb_a, const uint8_t* x_codes, const float* x_norm, int64_t M,
                              orbit_codebook cb_w, const uint8_t* w_codes, const uint16_t* w_norm, int64_t N,
                              int64_t K, const uint16_t* bias, int32_t act, int32_t out_dtype, void* Y, int64_t ldy,
                              void* workspace, size_t workspace_bytes, void* stream) {
    clear_error();
    if (!cb_a || !cb_w) return fail(ORBIT_EINVAL, "orbit_qlinear: codebook is NULL");
    if (M < 0 || N < 0) return fail(ORBIT_EINVAL, "orbit_qlinear: negative M or N");
    if (K != cb_a->d || K != cb_w->d)
        return fail(ORBIT_EINVAL, "orbit_qlinear: K=%lld but codebooks have d=%lld and d=%lld", (long long)K,
                    (long long)cb_a->d, (long long)cb_w->d);
    if (ldy < N) return fail(ORBIT_EINVAL, "orbit_qlinear: ldy=%lld < N=%lld", (long long)ldy, (long long)N);
    if (act != ORBIT_ACT_NONE && act != ORBIT_ACT_GELU) return fail(ORBIT_EINVAL, "orbit_qlinear: unknown act %d", act);
    if (out_dtype != ORBIT_OUT_F32 && out_dtype != ORBIT_OUT_BF16)
        return fail(ORBIT_EINVAL, "orbit_qlinear: unknown out_dtype %d", out_dtype);
    if (cb_a->bits < 2 || cb_a->bits > 6 || cb_a->bits == 5 || cb_w->bits < 2 || cb_w->bits > 4)
        return fail(ORBIT_EUNSUPPORTED,
                    "orbit_qlinear: bit-widths (a %d, w %d) not implemented (activations 2, 3, 4, 6; weights 2..4)",
                    cb_a->bits, cb_w->bits);
    if (K % 64 != 0 || K > (int64_t)1 << 30) return fail(ORBIT_EUNSUPPORTED, "orbit_qlinear: K=%lld must be a multiple of 64", (long long)K);
    // tile counts and grid sizes are 32-bit
    if (M > INT32_MAX || N > INT32_MAX || ((M + 255) / 256) * ((N + 255) / 256) > (INT32_MAX >> 4))
        return fail(ORBIT_EUNSUPPORTED, "orbit_qlinear: M=%lld x N=%lld exceeds the launch grid", (long long)M,
                    (long long)N);
    if (M == 0 || N == 0) return ORBIT_OK;
    const int ysize = out_dtype == ORBIT_OUT_BF16 ? 2 : 4;
    if (!x_codes || !x_norm || !w_codes || !w_norm || !Y) return fail(ORBIT_EINVAL, "orbit_qlinear: null device pointer");
    if (!aligned(x_codes, 16) || !aligned(w_codes, 16) || !aligned(x_norm, 4) || !aligned(w_norm, 2) ||
        !aligned(Y, ysize) || (bias && !aligned(bias, 2)))
        return fail(ORBIT_EINVAL, "orbit_qlinear: misaligned pointer (codes need 16 bytes)");
    int dev;
    DeviceInfo info;
    orbit_status st = current_device(&dev, &info);
    if (st != ORBIT_OK) return st;
    GemmParams g{};
    g.xc = x_codes;
    g.xn = x_norm;
    g.wc = w_codes;
    g.wn = w_norm;
    g.Y = Y;
    g.M = M;
    g.N = N;
    g.ldy = ldy;
    g.K = (int)K;
    g.bias = bias;
    g.gelu = act == ORBIT_ACT_GELU;
    g.out_bf16 = out_dtype == ORBIT_OUT_BF16;
    g.vec4 = aligned(Y, 4 * ysize) && ldy % 4 == 0 && aligned(w_norm, 8) && (!bias || aligned(bias, 8));
    // K-split of the rows the 128x128 kernel runs, when the caller's workspace holds the partial sums
    const int64_t m_small = M - lut_gemm_big_rows(M, N, info.cus);
    g.splits = m_small > 0 ? lut_gemm_small_splits(m_small, N, K, info.cus, &g.split_steps) : 1;
    if (g.splits > 1 && workspace && aligned(workspace, 16) &&
        workspace_bytes >= (size_t)g.splits * (size_t)m_small * (size_t)N * sizeof(float))
        g.ws = (float*)workspace;
    else
        g.splits = 1;
    for (const orbit_codebook_s* cb : {cb_a, cb_w}) {
        // the 4-bit decoder reads the positive half and takes the sign from the label's top bit
        if (cb->bits != 4) continue;
        for (int c = 0; c < 8; ++c)
            if (cb->lut_bf16[15 - c] != (uint16_t)(cb->lut_bf16[c] ^ 0x8000u))
                return fail(ORBIT_EINTERNAL, "orbit_qlinear: 4-bit bf16 levels are not antisymmetric");
    }
    // the levels in label order: label l < 2^(b-1) is level index 2^(b-1) + l, label l above that
    // is level index 2^b - 1 - l
    auto by_label = [](const orbit_codebook_s* cb, int l) -> uint16_t {
        const int n = 1 << cb->bits, half = n / 2;
        return cb->lut_bf16[l < half ? half + l : n - 1 - l];
    };
    for (int j = 0; j < 64; ++j) g.lut_a[j] = j < (1 << cb_a->bits) ? by_label(cb_a, j) : 0;
    for (int j = 0; j < 16; ++j) g.lut_w[j] = j < (1 << cb_w->bits) ? by_label(cb_w, j) : 0;
    hipError_t e = launch_lut_gemm(g, cb_a->bits, cb_w->bits, info.cus, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "orbit_qlinear");
    return ORBIT_OK;
}

orbit_status adaln_int4_quantize_weights(const uint16_t* W, int64_t N, int64_t K, int64_t ldw, uint8_t* q,
                                         uint16_t* scales, void* stream) {
    clear_error();
    if (N < 0) return fail(ORBIT_EINVAL, "adaln_int4_quantize_weights: negative N");
    if (K <= 0 || K % 64 != 0) return fail(ORBIT_EINVAL, "adaln_int4_quantize_weights: K=%lld must be a positive multiple of 64", (long long)K);
    if (ldw < K || ldw % 8 != 0) return fail(ORBIT_EINVAL, "adaln_int4_quantize_weights: ldw=%lld must be >= K and a multiple of 8", (long long)ldw);
    // one thread per group of 64: the launch grid is 32-bit
    if (K > (int64_t)1 << 30 || N > INT32_MAX || N * (K / 64) > (int64_t)INT32_MAX * 256)
        return fail(ORBIT_EUNSUPPORTED, "adaln_int4_quantize_weights: N or K too large");
    if (N == 0) return ORBIT_OK;
    if (!W || !q || !scales) return fail(ORBIT_EINVAL, "adaln_int4_quantize_weights: null device pointer");
    if (!aligned(W, 16) || !aligned(q, 16) || !aligned(scales, 2))
        return fail(ORBIT_EINVAL, "adaln_int4_quantize_weights: misaligned pointer (W and q need 16 bytes)");
    int dev;
    DeviceInfo info;
    orbit_status st = current_device(&dev, &info);
    if (st != ORBIT_OK) return st;
    hipError_t e = launch_adaln_int4_quantize(W, N, (int)K, ldw, q, scales, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "adaln_int4_quantize_weights");
    return ORBIT_OK;
}

orbit_status adaln_int4_linear(const uint16_t* X, int64_t M, int64_t ldx, const uint8_t* q, const uint16_t* scales,
                               int64_t N, int64_t K, const uint16_t* bias, float* Y, int64_t ldy, void* stream) {
    clear_error();
    if (M < 0 || N < 0) return fail(ORBIT_EINVAL, "adaln_int4_linear: negative M or N");
    if (K <= 0 || K % 64 != 0) return fail(ORBIT_EINVAL, "adaln_int4_linear: K=%lld must be a positive multiple of 64", (long long)K);
    if (ldx < K || ldx % 8 != 0) return fail(ORBIT_EINVAL, "adaln_int4_linear: ldx=%lld must be >= K and a multiple of 8", (long long)ldx);
    if (ldy < N) return fail(ORBIT_EINVAL, "adaln_int4_linear: ldy=%lld < N=%lld", (long long)ldy, (long long)N);
    // the activations of two tokens are staged in LDS: K up to 16384
    if (K > 16384 || N > INT32_MAX || M > 65535 * 2)
        return fail(ORBIT_EUNSUPPORTED, "adaln_int4_linear: M=%lld, N=%lld or K=%lld too large", (long long)M,
                    (long long)N, (long long)K);
    if (M == 0 || N == 0) return ORBIT_OK;
    if (!X || !q || !scales || !Y) return fail(ORBIT_EINVAL, "adaln_int4_linear: null device pointer");
    if (!aligned(X, 16) || !aligned(q, 16) || !aligned(scales, 2) || !aligned(Y, 4) || (bias && !aligned(bias, 2)))
        return fail(ORBIT_EINVAL, "adaln_int4_linear: misaligned pointer (X and q need 16 bytes)");
    int dev;
    DeviceInfo info;
    orbit_status st = current_device(&dev, &info);
    if (st != ORBIT_OK) return st;
    RtnLinearParams r{};
    r.X = X;
    r.M = M;
    r.ldx = ldx;
    r.q = q;
    r.scales = scales;
    r.N = N;
    r.K = (int)K;
    r.bias = bias;
    r.Y = Y;
    r.ldy = ldy;
    hipError_t e = launch_adaln_int4_linear(r, info.cus, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "adaln_int4_linear");
    return ORBIT_OK;
}

orbit_status orbit_qlinear(orbit_codebook cb_a, const uint8_t* x_codes, const float* x_norm, int64_t M,
                           orbit_codebook cb_w, const uint8_t* w_codes, const uint16_t* w_norm, int64_t N, int64_t K,
                           float* Y, int64_t ldy, void* stream) {
    return orbit_qlinear_ex(cb_a, x_codes, x_norm, M, cb_w, w_codes, w_norm, N, K, nullptr, ORBIT_ACT_NONE,
                            ORBIT_OUT_F32, Y, ldy, stream);
}

orbit_status orbit_qlinear_ex(orbit_codebook cb_a, const uint8_t* x_codes, const float* x_norm, int64_t M,
                              orbit_codebook cb_w, const uint8_t* w_codes, const uint16_t* w_norm, int64_t N,
                              int64_t K, const uint16_t* bias, int32_t act, int32_t out_dtype, void* Y, int64_t ldy,
                              void* stream) {
    return orbit_qlinear_ws(cb_a, x_codes, x_norm, M, cb_w, w_codes, w_norm, N, K, bias, act, out_dtype, Y, ldy,
                            nullptr, 0, stream);
}

orbit_status orbit_qlinear_workspace_size(int64_t M, int64_t N, int64_t K, size_t* bytes) {
    clear_error();
    if (!bytes) return fail(ORBIT_EINVAL, "orbit_qlinear_workspace_size: null output pointer");
    *bytes = 0;
    if (M < 0 || N < 0) return fail(ORBIT_EINVAL, "orbit_qlinear_workspace_size: negative M or N");
    if (K <= 0 || K % 64 != 0 || K > (int64_t)1 << 30)
        return fail(ORBIT_EINVAL, "orbit_qlinear_workspace_size: K=%lld must be a positive multiple of 64", (long long)K);
    if (M == 0 || N == 0) return ORBIT_OK;
    int dev;
    DeviceInfo info;
    orbit_status st = current_device(&dev, &info);
    if (st != ORBIT_OK) return st;
    const int64_t m_small = M - lut_gemm_big_rows(M, N, info.cus);
    int steps = 0;
    const int splits = m_small > 0 ? lut_gemm_small_splits(m_small, N, K, info.cus, &steps) : 1;
    if (splits > 1) *bytes = (size_t)splits * (size_t)m_small * (size_t)N * sizeof(float);
    return ORBIT_OK;
}

orbit_status orbit_qlinear_schedule(int64_t M, int64_t N, int64_t K, int64_t* rows_large, int32_t* splits) {
    clear_error();
    if (!rows_large || !splits) return fail(ORBIT_EINVAL, "orbit_qlinear_schedule: null output pointer");
    *rows_large = 0;
    *splits = 1;
    if (M < 0 || N < 0) return fail(ORBIT_EINVAL, "orbit_qlinear_schedule: negative M or N");
    if (K <= 0 || K % 64 != 0 || K > (int64_t)1 << 30)
        return fail(ORBIT_EINVAL, "orbit_qlinear_schedule: K=%lld must be a positive multiple of 64", (long long)K);
    if (M == 0 || N == 0) return ORBIT_OK;
    int dev;
    DeviceInfo info;
    orbit_status st = current_device(&dev, &info);
    if (st != ORBIT_OK) return st;
    *rows_large = lut_gemm_big_rows(M, N, info.cus);
    const int64_t m_small = M - *rows_large;
    int steps = 0;
    *splits = m_small > 0 ? lut_gemm_small_splits(m_small, N, K, info.cus, &steps) : 1;
    return ORBIT_OK;
}

orbit_status orbit_qlinear_noalloc(orbit_codebook cb_a, const uint8_t* x_codes, const float* x_norm, int64_t M,
                                   orbit_codebook cb_w, const uint8_t* w_codes, const uint16_t* w_norm, int64_t N,
                                   int64_t K, const uint16_t* bias, int32_t act, int32_t out_dtype, void* Y,
                                   int64_t ldy, void* stream) {
    clear_error();
    // the split's partial sums must fit the scratch array; the other checks are orbit_qlinear_ws's
    size_t need = 0;
    if (M > 0 && N > 0 && K > 0 && K % 64 == 0 && K <= (int64_t)1 << 30) {
        orbit_status st = orbit_qlinear_workspace_size(M, N, K, &need);
        if (st != ORBIT_OK) return st;
        if (need > kScratchBytes)
            return fail(ORBIT_EUNSUPPORTED,
                        "orbit_qlinear_noalloc: a %lld x %lld x %lld layer splits over K into %zu bytes of partial sums, "
                        "above the %zu-byte scratch limit (use orbit_qlinear_ws with a workspace of that size)",
                        (long long)M, (long long)N, (long long)K, need, kScratchBytes);
    }
    void* ws = nullptr;
    if (need > 0) {
        int dev;
        DeviceInfo info;
        orbit_status st = current_device(&dev, &info);
        if (st != ORBIT_OK) return st;
        st = scratch_on(dev, &ws);
        if (st != ORBIT_OK) return st;
    }
    return orbit_qlinear_ws(cb_a, x_codes, x_norm, M, cb_w, w_codes, w_norm, N, K, bias, act, out_dtype, Y, ldy, ws,
                            ws ? kScratchBytes : 0, stream);
}

}  // extern "C"
