// Host side of the OrbitQuant library: error reporting, the RPBH plan generator and the
// Lloyd-Max codebook solver.  No HIP calls here; everything runs without a GPU.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>

#include "internal.h"

namespace orbit {

namespace {
thread_local std::string g_last_error;
}

orbit_status fail(orbit_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

void clear_error() { g_last_error.clear(); }

// ---------------------------------------------------------------------------------------------
// SplitMix64 (Steele, Lea & Flood, OOPSLA 2014): a Weyl sequence with golden-ratio increment
// passed through a 64-bit finalizer.  Output n is a function of (seed, n) only.
namespace {
struct SplitMix64 {
    uint64_t state;
    uint64_t next() {
        state += 0x9E3779B97F4A7C15ull;
        uint64_t z = state;
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        return z ^ (z >> 31);
    }
    // exactly uniform in [0, n): reject the first (2^64 mod n) values of the 64-bit range
    uint64_t below(uint64_t n) {
        const uint64_t t = (0 - n) % n;  // (2^64 - n) mod n == 2^64 mod n
        for (;;) {
            uint64_t u = next();
            if (u >= t) return u % n;
        }
    }
};
}  // namespace

// ---------------------------------------------------------------------------------------------
// Lloyd-Max on f_d(t) = C_d (1 - t^2)^((d-3)/2), t in [-1, 1]  (Sec. 3.2, Eq. (2)).
//
// Cell masses are integrated after t = sin(theta), where the integrand C_d cos^(d-2)(theta) is
// smooth, with composite 16-point Gauss-Legendre panels no wider than a quarter of the
// marginal's standard deviation.  First moments use the closed-form antiderivative
// -(1 - t^2)^((d-1)/2) / (d-1) of t (1 - t^2)^((d-3)/2).  By symmetry only the positive half
// line is solved (the fixed point is unique because f_d is log-concave, so it is symmetric);
// a few plain Lloyd steps are followed by Newton steps on  centroid(thresholds(p)) - p = 0
// with the exact tridiagonal Jacobian.
namespace {

constexpr int kGL = 16;
struct GaussLegendre {
    double x[kGL], w[kGL];
    GaussLegendre() {
        // roots of P_16 by Newton from Chebyshev-like starts; weights 2 / ((1-x^2) P'(x)^2)
        for (int i = 0; i < kGL; ++i) {
            double z = std::cos(M_PI * (i + 0.75) / (kGL + 0.5));
            double dp = 0.0;
            for (int it = 0; it < 100; ++it) {
                double p0 = 1.0, p1 = 0.0;
                for (int k = 1; k <= kGL; ++k) {
                    double p2 = p1;
                    p1 = p0;
                    p0 = ((2.0 * k - 1.0) * z * p1 - (k - 1.0) * p2) / k;
                }
                dp = kGL * (z * p0 - p1) / (z * z - 1.0);
                double dz = p0 / dp;
                z -= dz;
                if (std::fabs(dz) < 1e-17) break;
            }
            x[i] = z;
            w[i] = 2.0 / ((1.0 - z * z) * dp * dp);
        }
    }
};
const GaussLegendre& gl() {
    static const GaussLegendre g;
    return g;
}

struct Marginal {
    int64_t d;
    double log_c;      // log C_d
    double sd;         // 1/sqrt(d)
    double theta_max;  // |theta| beyond which the density is below exp(-800)

    explicit Marginal(int64_t d_) : d(d_) {
        long double dl = (long double)d_;
        log_c = (double)(lgammal(dl / 2.0L) - lgammal((dl - 1.0L) / 2.0L) - 0.5L * logl(3.141592653589793238462643383279503L));
        sd = 1.0 / std::sqrt((double)d_);
        theta_max = std::min(M_PI / 2.0, 40.0 / std::sqrt((double)std::max<int64_t>(d_ - 2, 1)));
    }
    double pdf(double t) const {
        if (std::fabs(t) >= 1.0) return (d == 3) ? 0.5 : 0.0;
        return std::exp(log_c + 0.5 * (double)(d - 3) * std::log1p(-t * t));
    }
    // P(a < t < b)
    double mass(double a, double b) const {
        double ta = std::asin(std::max(-1.0, std::min(1.0, a)));
        double tb = std::asin(std::max(-1.0, std::min(1.0, b)));
        ta = std::max(ta, -theta_max);
        tb = std::min(tb, theta_max);
        if (tb <= ta) return 0.0;
        const double width = 0.25 / std::sqrt((double)std::max<int64_t>(d - 2, 1));
        int panels = (int)std::ceil((tb - ta) / width);
        panels = std::max(1, std::min(panels, 1 << 16));
        const GaussLegendre& g = gl();
        // cos^(d-2)(theta) = exp((d-2)/2 * log1p(-sin^2 theta)): cos(theta) itself would be rounded
        // next to 1 and the error amplified d-fold in the exponent
        const double e = 0.5 * (double)(d - 2);
        double total = 0.0;
        for (int p = 0; p < panels; ++p) {
            double lo = ta + (tb - ta) * p / panels, hi = ta + (tb - ta) * (p + 1) / panels;
            double half = 0.5 * (hi - lo), mid = 0.5 * (hi + lo), s = 0.0;
            for (int i = 0; i < kGL; ++i) {
                const double sn = std::sin(mid + half * g.x[i]);
                const double q = sn * sn;
                s += g.w[i] * (q < 1.0 ? std::exp(log_c + e * std::log1p(-q)) : 0.0);
            }
            total += half * s;
        }
        return total;
    }
    // int_a^b t f_d(t) dt = C_d/(d-1) * [(1-a^2)^e - (1-b^2)^e], e = (d-1)/2, for |a| <= |b| written as
    // (1-b^2)^e * expm1(e * log1p((b-a)(b+a)/(1-b^2))) so that narrow cells lose no digits
    double moment(double a, double b) const {
        const double e = 0.5 * (double)(d - 1);
        const double sgn = (std::fabs(a) <= std::fabs(b)) ? 1.0 : -1.0;
        if (sgn < 0) std::swap(a, b);  // now |a| <= |b|; the integral changes sign
        const double qb = 1.0 - b * b;
        double diff;
        if (qb <= 0.0) {
            diff = std::exp(e * std::log1p(-a * a));
        } else {
            const double gb = std::exp(e * std::log1p(-b * b));
            diff = gb * std::expm1(e * std::log1p((b - a) * (b + a) / qb));
        }
        return sgn * std::exp(log_c) / (double)(d - 1) * diff;
    }
};

// Solve A x = r (dense, partial pivoting), n <= 32.
bool solve(std::vector<double>& A, std::vector<double>& r, int n) {
    for (int c = 0; c < n; ++c) {
        int piv = c;
        for (int i = c + 1; i < n; ++i)
            if (std::fabs(A[i * n + c]) > std::fabs(A[piv * n + c])) piv = i;
        if (A[piv * n + c] == 0.0) return false;
        if (piv != c) {
            for (int k = 0; k < n; ++k) std::swap(A[c * n + k], A[piv * n + k]);
            std::swap(r[c], r[piv]);
        }
        for (int i = c + 1; i < n; ++i) {
            double f = A[i * n + c] / A[c * n + c];
            for (int k = c; k < n; ++k) A[i * n + k] -= f * A[c * n + k];
            r[i] -= f * r[c];
        }
    }
    for (int i = n - 1; i >= 0; --i) {
        double s = r[i];
        for (int k = i + 1; k < n; ++k) s -= A[i * n + k] * r[k];
        r[i] = s / A[i * n + i];
    }
    return true;
}

// Positive-half levels p[0..m-1] of the 2m-level quantizer; cells [t_i, t_{i+1}] with t_0 = 0,
// t_i = (p_{i-1} + p_i)/2, t_m = 1.
struct HalfLine {
    const Marginal& f;
    int m;
    std::vector<double> edges(const std::vector<double>& p) const {
        std::vector<double> t(m + 1);
        t[0] = 0.0;
        for (int i = 1; i < m; ++i) t[i] = 0.5 * (p[i - 1] + p[i]);
        t[m] = 1.0;
        return t;
    }
    void centroids(const std::vector<double>& p, std::vector<double>& c, std::vector<double>& mass) const {
        std::vector<double> t = edges(p);
        for (int i = 0; i < m; ++i) {
            mass[i] = f.mass(t[i], t[i + 1]);
            c[i] = f.moment(t[i], t[i + 1]) / mass[i];
        }
    }
};

bool lloyd_max_positive_half(int64_t d, int bits, std::vector<double>& p_out) {
    Marginal f(d);
    const int m = 1 << (bits - 1);
    HalfLine H{f, m};
    std::vector<double> p(m), c(m), mass(m);
    const double spread = std::min(2.5 * f.sd, 0.8);
    for (int i = 0; i < m; ++i) p[i] = spread * (i + 0.5) / m;
    // plain Lloyd steps until the step is small
    for (int it = 0; it < 20000; ++it) {
        H.centroids(p, c, mass);
        double step = 0.0;
        for (int i = 0; i < m; ++i) step = std::max(step, std::fabs(c[i] - p[i]));
        p = c;
        if (step < 1e-7 * f.sd) break;
    }
    // Newton on G(p) = centroid(t(p)) - p
    for (int it = 0; it < 50; ++it) {
        H.centroids(p, c, mass);
        std::vector<double> t = H.edges(p);
        std::vector<double> A((size_t)m * m, 0.0), r(m);
        for (int i = 0; i < m; ++i) {
            r[i] = -(c[i] - p[i]);
            // dc_i/dt_{i+1} = f(t_{i+1}) (t_{i+1} - c_i) / mass_i ; dc_i/dt_i = f(t_i) (c_i - t_i) / mass_i
            double dhi = (i + 1 < m) ? f.pdf(t[i + 1]) * (t[i + 1] - c[i]) / mass[i] : 0.0;
            double dlo = (i > 0) ? f.pdf(t[i]) * (c[i] - t[i]) / mass[i] : 0.0;
            // t_{i+1} = (p_i + p_{i+1})/2 ; t_i = (p_{i-1} + p_i)/2
            if (i + 1 < m) {
                A[i * m + i] += 0.5 * dhi;
                A[i * m + i + 1] += 0.5 * dhi;
            }
            if (i > 0) {
                A[i * m + i - 1] += 0.5 * dlo;
                A[i * m + i] += 0.5 * dlo;
            }
            A[i * m + i] -= 1.0;
        }
        if (!solve(A, r, m)) return false;
        double step = 0.0;
        for (int i = 0; i < m; ++i) {
            p[i] += r[i];
            step = std::max(step, std::fabs(r[i]));
        }
        if (step < 1e-16 * f.sd) break;
    }
    // residual of the centroid condition
    H.centroids(p, c, mass);
    for (int i = 0; i < m; ++i) {
        if (!std::isfinite(p[i]) || std::fabs(c[i] - p[i]) > 1e-12 * f.sd) return false;
        if (i > 0 && !(p[i] > p[i - 1])) return false;
    }
    p_out = p;
    return true;
}

// BF16 bit pattern of an fp64 value, rounded once to 8 significant bits, ties to even (no double
// rounding through fp32).  Levels are finite and far inside the bf16 range.
uint16_t bf16_bits_rne(double v) {
    if (v == 0.0) return std::signbit(v) ? 0x8000u : 0u;
    int e;
    const double m = std::frexp(v, &e);                       // v = m 2^e, 0.5 <= |m| < 1
    const float r = (float)std::ldexp(std::nearbyint(std::ldexp(m, 8)), e - 8);  // exact in fp32
    uint32_t u;
    std::memcpy(&u, &r, 4);
    return (uint16_t)(u >> 16);
}

}  // namespace

void build_enc_table(orbit_codebook_s* c) {
    const std::vector<double>& tau = c->thresholds;
    double min_gap = 2.0 * kEncRange;
    for (size_t j = 1; j < tau.size(); ++j) min_gap = std::min(min_gap, tau[j] - tau[j - 1]);
    EncTable& e = c->enc;
    // u = 0 (an all-zero row, for one) lands on t = C exactly, in the middle of cell C, where the
    // middle threshold sits; biases of threshold cells are rounded up, so an exact tie there
    // resolves to the upper code as Eq. (3)'s reading here prescribes.
    const double w = 0.9 * min_gap;
    const int C = (int)std::ceil(kEncRange / w) + 1;
    const int ncell = 2 * C + 1;
    e.inv_w = (float)(1.0 / w);
    e.center = (float)C;
    e.ncell = ncell;
    e.bias.assign((size_t)ncell, 0.f);
    size_t j = 0;  // thresholds at or below the current cell start
    for (int cell = 0; cell < ncell; ++cell) {
        const double lo = (cell - 0.5 - C) * w, hi = (cell + 0.5 - C) * w;
        while (j < tau.size() && tau[j] <= lo) ++j;
        const double base = (double)j;
        if (j < tau.size() && tau[j] < hi) {
            const double b = base + 0.5 - 0.5 * (tau[j] / w);
            float bf = (float)b;
            if ((double)bf < b) bf = std::nextafter(bf, INFINITY);
            e.bias[cell] = bf;
        } else {
            e.bias[cell] = (float)(base - 0.5 * (cell - C));
        }
    }
}

}  // namespace orbit

using namespace orbit;

extern "C" {

const char* orbit_last_error(void) { return orbit::g_last_error.c_str(); }

const char* orbit_version(void) { return "orbitquant-mi355x 0.1.0 gfx950"; }

orbit_status rpbh_plan_from_arrays(int64_t d, int32_t h, const int32_t* perm, const int8_t* sign,
                                   orbit_plan* out) {
    clear_error();
    if (!out) return fail(ORBIT_EINVAL, "rpbh_plan: out is NULL");
    *out = nullptr;
    if (d < 1 || d > (int64_t)1 << 30) return fail(ORBIT_EINVAL, "rpbh_plan: d=%lld out of range", (long long)d);
    if (h == 0) h = (int32_t)std::min<int64_t>(d & -d, (int64_t)1 << 30);  // largest 2^p dividing d
    if (h < 1 || (h & (h - 1)) != 0 || d % h != 0)
        return fail(ORBIT_EINVAL, "rpbh_plan: h=%d must be a power of two dividing d=%lld", h, (long long)d);
    if (!perm || !sign) return fail(ORBIT_EINVAL, "rpbh_plan_from_arrays: perm/sign is NULL");
    orbit_plan p = new (std::nothrow) orbit_plan_s;
    if (!p) return fail(ORBIT_ENOMEM, "rpbh_plan: out of host memory");
    try {
        p->perm.assign(perm, perm + d);
        p->sign.assign(sign, sign + d);
    } catch (...) {
        delete p;
        return fail(ORBIT_ENOMEM, "rpbh_plan: out of host memory");
    }
    std::vector<char> seen((size_t)d, 0);
    for (int64_t j = 0; j < d; ++j) {
        int32_t v = p->perm[j];
        if (v < 0 || v >= d || seen[v]) {
            delete p;
            return fail(ORBIT_EINVAL, "rpbh_plan_from_arrays: perm is not a permutation (entry %lld)", (long long)j);
        }
        seen[v] = 1;
        if (p->sign[j] != 1 && p->sign[j] != -1) {
            delete p;
            return fail(ORBIT_EINVAL, "rpbh_plan_from_arrays: sign[%lld] = %d is not +-1", (long long)j, p->sign[j]);
        }
    }
    p->d = d;
    p->h = h;
    p->identity = true;
    for (int64_t j = 0; j < d && p->identity; ++j) p->identity = p->perm[j] == j;
    const orbit_status st = upload_on_create(p, nullptr);
    if (st != ORBIT_OK) {
        rpbh_plan_destroy(p);
        return st;
    }
    *out = p;
    return ORBIT_OK;
}

orbit_status rpbh_plan(int64_t d, int32_t h, uint64_t seed, orbit_plan* out) {
    clear_error();
    if (!out) return fail(ORBIT_EINVAL, "rpbh_plan: out is NULL");
    *out = nullptr;
    if (d < 1 || d > (int64_t)1 << 30) return fail(ORBIT_EINVAL, "rpbh_plan: d=%lld out of range", (long long)d);
    std::vector<int32_t> perm;
    std::vector<int8_t> sign;
    try {
        perm.resize(d);
        sign.resize(d);
    } catch (...) {
        return fail(ORBIT_ENOMEM, "rpbh_plan: out of host memory");
    }
    for (int64_t j = 0; j < d; ++j) perm[j] = (int32_t)j;
    SplitMix64 g{seed};
    for (int64_t j = d - 1; j >= 1; --j) {
        int64_t k = (int64_t)g.below((uint64_t)j + 1);
        std::swap(perm[j], perm[k]);
    }
    for (int64_t j = 0; j < d; ++j) sign[j] = (g.next() >> 63) ? -1 : 1;
    return rpbh_plan_from_arrays(d, h, perm.data(), sign.data(), out);
}

orbit_status rpbh_plan_get(orbit_plan p, int64_t* d, int32_t* h, int32_t* perm, int8_t* sign) {
    clear_error();
    if (!p) return fail(ORBIT_EINVAL, "rpbh_plan_get: plan is NULL");
    if (d) *d = p->d;
    if (h) *h = p->h;
    if (perm) std::memcpy(perm, p->perm.data(), sizeof(int32_t) * p->d);
    if (sign) std::memcpy(sign, p->sign.data(), p->d);
    return ORBIT_OK;
}

orbit_status lloydmax_codebook(int32_t bits, int64_t d, orbit_codebook* out) {
    clear_error();
    if (!out) return fail(ORBIT_EINVAL, "lloydmax_codebook: out is NULL");
    *out = nullptr;
    if (bits < 1 || bits > kMaxBits) return fail(ORBIT_EINVAL, "lloydmax_codebook: bits=%d outside 1..%d", bits, kMaxBits);
    if (d < 3 || d > (int64_t)1 << 30) return fail(ORBIT_EINVAL, "lloydmax_codebook: d=%lld outside 3..2^30", (long long)d);
    std::vector<double> half;
    if (!lloyd_max_positive_half(d, bits, half))
        return fail(ORBIT_EINTERNAL, "lloydmax_codebook: iteration did not converge (bits=%d, d=%lld)", bits, (long long)d);
    orbit_codebook c = new (std::nothrow) orbit_codebook_s;
    if (!c) return fail(ORBIT_ENOMEM, "lloydmax_codebook: out of host memory");
    const int n = 1 << bits, m = n / 2;
    c->bits = bits;
    c->d = d;
    c->levels.resize(n);
    for (int i = 0; i < m; ++i) {
        c->levels[m + i] = half[i];
        c->levels[m - 1 - i] = -half[i];
    }
    c->thresholds.resize(n - 1);
    for (int j = 0; j + 1 < n; ++j) c->thresholds[j] = 0.5 * (c->levels[j] + c->levels[j + 1]);
    build_enc_table(c);
    c->lut_bf16.resize(n);
    for (int j = 0; j < n; ++j) c->lut_bf16[j] = bf16_bits_rne(c->levels[j]);
    const orbit_status st = upload_on_create(nullptr, c);
    if (st != ORBIT_OK) {
        lloydmax_codebook_destroy(c);
        return st;
    }
    *out = c;
    return ORBIT_OK;
}

orbit_status lloydmax_codebook_get(orbit_codebook c, int32_t* bits, int64_t* d, double* levels, double* thresholds,
                                   uint16_t* lut_bf16) {
    clear_error();
    if (!c) return fail(ORBIT_EINVAL, "lloydmax_codebook_get: codebook is NULL");
    if (bits) *bits = c->bits;
    if (d) *d = c->d;
    const size_t n = c->levels.size();
    if (levels) std::memcpy(levels, c->levels.data(), n * sizeof(double));
    if (thresholds) std::memcpy(thresholds, c->thresholds.data(), (n - 1) * sizeof(double));
    if (lut_bf16) std::memcpy(lut_bf16, c->lut_bf16.data(), n * sizeof(uint16_t));
    return ORBIT_OK;
}

}  // extern "C"
