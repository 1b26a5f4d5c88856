// runtime.cpp -- host side of the C ABI declared in include/mi355fft.h.
//
// Plans validate the layout, pick the row or column kernel family, and share
// one device twiddle table per (device, N).  Execution is one stream-ordered
// kernel launch per call; nothing here synchronises.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <map>
#include <mutex>
#include <new>
#include <random>
#include <utility>
#include <vector>

#include "fft_launch.h"
#include "mi355fft.h"

using mi355fft::KArgs;

struct fft_plan {
    int64_t n, batch, stride, dist;
    int storage, dir, device, layout, xcd_remap, variant;
    float scale;  // output scale 2^-s (exact)
    // The split forms spread that scale over their passes so that no stored
    // intermediate grows past the final bound (FP16 storage): 2^-s1 in the
    // first pass, 2^-s2 in the middle pass of three, the rest in the last.
    // Powers of two are exact, so FP32 results are those of one final scale.
    float scale1, scale2, scale_last;
    int mfma;     // radix-16 butterflies on the matrix cores (FP16 storage)
    const void *amat;
    const float2 *tw;
    // four-step (n > 16384): n = n1 * n2; pass 1 runs n2 columns of length n1,
    // pass 2 n1 columns of length n2
    int64_t n1, n2;
    int log2s, v1, v2;
    const float2 *tw1, *tw2, *ftab;
    // three passes (n > 2^24): n2 = na * nb, pass 2 split into a pass of
    // na-point and a pass of nb-point columns (0: two passes)
    int64_t na, nb;
    int log2s2, va, vb;
    const float2 *twa, *twb, *ftab2;
    // long interleaved columns as two passes of short columns (out of place)
    bool colsplit;
};

namespace {

constexpr int64_t kMinN = 1024, kMaxN = 16384;      // single-pass transforms
constexpr int64_t kMaxFourStep = int64_t(1) << 28;  // longest transform
constexpr int64_t kMaxTwoPass = int64_t(1) << 22;   // two passes up to here, then three
constexpr int64_t kMaxIndex = int64_t(1) << 40;  // largest element index accepted

bool is_pow2(int64_t n) { return n > 0 && (n & (n - 1)) == 0; }
bool supported_n(int64_t n) { return is_pow2(n) && n >= kMinN && n <= kMaxN; }
int ilog2(int64_t n) {
    int l = 0;
    while ((int64_t(1) << (l + 1)) <= n) ++l;
    return l;
}

bool fail_alloc_hook() {
    const char *e = std::getenv("MI355FFT_TEST_FAIL_ALLOC");
    return e && e[0] == '1';
}

int map_hip(hipError_t e) {
    if (e == hipSuccess) return FFT_OK;
    if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation) return FFT_ENOMEM;
    return FFT_EHIP;
}

// Twiddle tables: exp(-2 pi i m / n), m in [0, n), computed in double with the
// angle 2 pi (m / n) (m / n is exact), rounded once to FP32.
std::mutex g_tw_mutex;
std::map<std::pair<int, int64_t>, float2 *> g_tw;

void host_twiddles(int64_t n, std::vector<float2> &host) {
    host.resize((size_t)mi355fft::twiddle_entries(n));
    const double two_pi = 6.283185307179586476925286766559;
    for (int64_t m = 0; m < n; ++m) {
        const double ang = two_pi * ((double)m / (double)n);
        host[(size_t)m] = make_float2((float)std::cos(ang), (float)-std::sin(ang));
    }
    // per-stage tables: W_(ns r)^(k j) at [(j - 1) ns + k], the angle reduced
    // exactly (k j mod ns r) before it is scaled
    for (int r : mi355fft::kStageRadices) {
        for (int64_t ns = 2; ns <= n / r; ns *= 2) {
            const int64_t base = mi355fft::stage_table_offset(n, (int)ns, r), len = ns * r;
            for (int j = 1; j < r; ++j)
                for (int64_t k = 0; k < ns; ++k) {
                    const double ang = two_pi * ((double)((k * j) % len) / (double)len);
                    host[(size_t)(base + (j - 1) * ns + k)] = make_float2((float)std::cos(ang), (float)-std::sin(ang));
                }
        }
    }
}

int get_twiddles(int device, int64_t n, const float2 **out) {
    std::lock_guard<std::mutex> lock(g_tw_mutex);
    auto it = g_tw.find({device, n});
    if (it != g_tw.end()) {
        *out = it->second;
        return FFT_OK;
    }
    if (fail_alloc_hook()) return FFT_ENOMEM;
    std::vector<float2> host;
    host_twiddles(n, host);
    float2 *dev = nullptr;
    hipError_t e = hipMalloc((void **)&dev, sizeof(float2) * host.size());
    if (e != hipSuccess) return map_hip(e);
    e = hipMemcpy(dev, host.data(), sizeof(float2) * host.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(dev);
        return map_hip(e);
    }
    g_tw[{device, n}] = dev;
    *out = dev;
    return FFT_OK;
}

// The migration-correction interpolator (Section X): an 8-tap sinc under a
// Kaiser window (beta 2.5) spanning the 8 taps, at the 129 fractional shifts
// mu = q / 128, each row normalised to unit sum, stored as FP32 pairs
// {g_q[j], g_{q+1}[j] - g_q[j]} for linear blending between rows (Section X's
// third fix).  Tap j sits at offset j - 3 from the integer part of the
// position.  Computed in double once per device.
std::mutex g_interp_mutex;
std::map<int, float2 *> g_interp;

double bessel_i0(double x) {  // sum_m ((x/2)^m / m!)^2
    double term = 1.0, sum = 1.0;
    const double h = 0.25 * x * x;
    for (int m = 1; m < 200 && term >= 1e-18 * sum; ++m) {
        term *= h / ((double)m * (double)m);
        sum += term;
    }
    return sum;
}

void interp_row(int q, double *g) {
    using mi355fft::kRcmcSub;
    using mi355fft::kRcmcTaps;
    const double pi = 3.141592653589793238462643383279, beta = 2.5;
    const double mu = (double)q / kRcmcSub, inv_i0 = 1.0 / bessel_i0(beta);
    double sum = 0.0;
    for (int j = 0; j < kRcmcTaps; ++j) {
        const double x = (double)(j - 3) - mu;
        const double sinc = x == 0.0 ? 1.0 : std::sin(pi * x) / (pi * x);
        const double r = 0.25 * x, arg = 1.0 - r * r;
        g[j] = sinc * bessel_i0(beta * std::sqrt(arg > 0.0 ? arg : 0.0)) * inv_i0;
        sum += g[j];
    }
    for (int j = 0; j < kRcmcTaps; ++j) g[j] /= sum;
}

int get_interp(int device, const float2 **out) {
    using mi355fft::kRcmcSub;
    using mi355fft::kRcmcTaps;
    std::lock_guard<std::mutex> lock(g_interp_mutex);
    auto it = g_interp.find(device);
    if (it != g_interp.end()) {
        *out = it->second;
        return FFT_OK;
    }
    std::vector<float2> host((size_t)(kRcmcSub + 1) * kRcmcTaps);
    double g[kRcmcTaps], g1[kRcmcTaps];
    for (int q = 0; q <= kRcmcSub; ++q) {
        interp_row(q, g);
        if (q < kRcmcSub) interp_row(q + 1, g1);
        for (int j = 0; j < kRcmcTaps; ++j) {
            const float lo = (float)g[j];
            host[(size_t)(q * kRcmcTaps + j)] = make_float2(lo, q < kRcmcSub ? (float)(g1[j] - (double)lo) : 0.0f);
        }
    }
    float2 *dev = nullptr;
    hipError_t e = hipMalloc((void **)&dev, sizeof(float2) * host.size());
    if (e != hipSuccess) return map_hip(e);
    e = hipMemcpy(dev, host.data(), sizeof(float2) * host.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(dev);
        return map_hip(e);
    }
    g_interp[device] = dev;
    *out = dev;
    return FFT_OK;
}

// Four-step twiddles W_N^m = exp(-2 pi i m / N), m < N, as two tables of
// about sqrt(N) entries: lo[m] = W_N^m for m < S, hi[m] = W_N^(S m) for
// m < N / S (S = 2^ceil(log2(N) / 2)), each computed in double with the
// angle 2 pi (m / N) and rounded once; W_N^m = lo[m mod S] * hi[m div S].
std::mutex g_ftab_mutex;
std::map<std::pair<int, int64_t>, float2 *> g_ftab;

void host_fourstep_table(int64_t n, int log2s, std::vector<float2> &host) {
    const int64_t s = int64_t(1) << log2s, h = n / s;
    host.resize((size_t)(s + h));
    const double two_pi = 6.283185307179586476925286766559;
    for (int64_t m = 0; m < s; ++m) {
        const double ang = two_pi * ((double)m / (double)n);
        host[(size_t)m] = make_float2((float)std::cos(ang), (float)-std::sin(ang));
    }
    for (int64_t m = 0; m < h; ++m) {
        const double ang = two_pi * ((double)(m * s) / (double)n);
        host[(size_t)(s + m)] = make_float2((float)std::cos(ang), (float)-std::sin(ang));
    }
}

int get_fourstep_table(int device, int64_t n, int log2s, const float2 **out) {
    std::lock_guard<std::mutex> lock(g_ftab_mutex);
    auto it = g_ftab.find({device, n});
    if (it != g_ftab.end()) {
        *out = it->second;
        return FFT_OK;
    }
    std::vector<float2> host;
    host_fourstep_table(n, log2s, host);
    float2 *dev = nullptr;
    hipError_t e = hipMalloc((void **)&dev, sizeof(float2) * host.size());
    if (e != hipSuccess) return map_hip(e);
    e = hipMemcpy(dev, host.data(), sizeof(float2) * host.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(dev);
        return map_hip(e);
    }
    g_ftab[{device, n}] = dev;
    *out = dev;
    return FFT_OK;
}

// Lane fragments of the real 32 x 32 matrix of the 16-point DFT for the
// matrix-core kernels, both directions, split into binary16 hi + lo parts
// (computed in double once per device; layout in fft_mfma.hpp).
std::mutex g_amat_mutex;
std::map<int, void *> g_amat;

int get_dft16_matrix(int device, const void **out) {
    std::lock_guard<std::mutex> lock(g_amat_mutex);
    auto it = g_amat.find(device);
    if (it != g_amat.end()) {
        *out = it->second;
        return FFT_OK;
    }
    std::vector<_Float16> host(2 * 64 * 2 * 2 * 8);
    const double two_pi = 6.283185307179586476925286766559;
    for (int d = 0; d < 2; ++d)
        for (int l = 0; l < 64; ++l)
            for (int s = 0; s < 2; ++s)
                for (int e = 0; e < 8; ++e) {
                    const int m = l % 32, kp = m >> 1, co = m & 1;
                    const int k = 16 * s + 8 * (l / 32) + e, r = k >> 1, ci = k & 1;
                    const double th = two_pi * (double)((kp * r) % 16) / 16.0;
                    const double c = std::cos(th), sn = d ? -std::sin(th) : std::sin(th);
                    const double f = co == 0 ? (ci == 0 ? c : sn) : (ci == 0 ? -sn : c);
                    const _Float16 hi = (_Float16)f;
                    const size_t base = (size_t)((((d * 64 + l) * 2 + s) * 2) * 8 + e);
                    host[base] = hi;
                    host[base + 8] = (_Float16)(f - (double)hi);
                }
    void *dev = nullptr;
    hipError_t e = hipMalloc(&dev, sizeof(_Float16) * host.size());
    if (e != hipSuccess) return map_hip(e);
    e = hipMemcpy(dev, host.data(), sizeof(_Float16) * host.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(dev);
        return map_hip(e);
    }
    g_amat[device] = dev;
    *out = dev;
    return FFT_OK;
}

hipError_t launch_fft(int64_t n, int variant, int layout, int in_st, int out_st, int inv, int epi, const void *in,
                      void *out, const float2 *tw, const float2 *spec, const KArgs &a, hipStream_t s) {
    using namespace mi355fft;
    switch (n) {
        case 64: return launch_fft_n64(variant, layout, in_st, out_st, inv, epi, in, out, tw, spec, a, s);
        case 128: return launch_fft_n128(variant, layout, in_st, out_st, inv, epi, in, out, tw, spec, a, s);
        case 256: return launch_fft_n256(variant, layout, in_st, out_st, inv, epi, in, out, tw, spec, a, s);
        case 512: return launch_fft_n512(variant, layout, in_st, out_st, inv, epi, in, out, tw, spec, a, s);
        case 1024: return launch_fft_n1024(variant, layout, in_st, out_st, inv, epi, in, out, tw, spec, a, s);
        case 2048: return launch_fft_n2048(variant, layout, in_st, out_st, inv, epi, in, out, tw, spec, a, s);
        case 4096: return launch_fft_n4096(variant, layout, in_st, out_st, inv, epi, in, out, tw, spec, a, s);
        case 8192: return launch_fft_n8192(variant, layout, in_st, out_st, inv, epi, in, out, tw, spec, a, s);
        case 16384: return launch_fft_n16384(variant, layout, in_st, out_st, inv, epi, in, out, tw, spec, a, s);
        default: return hipErrorInvalidValue;
    }
}

int variant_count(int64_t n, int layout) {
    using namespace mi355fft;
    switch (n) {
        case 64: return variants_n64(layout);
        case 128: return variants_n128(layout);
        case 256: return variants_n256(layout);
        case 512: return variants_n512(layout);
        case 1024: return variants_n1024(layout);
        case 2048: return variants_n2048(layout);
        case 4096: return variants_n4096(layout);
        case 8192: return variants_n8192(layout);
        case 16384: return variants_n16384(layout);
        default: return 0;
    }
}

// Kernel-shape override for tests and tuning: MI355FFT_ROW_VARIANT /
// MI355FFT_COL_VARIANT / MI355FFT_RCMC_VARIANT = index into the size's list of
// row, column or migration-correction kernels (unset: default).
// Returns -1 for the default, -2 for an index the size does not have.
int chosen_variant(int64_t n, int layout) {
    const char *e = std::getenv(layout == mi355fft::LAYOUT_ROWS   ? "MI355FFT_ROW_VARIANT"
                                : layout == mi355fft::LAYOUT_COLS ? "MI355FFT_COL_VARIANT"
                                : layout == mi355fft::LAYOUT_RCMC ? "MI355FFT_RCMC_VARIANT"
                                                                  : "MI355FFT_HALF_VARIANT");
    if (!e || !e[0]) return -1;
    char *end = nullptr;
    long v = std::strtol(e, &end, 10);
    if (*end != '\0' || v < 0 || v >= variant_count(n, layout)) return -2;
    return (int)v;
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Block -> strip map for column strips whose rows are row_bytes apart: the
// line groups spread over the XCDs for rows of 32 KiB and more, contiguous
// ranges per XCD for shorter rows (measured on MI355X, see logical_block).
int strip_map(int64_t row_bytes) { return row_bytes >= 32768 ? mi355fft::XCD_GROUPS : mi355fft::XCD_CONTIG; }

// Largest batch of n-point transforms (4096 <= n <= 16384) run in the two-pass
// split form when out of place.  Measured on MI355X (event time of one call):
// at n = 16384 the split takes 15-17 us for 1-16 transforms against 17.6-18 us
// in one pass; at 4096 and 8192 one pass is always faster.  The tuning knob
// MI355FFT_SPLIT_BATCH overrides the limit for every n; a forced row shape
// (MI355FFT_ROW_VARIANT) turns the split off.
int64_t split_batch(int64_t n) {
    const char *rv = std::getenv("MI355FFT_ROW_VARIANT");
    if (rv && rv[0]) return 0;
    const char *e = std::getenv("MI355FFT_SPLIT_BATCH");
    if (!e || !e[0]) return n == 16384 ? 16 : 0;
    char *end = nullptr;
    const long long v = std::strtoll(e, &end, 10);
    return (*end == '\0' && v > 0) ? v : 0;
}

// Long strided columns (8192 or 16384 points, interleaved: dist 1) executed
// out of place run as two passes of short columns: a 8192- or 16384-point
// column kernel holds one or two columns per workgroup, so it reads 8- or
// 16-byte pieces of each row, while 64- and 128-point column kernels hold
// 32-64 columns.  A forced column shape (MI355FFT_COL_VARIANT) keeps the
// single pass.
bool column_split(int64_t n, int64_t stride, int64_t dist) {
    const char *cv = std::getenv("MI355FFT_COL_VARIANT");
    if (cv && cv[0]) return false;
    return stride > 1 && dist == 1 && (n == 8192 || n == 16384);
}

bool overlaps(const void *a, size_t na, const void *b, size_t nb) {
    const char *pa = (const char *)a, *pb = (const char *)b;
    return pa < pb + nb && pb < pa + na;
}

// Full range-Doppler chain: the migration-correction pass addresses the whole
// intermediate image through one 31-bit buffer offset, so n_az * n_rg * 8
// bytes must stay below 2 GiB.
constexpr int64_t kMaxRdPoints = int64_t(1) << 27;
constexpr double kMaxDopplerRatio = 1.0 / 3.0;  // 15 (1 / sqrt(1 - 1/9) - 1) = 0.91

// Workspace of sar_rd_form_image: range reference spectrum, tables, image.
// Every chain workspace holds one 256-byte slot for the flag with which the
// range pass's workgroup 0 publishes the range reference spectrum.
constexpr size_t kChainFlagBytes = 256;

// A fresh value per chain call for that flag: 64 bits from a per-process
// random start, never 0 (the value the pass after the range pass leaves), so
// neither a stale flag of an earlier call nor uninitialised workspace memory
// reads as this call's.
unsigned long long next_chain_epoch() {
    static std::atomic<unsigned long long> counter{[] {
        unsigned long long r = 0;
        try {  // no exception may leave the C ABI: without an entropy source, the clock alone
            std::random_device rd;
            r = ((unsigned long long)rd() << 32) ^ (unsigned long long)rd();
        } catch (...) {
        }
        const unsigned long long t = (unsigned long long)std::chrono::steady_clock::now().time_since_epoch().count();
        const unsigned long long here = (unsigned long long)(uintptr_t)&r;  // address-space randomisation
        return r ^ (t * 0x9E3779B97F4A7C15ull) ^ (here << 17);
    }()};
    unsigned long long e = counter.fetch_add(1, std::memory_order_relaxed);
    if (e == 0) e = counter.fetch_add(1, std::memory_order_relaxed);
    return e;
}

// range-Doppler workspace: H_r, the flag slot, the migration tables, the
// transposed range-Doppler image
size_t rd_flag_offset(int64_t n_rg) { return (size_t)n_rg * sizeof(float2); }
size_t rd_tables_offset(int64_t n_rg) { return rd_flag_offset(n_rg) + kChainFlagBytes; }  // n_rg >= 1024: 256-aligned
size_t rd_mid_offset(int64_t n_az, int64_t n_rg) {
    return rd_tables_offset(n_rg) + (size_t)mi355fft::rd_tables_layout(n_az, n_rg).bytes;
}

// The library-owned workspace of the fixed-size sar_form_image, per device.
std::mutex g_ws_mutex;
std::map<int, void *> g_ws;

}  // namespace

// Every entry point that allocates host memory is a function-try-block: no
// C++ exception leaves the C ABI (std::bad_alloc -> FFT_ENOMEM, anything
// else -> FFT_EHIP).
extern "C" {

int fft_plan_create(int64_t n, int64_t batch, int64_t stride, int64_t dist, int storage, int dir,
                    fft_plan **plan_out) try {
    return fft_plan_create_ex(n, batch, stride, dist, storage, dir, 0, 0u, plan_out);
} catch (const std::bad_alloc &) {
    return FFT_ENOMEM;
} catch (...) {
    return FFT_EHIP;
}

int fft_plan_create_ex(int64_t n, int64_t batch, int64_t stride, int64_t dist, int storage, int dir,
                       int scale_log2, unsigned flags, fft_plan **plan_out) try {
    if (!plan_out) return FFT_EINVAL;
    if (storage != FFT_STORAGE_FP32 && storage != FFT_STORAGE_FP16) return FFT_EINVAL;
    if (dir != FFT_FORWARD && dir != FFT_INVERSE) return FFT_EINVAL;
    if (n < 1 || batch < 1 || stride < 1 || dist < 1) return FFT_EINVAL;
    if (scale_log2 < 0 || scale_log2 > 60) return FFT_EINVAL;
    if (flags & ~(unsigned)(FFT_FLAG_FP16_EXCHANGE | FFT_FLAG_MATRIX_UNITS)) return FFT_EINVAL;
    const bool half_x = (flags & FFT_FLAG_FP16_EXCHANGE) != 0;
    const bool mfma = (flags & FFT_FLAG_MATRIX_UNITS) != 0;
    if ((half_x || mfma) && storage != FFT_STORAGE_FP16) return FFT_EINVAL;
    if (half_x && mfma) return FFT_EINVAL;
    if (mfma && (stride != 1 || (n != 4096 && n != 16384))) return FFT_EUNSUPPORTED;
    if (mfma && scale_log2 != 0) return FFT_EUNSUPPORTED;
    // Transforms longer than 16384 take the four-step form.  A short batch of
    // 4096..16384-point transforms may take it too when run out of place
    // (Section VI: split one transform over several workgroups when the batch
    // is too small to fill the device): at most split_batch() transforms.
    const bool four_step = is_pow2(n) && n > kMaxN && n <= kMaxFourStep;
    const bool may_split =
        !half_x && !mfma && is_pow2(n) && n >= 4096 && n <= kMaxN && stride == 1 && batch <= split_batch(n);
    if (half_x && (four_step || stride != 1)) return FFT_EUNSUPPORTED;  // single-pass rows only
    if (!supported_n(n) && !four_step) return FFT_EUNSUPPORTED;
    if (four_step && stride != 1) return FFT_EUNSUPPORTED;  // long transforms: contiguous only
    // extent of the layout must be addressable
    if (batch - 1 > kMaxIndex / dist || n - 1 > kMaxIndex / stride ||
        (batch - 1) * dist > kMaxIndex - (n - 1) * stride)
        return FFT_EINVAL;
    // transforms must not overlap: disjoint blocks or interleaved
    const bool blocks = batch == 1 || dist >= (n - 1) * stride + 1;
    const bool interleaved = stride >= (batch - 1) * dist + 1;
    if (!blocks && !interleaved) return FFT_EINVAL;
    if (batch > (int64_t)0x7fffffff) return FFT_EUNSUPPORTED;  // grid size limit
    const int layout = half_x ? mi355fft::LAYOUT_ROWS_HALF
                              : stride == 1 ? mi355fft::LAYOUT_ROWS : mi355fft::LAYOUT_COLS;
    // four-step split: n2 = 2^floor(log2 n / 2), n1 = n / n2 (both in [128, 2048]).
    // Beyond 2^22 a two-factor split needs columns of 4096 points or more,
    // whose strips are 8 columns or fewer wide (64-, 16- or 8-byte pieces of
    // each row); three passes of at most 1024-point columns move the data
    // once more but faster: n1 = 2^floor(log2 n / 3) and n2 = n / n1 =
    // na * nb, na = 2^floor(log2 n2 / 2).  Measured on MI355X (1 GiB,
    // 16 B/pt): 2^23 1.74 against 1.59 TB/s, 2^24 1.81 against 1.69,
    // 2^28 1.25 against 0.47; at 2^20-2^22 two passes stay ahead.
    const bool colsplit = !half_x && !mfma && column_split(n, stride, dist);
    const bool split = four_step || may_split || colsplit;
    const bool three = four_step && n > kMaxTwoPass;
    // long columns: n1 = 128, n2 = 64 or 128
    const int64_t n2 = !split ? 0 : three ? n >> (ilog2(n) / 3) : colsplit ? n / 128 : int64_t(1) << (ilog2(n) / 2);
    const int64_t n1 = split ? n / n2 : 0;
    const int64_t na = three ? int64_t(1) << (ilog2(n2) / 2) : 0, nb = three ? n2 / na : 0;
    const int variant = four_step ? -1 : chosen_variant(n, layout);
    const int v1 = split ? chosen_variant(n1, mi355fft::LAYOUT_COLS) : -1;
    const int v2 = split && !three ? chosen_variant(n2, mi355fft::LAYOUT_COLS) : -1;
    const int va = three ? chosen_variant(na, mi355fft::LAYOUT_COLS) : -1;
    const int vb = three ? chosen_variant(nb, mi355fft::LAYOUT_COLS) : -1;
    if (variant == -2 || v1 == -2 || v2 == -2 || va == -2 || vb == -2) return FFT_EINVAL;
    if (four_step && batch > (int64_t)0x7fffffff) return FFT_EUNSUPPORTED;
    if (fail_alloc_hook()) return FFT_ENOMEM;  // test hook: device allocation fails

    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return map_hip(e);
    const float2 *tw = nullptr, *tw1 = nullptr, *tw2 = nullptr, *ftab = nullptr;
    const float2 *twa = nullptr, *twb = nullptr, *ftab2 = nullptr;
    const int log2s = split ? (ilog2(n) + 1) / 2 : 0;
    const int log2s2 = three ? (ilog2(n2) + 1) / 2 : 0;
    int rc = FFT_OK;
    if (split) {
        rc = get_twiddles(device, n1, &tw1);
        if (rc == FFT_OK && !three) rc = get_twiddles(device, n2, &tw2);
        if (rc == FFT_OK) rc = get_fourstep_table(device, n, log2s, &ftab);
    }
    if (three) {
        if (rc == FFT_OK) rc = get_twiddles(device, na, &twa);
        if (rc == FFT_OK) rc = get_twiddles(device, nb, &twb);
        if (rc == FFT_OK) rc = get_fourstep_table(device, n2, log2s2, &ftab2);
    }
    if (rc == FFT_OK && !four_step) rc = get_twiddles(device, n, &tw);
    const void *amat = nullptr;
    if (rc == FFT_OK && mfma) rc = get_dft16_matrix(device, &amat);
    if (rc != FFT_OK) return rc;
    fft_plan *p = new (std::nothrow) fft_plan;
    if (!p) return FFT_ENOMEM;
    p->scale = std::ldexp(1.0f, -scale_log2);
    {
        const int s1 = split ? std::min(scale_log2, ilog2(n1)) : 0;
        const int s2 = three ? std::min(scale_log2 - s1, ilog2(na)) : 0;
        p->scale1 = std::ldexp(1.0f, -s1);
        p->scale2 = std::ldexp(1.0f, -s2);
        p->scale_last = std::ldexp(1.0f, -(scale_log2 - s1 - s2));
    }
    p->mfma = mfma;
    p->amat = amat;
    p->n1 = n1;
    p->n2 = n2;
    p->log2s = log2s;
    p->v1 = v1;
    p->v2 = v2;
    p->tw1 = tw1;
    p->tw2 = tw2;
    p->ftab = ftab;
    p->colsplit = colsplit;
    p->na = na;
    p->nb = nb;
    p->log2s2 = log2s2;
    p->va = va;
    p->vb = vb;
    p->twa = twa;
    p->twb = twb;
    p->ftab2 = ftab2;
    p->n = n;
    p->batch = batch;
    p->stride = stride;
    p->dist = dist;
    p->storage = storage;
    p->dir = dir;
    p->device = device;
    p->layout = layout;
    p->variant = variant;
    // columns: strips of a line on one XCD; rows: about 1 MiB of consecutive
    // transforms per XCD at a time (logical_block)
    p->xcd_remap = layout == mi355fft::LAYOUT_COLS && dist == 1
                       ? strip_map(stride * (storage == FFT_STORAGE_FP32 ? 8 : 4))
                   : layout == mi355fft::LAYOUT_ROWS || layout == mi355fft::LAYOUT_ROWS_HALF ? mi355fft::XCD_ROWS
                                                     : mi355fft::XCD_NONE;
    p->tw = tw;
    *plan_out = p;
    return FFT_OK;
} catch (const std::bad_alloc &) {
    return FFT_ENOMEM;
} catch (...) {
    return FFT_EHIP;
}

// Three passes for n = n1 * na * nb (x viewed as n1 x n2, n2 = na * nb, j =
// n2 j1 + j2, j2 = nb ja + jb):
//   pass 1  the n2 columns of length n1, times W_n^(j2 k1), column j2 written
//           as row na (j2 mod nb) + (j2 div nb) of `out`: each problem's nb
//           groups of na rows then sit together;
//   pass 2  in place, for each jb, the n1 columns of length na of its group
//           of rows, output ka times W_n2^(jb ka);
//   pass 3  in place, for each ka, the n1 columns of length nb through rows
//           ka, ka + na, ... : row ka + na kb then holds X[k1 + n1 (ka + na kb)],
//           the natural order.
static int execute_three_pass(const fft_plan *plan, const void *in, void *out, int inv, hipStream_t stream) {
    const size_t el = plan->storage == FFT_STORAGE_FP32 ? 8 : 4;
    const int64_t n1 = plan->n1, n2 = plan->n2, na = plan->na, nb = plan->nb;
    for (int64_t b0 = 0; b0 < plan->batch; b0 += 65535) {
        const int64_t nbat = plan->batch - b0 < 65535 ? plan->batch - b0 : 65535;
        const char *pin = (const char *)in + (size_t)(b0 * plan->dist) * el;
        char *pout = (char *)out + (size_t)(b0 * plan->dist) * el;
        KArgs a1{n2, n2, 1, n1, plan->scale1, strip_map(n2 * (int64_t)el)};
        a1.out_stride = 1;
        a1.outer = (int)nbat;
        a1.outer_in_dist = a1.outer_out_dist = plan->dist;
        a1.aux = plan->log2s;
        a1.perm_a = ilog2(na);
        a1.perm_b = ilog2(nb);
        hipError_t e = launch_fft(n1, plan->v1, mi355fft::LAYOUT_COLS, plan->storage, plan->storage, inv,
                                  mi355fft::EPI_TWIDDLE, pin, pout, plan->tw1, plan->ftab, a1, stream);
        if (e != hipSuccess) return map_hip(e);
    }
    // passes 2 and 3 use the grid's second axis for the groups and its third
    // for the problems (at most 65535 per launch)
    for (int64_t b0 = 0; b0 < plan->batch; b0 += 65535) {
        const int64_t nbat = plan->batch - b0 < 65535 ? plan->batch - b0 : 65535;
        char *p = (char *)out + (size_t)(b0 * plan->dist) * el;
        KArgs a2{n1, n1, 1, 1, plan->scale2, strip_map(n1 * (int64_t)el)};
        a2.outer = (int)nb;
        a2.outer_in_dist = a2.outer_out_dist = na * n1;
        a2.outer2 = (int)nbat;
        a2.outer2_dist = plan->dist;
        a2.aux = plan->log2s2;
        hipError_t e = launch_fft(na, plan->va, mi355fft::LAYOUT_COLS, plan->storage, plan->storage, inv,
                                  mi355fft::EPI_TWIDDLE_Y, p, p, plan->twa, plan->ftab2, a2, stream);
        if (e != hipSuccess) return map_hip(e);
        KArgs a3{n1, na * n1, 1, 1, plan->scale_last, strip_map(na * n1 * (int64_t)el)};
        a3.outer = (int)na;
        a3.outer_in_dist = a3.outer_out_dist = n1;
        a3.outer2 = (int)nbat;
        a3.outer2_dist = plan->dist;
        e = launch_fft(nb, plan->vb, mi355fft::LAYOUT_COLS, plan->storage, plan->storage, inv, mi355fft::EPI_NONE,
                       p, p, plan->twb, nullptr, a3, stream);
        if (e != hipSuccess) return map_hip(e);
    }
    return FFT_OK;
}

// Columns of length n = n1 * n2 (point j of column c at j S + c, S the
// stride), j = n2 j1 + j2:
//   pass 1  for each j2 (the grid's second axis), the columns of length n1
//           through rows n2 j1 + j2, output k1 times W_n^(j2 k1), written to
//           rows j2 n1 + k1 of `out`;
//   pass 2  in place, for each k1, the columns of length n2 through rows
//           j2 n1 + k1: row k1 + n1 k2 then holds X[k1 + n1 k2].
static int execute_column_split(const fft_plan *plan, const void *in, void *out, int inv, hipStream_t stream) {
    const int64_t n1 = plan->n1, n2 = plan->n2, s = plan->stride;
    const size_t el = plan->storage == FFT_STORAGE_FP32 ? 8 : 4;
    KArgs a1{plan->batch, n2 * s, 1, 1, plan->scale1, strip_map(n2 * s * (int64_t)el)};
    a1.out_stride = s;
    a1.outer = (int)n2;
    a1.outer_in_dist = s;
    a1.outer_out_dist = n1 * s;
    a1.aux = plan->log2s;
    hipError_t e = launch_fft(n1, plan->v1, mi355fft::LAYOUT_COLS, plan->storage, plan->storage, inv,
                              mi355fft::EPI_TWIDDLE_Y, in, out, plan->tw1, plan->ftab, a1, stream);
    if (e != hipSuccess) return map_hip(e);
    KArgs a2{plan->batch, n1 * s, 1, 1, plan->scale_last, strip_map(n1 * s * (int64_t)el)};
    a2.outer = (int)n1;
    a2.outer_in_dist = a2.outer_out_dist = s;
    e = launch_fft(n2, plan->v2, mi355fft::LAYOUT_COLS, plan->storage, plan->storage, inv, mi355fft::EPI_NONE, out,
                   out, plan->tw2, nullptr, a2, stream);
    return map_hip(e);
}

int fft_execute(const fft_plan *plan, const void *in, void *out, hipStream_t stream) try {
    if (!plan || !in || !out) return FFT_EINVAL;
    const size_t el = plan->storage == FFT_STORAGE_FP32 ? 8 : 4;
    if (!aligned(in, el) || !aligned(out, el)) return FFT_EALIGN;
    // in place, or two disjoint extents (the plan bounded the extent by 2^40 elements)
    const size_t extent = (size_t)((plan->batch - 1) * plan->dist + (plan->n - 1) * plan->stride + 1) * el;
    if (in != out && overlaps(in, extent, out, extent)) return FFT_EINVAL;
    // the plan's tables live on the device it was created on
    int device = 0;
    const hipError_t de = hipGetDevice(&device);
    if (de != hipSuccess) return map_hip(de);
    if (device != plan->device) return FFT_EINVAL;
    if (plan->colsplit && in != out) return execute_column_split(plan, in, out, plan->dir == FFT_INVERSE, stream);
    if (plan->n1 && !plan->colsplit && (plan->n > kMaxN || in != out)) {
        // four-step (Section VI's two-pass transform for lengths beyond the
        // chip): pass 1 transforms the n2 columns of length n1 of each
        // problem viewed as an n1 x n2 matrix, multiplies point k1 of column
        // n2 by W_N^(n2 k1) and writes the columns as rows of `out`; pass 2
        // transforms, in place, the n1 columns of length n2 of that n2 x n1
        // matrix, which leaves X[k1 + n1 k2] in natural order.
        if (in == out) return FFT_EINVAL;
        const int inv = plan->dir == FFT_INVERSE;
        const int64_t n1 = plan->n1, n2 = plan->n2;
        if (plan->na) return execute_three_pass(plan, in, out, inv, stream);
        for (int64_t b0 = 0; b0 < plan->batch; b0 += 65535) {
            const int64_t nb = plan->batch - b0 < 65535 ? plan->batch - b0 : 65535;
            const char *pin = (const char *)in + (size_t)(b0 * plan->dist) * el;
            char *pout = (char *)out + (size_t)(b0 * plan->dist) * el;
            KArgs a1{n2, n2, 1, n1, plan->scale1, strip_map(n2 * (int64_t)el)};
            a1.out_stride = 1;
            a1.outer = (int)nb;
            a1.outer_in_dist = a1.outer_out_dist = plan->dist;
            a1.aux = plan->log2s;
            hipError_t e = launch_fft(n1, plan->v1, mi355fft::LAYOUT_COLS, plan->storage, plan->storage, inv,
                                      mi355fft::EPI_TWIDDLE, pin, pout, plan->tw1, plan->ftab, a1, stream);
            if (e != hipSuccess) return map_hip(e);
            KArgs a2{n1, n1, 1, 1, plan->scale_last, strip_map(n1 * (int64_t)el)};
            a2.outer = (int)nb;
            a2.outer_in_dist = a2.outer_out_dist = plan->dist;
            e = launch_fft(n2, plan->v2, mi355fft::LAYOUT_COLS, plan->storage, plan->storage, inv,
                           mi355fft::EPI_NONE, pout, pout, plan->tw2, nullptr, a2, stream);
            if (e != hipSuccess) return map_hip(e);
        }
        return FFT_OK;
    }
    const KArgs a{plan->batch, plan->stride, plan->dist, plan->dist, plan->scale, plan->xcd_remap};
    const int inv = plan->dir == FFT_INVERSE;
    if (plan->mfma) {
        return map_hip(plan->n == 4096 ? mi355fft::launch_fft_mfma_n4096(inv, in, out, plan->tw, plan->amat, a, stream)
                                       : mi355fft::launch_fft_mfma_n16384(inv, in, out, plan->tw, plan->amat, a,
                                                                          stream));
    }
    return map_hip(launch_fft(plan->n, plan->variant, plan->layout, plan->storage, plan->storage, inv,
                              mi355fft::EPI_NONE, in, out, plan->tw, nullptr, a, stream));
} catch (const std::bad_alloc &) {
    return FFT_ENOMEM;
} catch (...) {
    return FFT_EHIP;
}

int fft_plan_destroy(fft_plan *plan) {
    delete plan;
    return FFT_OK;
}

size_t sar_workspace_bytes(int64_t n_az, int64_t n_rg, int inter_storage) {
    if (!supported_n(n_az) || !supported_n(n_rg)) return 0;
    if (inter_storage != FFT_STORAGE_FP32 && inter_storage != FFT_STORAGE_FP16) return 0;
    const size_t spectra = (size_t)(n_az + n_rg) * sizeof(float2);  // multiple of 256 bytes
    const size_t el = inter_storage == FFT_STORAGE_FP32 ? 8 : 4;
    return spectra + kChainFlagBytes + (size_t)n_az * (size_t)n_rg * el;
}

// An azimuth pass over 8192- or 16384-point columns holds one or two columns
// per workgroup (8- or 16-byte pieces of each row).  With FP32 intermediates
// it runs instead as three passes of short columns in the four-step form
// (n_az = n1 * n2, n1 = 128, j = n2 j1 + j2, k = k1 + n1 k2), each reading
// and writing wide pieces of the rows:
//   B1  for each j2: 128-point FFTs down rows n2 j1 + j2, output k1 times
//       W^(j2 k1), to rows j2 n1 + k1 of the workspace;
//   B2  in place, for each k1: n2-point FFT down rows j2 n1 + k1 (giving
//       X[k1 + n1 k2]), times conj(H_a[k1 + n1 k2]) / n_az, n2-point inverse
//       FFT, output j2 times conj(W^(j2 k1));
//   B3  for each j2: 128-point inverse FFTs down rows j2 n1 + k1, output j1 to
//       row n2 j1 + j2 of the image.
// The range pass then writes its result into `out`, which B1 reads.  A forced
// column shape (MI355FFT_COL_VARIANT) keeps the single column pass.
static bool long_azimuth(int64_t n_az, int inter_storage) {
    const char *cv = std::getenv("MI355FFT_COL_VARIANT");
    if (cv && cv[0]) return false;
    return inter_storage == FFT_STORAGE_FP32 && (n_az == 8192 || n_az == 16384);
}

}  // extern "C"

namespace {

// Device tables one SAR image needs: the twiddles of both axes and, for the
// long-azimuth form, those of its 128-point and n2-point columns and the
// two-level table of the azimuth length.
struct SarTables {
    const float2 *tw_rg, *tw_az, *tw1, *tw2, *ftab;
};

int sar_long_azimuth(int64_t n_az, int64_t n_rg, const void *raw, void *out, void *mid, const float2 *h_rg,
                            const float2 *h_az, const SarTables &t, int vrow, hipStream_t stream) {
    using mi355fft::LAYOUT_COLS;
    const int64_t n1 = 128, n2 = n_az / n1;
    const int log2s = (ilog2(n_az) + 1) / 2;
    // range pass into `out` (H_r already carries 1/n_rg)
    const KArgs ar{n_az, 1, n_rg, n_rg, 1.0f, 0};
    hipError_t e = launch_fft(n_rg, vrow, mi355fft::LAYOUT_ROWS, FFT_STORAGE_FP32, FFT_STORAGE_FP32, 0,
                              mi355fft::EPI_MATCHED, raw, out, t.tw_rg, h_rg, ar, stream);
    if (e != hipSuccess) return map_hip(e);
    KArgs b1{n_rg, n2 * n_rg, 1, 1, 1.0f, strip_map(n2 * n_rg * 8)};
    b1.out_stride = n_rg;
    b1.outer = (int)n2;
    b1.outer_in_dist = n_rg;
    b1.outer_out_dist = n1 * n_rg;
    b1.aux = log2s;
    e = launch_fft(n1, -1, LAYOUT_COLS, FFT_STORAGE_FP32, FFT_STORAGE_FP32, 0, mi355fft::EPI_TWIDDLE_Y, out, mid,
                   t.tw1, t.ftab, b1, stream);
    if (e != hipSuccess) return map_hip(e);
    KArgs b2{n_rg, n1 * n_rg, 1, 1, 1.0f, strip_map(n1 * n_rg * 8)};  // H_a carries 1/n_az
    b2.outer = (int)n1;
    b2.outer_in_dist = b2.outer_out_dist = n_rg;
    b2.aux = log2s;
    b2.spec_shift = ilog2(n1);
    b2.tab2 = t.ftab;
    e = launch_fft(n2, -1, LAYOUT_COLS, FFT_STORAGE_FP32, FFT_STORAGE_FP32, 0, mi355fft::EPI_MATCHED_Y, mid, mid,
                   t.tw2, h_az, b2, stream);
    if (e != hipSuccess) return map_hip(e);
    KArgs b3{n_rg, n_rg, 1, 1, 1.0f, strip_map(n_rg * 8)};
    b3.out_stride = n2 * n_rg;
    b3.outer = (int)n2;
    b3.outer_in_dist = n1 * n_rg;
    b3.outer_out_dist = n_rg;
    e = launch_fft(n1, -1, LAYOUT_COLS, FFT_STORAGE_FP32, FFT_STORAGE_FP32, 1, mi355fft::EPI_NONE, mid, out, t.tw1,
                   nullptr, b3, stream);
    return map_hip(e);
}

// Argument checks shared by both SAR entry points (no HIP call).
int sar_check(int64_t n_az, int64_t n_rg, int inter_storage, const void *raw, const void *range_ref,
                     const void *az_ref, const void *out) {
    if (!raw || !range_ref || !az_ref || !out) return FFT_EINVAL;
    if (inter_storage != FFT_STORAGE_FP32 && inter_storage != FFT_STORAGE_FP16) return FFT_EINVAL;
    if (n_az < 1 || n_rg < 1) return FFT_EINVAL;
    if (!supported_n(n_az) || !supported_n(n_rg)) return FFT_EUNSUPPORTED;
    if (!aligned(raw, 8) || !aligned(range_ref, 8) || !aligned(az_ref, 8) || !aligned(out, 8)) return FFT_EALIGN;
    const size_t img = (size_t)n_az * (size_t)n_rg * 8;
    if (overlaps(out, img, raw, img)) return FFT_EINVAL;
    return FFT_OK;
}

// The chain itself, on checked arguments, with its tables and workspace given.
int sar_run(int64_t n_az, int64_t n_rg, int inter_storage, const void *raw, const void *range_ref,
                   const void *az_ref, void *out, void *workspace, const SarTables &t, hipStream_t stream) {
    const int vrow = chosen_variant(n_rg, mi355fft::LAYOUT_ROWS);
    const int vcol = chosen_variant(n_az, mi355fft::LAYOUT_COLS);
    const int vref = chosen_variant(n_az, mi355fft::LAYOUT_ROWS);
    if (vrow == -2 || vcol == -2 || vref == -2) return FFT_EINVAL;

    float2 *h_rg = reinterpret_cast<float2 *>(workspace);
    float2 *h_az = h_rg + n_rg;
    auto *flag = reinterpret_cast<unsigned long long *>(h_az + n_az);
    void *mid = reinterpret_cast<char *>(flag) + kChainFlagBytes;
    using mi355fft::EPI_MATCHED;
    using mi355fft::EPI_NONE;
    using mi355fft::LAYOUT_COLS;
    using mi355fft::LAYOUT_ROWS;
    hipError_t e;

    // reference spectra into the workspace, each with its pass's scale folded
    // in (a power of two, so exact): H_r / n_rg and H_a / n_az; the passes
    // multiply by their conjugates.
    const float s_rg = (float)(1.0 / (double)n_rg), s_az = (float)(1.0 / (double)n_az);
    auto separate_references = [&](bool range, bool azimuth) -> hipError_t {
        hipError_t err = hipSuccess;
        if (range && azimuth && n_rg == n_az) {
            // one launch of two transforms (the input distance is the signed
            // distance between the two reference buffers)
            const long long gap = ((const char *)az_ref - (const char *)range_ref) / (long long)sizeof(float2);
            const KArgs a{2, 1, gap, n_rg, s_rg, 0};
            return launch_fft(n_rg, vrow, LAYOUT_ROWS, 0, 0, 0, EPI_NONE, range_ref, h_rg, t.tw_rg, nullptr, a,
                              stream);
        }
        if (range) {
            const KArgs a1{1, 1, n_rg, n_rg, s_rg, 0};
            err = launch_fft(n_rg, vrow, LAYOUT_ROWS, 0, 0, 0, EPI_NONE, range_ref, h_rg, t.tw_rg, nullptr, a1, stream);
            if (err != hipSuccess) return err;
        }
        if (azimuth) {
            const KArgs a2{1, 1, n_az, n_az, s_az, 0};
            err = launch_fft(n_az, vref, LAYOUT_ROWS, 0, 0, 0, EPI_NONE, az_ref, h_az, t.tw_az, nullptr, a2, stream);
        }
        return err;
    };

    if (long_azimuth(n_az, inter_storage)) {
        e = separate_references(true, true);
        if (e != hipSuccess) return map_hip(e);
        return sar_long_azimuth(n_az, n_rg, raw, out, mid, h_rg, h_az, t, vrow, stream);
    }

    // pass 1, rows (range): FFT, * conj(H_r / n_rg), IFFT -> intermediate.
    // Its first workgroups compute the reference spectra (both of them when
    // the image is square, else H_r, with H_a a launch of its own), saving
    // the launch that would precede the pass; a row shape that cannot hold
    // them (persistent) falls back to that launch.
    const bool square = n_az == n_rg;
    if (!square) {
        e = separate_references(false, true);
        if (e != hipSuccess) return map_hip(e);
    }
    KArgs ar{n_az, 1, n_rg, n_rg, 1.0f, 0};
    ar.ref_rows = square ? 2 : 1;
    ar.ref_in[0] = reinterpret_cast<const float2 *>(range_ref);
    ar.ref_out[0] = h_rg;
    ar.ref_scale[0] = s_rg;
    ar.ref_in[1] = reinterpret_cast<const float2 *>(az_ref);
    ar.ref_out[1] = h_az;
    ar.ref_scale[1] = s_az;
    ar.ref_flag = flag;
    ar.ref_epoch = next_chain_epoch();
    e = launch_fft(n_rg, vrow, LAYOUT_ROWS, FFT_STORAGE_FP32, inter_storage, 0, EPI_MATCHED, raw, mid, t.tw_rg, h_rg,
                   ar, stream);
    if (e == hipErrorNotSupported) {
        e = separate_references(true, square);
        if (e != hipSuccess) return map_hip(e);
        const KArgs ar2{n_az, 1, n_rg, n_rg, 1.0f, 0};
        e = launch_fft(n_rg, vrow, LAYOUT_ROWS, FFT_STORAGE_FP32, inter_storage, 0, EPI_MATCHED, raw, mid, t.tw_rg,
                       h_rg, ar2, stream);
    }
    if (e != hipSuccess) return map_hip(e);

    // pass 2, columns (azimuth): FFT, * conj(H_a / n_az), IFFT -> image; it
    // clears the flag the range pass waited on
    KArgs ac{n_rg, n_rg, 1, 1, 1.0f, strip_map(n_rg * 8)};
    ac.clear_flag = flag;
    e = launch_fft(n_az, vcol, LAYOUT_COLS, inter_storage, FFT_STORAGE_FP32, 0, EPI_MATCHED, mid, out, t.tw_az, h_az,
                   ac, stream);
    return map_hip(e);
}

// The allocation-free SAR entry point's fixed device array (noalloc.hip):
// the twiddle tables of every length 64 ... 16384 and the two-level tables of
// 8192 and 16384, filled once per device, then the chain's workspace.
constexpr size_t na_tw_entries_below(int64_t n) {  // tables of the lengths 64 .. n / 2
    size_t e = 0;
    for (int64_t m = 64; m < n; m *= 2) e += (size_t)mi355fft::twiddle_entries(m);
    return e;
}
constexpr size_t kNaTwBytes = na_tw_entries_below(32768) * sizeof(float2);  // lengths 64 .. 16384
constexpr size_t kNaFtabOffset = kNaTwBytes;
constexpr size_t kNaFtabBytes = (size_t)(192 + 256) * sizeof(float2);  // 8192: 128 + 64; 16384: 128 + 128
constexpr size_t kNaWorkspaceOffset = mi355fft::round_up_256(kNaFtabOffset + kNaFtabBytes);
static_assert(kNaWorkspaceOffset + 2 * 16384 * sizeof(float2) + kChainFlagBytes + mi355fft::kNoallocMaxImageBytes <=
                  mi355fft::kNoallocScratchBytes,
              "the fixed array holds the tables, both spectra, the flag and the largest intermediate");

size_t na_tw_offset(int64_t n) { return na_tw_entries_below(n) * sizeof(float2); }
size_t na_ftab_offset(int64_t n) { return kNaFtabOffset + (n == 8192 ? 0 : 192 * sizeof(float2)); }

std::mutex g_na_mutex;
std::map<int, char *> g_na;  // device -> its array, tables filled

// This device's copy of the array with its tables filled: the array's address
// (looked up once per device in noalloc.hip) and, on the first call on the
// device, the tables copied in from the host (the same double-precision
// tables the plans use).
int noalloc_base(int device, char **base) {
    std::lock_guard<std::mutex> lock(g_na_mutex);
    auto it = g_na.find(device);
    if (it != g_na.end()) {
        *base = it->second;
        return FFT_OK;
    }
    void *p = nullptr;
    hipError_t e = mi355fft::noalloc_scratch(device, &p);
    if (e != hipSuccess) return map_hip(e);
    char *b = static_cast<char *>(p);
    std::vector<float2> host, all;
    for (int64_t n = 64; n <= 16384; n *= 2) {
        host_twiddles(n, host);
        all.insert(all.end(), host.begin(), host.end());
    }
    for (int64_t n : {int64_t(8192), int64_t(16384)}) {
        host_fourstep_table(n, (ilog2(n) + 1) / 2, host);
        all.insert(all.end(), host.begin(), host.end());
    }
    if (all.size() * sizeof(float2) != kNaTwBytes + kNaFtabBytes) return FFT_EINVAL;  // layout mismatch
    e = hipMemcpy(b, all.data(), all.size() * sizeof(float2), hipMemcpyHostToDevice);
    if (e != hipSuccess) return map_hip(e);
    g_na[device] = b;
    *base = b;
    return FFT_OK;
}

}  // namespace

extern "C" {

int sar_form_image_ex(int64_t n_az, int64_t n_rg, int inter_storage, const void *raw, const void *range_ref,
                      const void *az_ref, void *out, void *workspace, hipStream_t stream) try {
    if (!workspace) return FFT_EINVAL;
    int rc = sar_check(n_az, n_rg, inter_storage, raw, range_ref, az_ref, out);
    if (rc != FFT_OK) return rc;
    if (!aligned(workspace, 256)) return FFT_EALIGN;
    const size_t img = (size_t)n_az * (size_t)n_rg * 8;
    const size_t ws = sar_workspace_bytes(n_az, n_rg, inter_storage);
    if (overlaps(out, img, workspace, ws) || overlaps(raw, img, workspace, ws)) return FFT_EINVAL;
    // the range pass reads the references while it writes the spectra
    if (overlaps(range_ref, (size_t)n_rg * 8, workspace, ws) || overlaps(az_ref, (size_t)n_az * 8, workspace, ws))
        return FFT_EINVAL;

    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return map_hip(e);
    SarTables t{};
    rc = get_twiddles(device, n_rg, &t.tw_rg);
    if (rc == FFT_OK) rc = get_twiddles(device, n_az, &t.tw_az);
    if (rc == FFT_OK && long_azimuth(n_az, inter_storage)) {
        rc = get_twiddles(device, 128, &t.tw1);
        if (rc == FFT_OK) rc = get_twiddles(device, n_az / 128, &t.tw2);
        if (rc == FFT_OK) rc = get_fourstep_table(device, n_az, (ilog2(n_az) + 1) / 2, &t.ftab);
    }
    if (rc != FFT_OK) return rc;
    return sar_run(n_az, n_rg, inter_storage, raw, range_ref, az_ref, out, workspace, t, stream);
} catch (const std::bad_alloc &) {
    return FFT_ENOMEM;
} catch (...) {
    return FFT_EHIP;
}

int sar_form_image_noalloc(int64_t n_az, int64_t n_rg, int inter_storage, const void *raw, const void *range_ref,
                           const void *az_ref, void *out, hipStream_t stream) try {
    int rc = sar_check(n_az, n_rg, inter_storage, raw, range_ref, az_ref, out);
    if (rc != FFT_OK) return rc;
    const size_t el = inter_storage == FFT_STORAGE_FP32 ? 8 : 4;
    if ((size_t)n_az * (size_t)n_rg * el > mi355fft::kNoallocMaxImageBytes) return FFT_EUNSUPPORTED;
    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return map_hip(e);
    char *base = nullptr;
    rc = noalloc_base(device, &base);
    if (rc != FFT_OK) return rc;
    void *ws = base + kNaWorkspaceOffset;
    const size_t img = (size_t)n_az * (size_t)n_rg * 8;
    const size_t wsb = sar_workspace_bytes(n_az, n_rg, inter_storage);
    if (overlaps(out, img, ws, wsb) || overlaps(raw, img, ws, wsb)) return FFT_EINVAL;
    if (overlaps(range_ref, (size_t)n_rg * 8, ws, wsb) || overlaps(az_ref, (size_t)n_az * 8, ws, wsb))
        return FFT_EINVAL;
    auto tw = [&](int64_t n) { return reinterpret_cast<const float2 *>(base + na_tw_offset(n)); };
    SarTables t{tw(n_rg), tw(n_az), nullptr, nullptr, nullptr};
    if (long_azimuth(n_az, inter_storage)) {
        t.tw1 = tw(128);
        t.tw2 = tw(n_az / 128);
        t.ftab = reinterpret_cast<const float2 *>(base + na_ftab_offset(n_az));
    }
    return sar_run(n_az, n_rg, inter_storage, raw, range_ref, az_ref, out, ws, t, stream);
} catch (const std::bad_alloc &) {
    return FFT_ENOMEM;
} catch (...) {
    return FFT_EHIP;
}

size_t sar_rd_workspace_bytes(int64_t n_az, int64_t n_rg, int inter_storage) {
    if (!supported_n(n_az) || !supported_n(n_rg) || n_az * n_rg > kMaxRdPoints) return 0;
    if (inter_storage != FFT_STORAGE_FP32 && inter_storage != FFT_STORAGE_FP16) return 0;
    const size_t el = inter_storage == FFT_STORAGE_FP32 ? 8 : 4;
    return rd_mid_offset(n_az, n_rg) + (size_t)n_az * (size_t)n_rg * el;
}

int sar_rd_form_image(int64_t n_az, int64_t n_rg, int inter_storage, const sar_geometry *geo, const void *raw,
                      const void *range_ref, void *out, void *workspace, hipStream_t stream) try {
    if (!geo || !raw || !range_ref || !out || !workspace) return FFT_EINVAL;
    if (inter_storage != FFT_STORAGE_FP32 && inter_storage != FFT_STORAGE_FP16) return FFT_EINVAL;
    if (n_az < 1 || n_rg < 1) return FFT_EINVAL;
    const double g[5] = {geo->wavelength, geo->speed, geo->prf, geo->range_bin, geo->r_near};
    for (double x : g)
        if (!(x > 0.0) || !std::isfinite(x)) return FFT_EINVAL;
    const double x_max = geo->wavelength * geo->prf / (4.0 * geo->speed);  // lambda f_a / 2v at prf / 2
    if (!(x_max < 1.0)) return FFT_EINVAL;
    if (!supported_n(n_az) || !supported_n(n_rg) || n_az * n_rg > kMaxRdPoints) return FFT_EUNSUPPORTED;
    // the migration-correction pass shares one window of rows across a strip
    // of up to 16 range bins, which needs the shift to change by less than a
    // bin across the strip: 15 (1/D - 1) < 1 at the band edge
    if (x_max > kMaxDopplerRatio) return FFT_EUNSUPPORTED;
    if (!aligned(raw, 8) || !aligned(range_ref, 8) || !aligned(out, 8) || !aligned(workspace, 256))
        return FFT_EALIGN;
    const size_t img = (size_t)n_az * (size_t)n_rg * 8;
    const size_t ws = sar_rd_workspace_bytes(n_az, n_rg, inter_storage);
    if (overlaps(out, img, raw, img) || overlaps(out, img, workspace, ws) || overlaps(raw, img, workspace, ws))
        return FFT_EINVAL;
    // the range pass reads the reference while it writes `out` and the spectrum
    if (overlaps(range_ref, (size_t)n_rg * 8, workspace, ws) || overlaps(range_ref, (size_t)n_rg * 8, out, img))
        return FFT_EINVAL;

    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return map_hip(e);
    const float2 *tw_rg = nullptr, *tw_az = nullptr;
    int rc = get_twiddles(device, n_rg, &tw_rg);
    if (rc == FFT_OK) rc = get_twiddles(device, n_az, &tw_az);
    if (rc != FFT_OK) return rc;
    const int vrow = chosen_variant(n_rg, mi355fft::LAYOUT_ROWS);
    const int vcol = chosen_variant(n_az, mi355fft::LAYOUT_COLS);
    const int vrcmc = chosen_variant(n_az, mi355fft::LAYOUT_RCMC);
    if (vrow == -2 || vcol == -2 || vrcmc == -2) return FFT_EINVAL;

    const float2 *interp = nullptr;
    rc = get_interp(device, &interp);
    if (rc != FFT_OK) return rc;

    using namespace mi355fft;
    char *wsb = reinterpret_cast<char *>(workspace);
    float2 *h_rg = reinterpret_cast<float2 *>(wsb);
    void *tables = wsb + rd_tables_offset(n_rg);
    void *zt = wsb + rd_mid_offset(n_az, n_rg);

    auto *flag = reinterpret_cast<unsigned long long *>(wsb + rd_flag_offset(n_rg));
    const float s_rg = (float)(1.0 / (double)n_rg);  // H_r / n_rg (exact)

    // 1: range compression, rows: FFT, * conj(H_r) / n_rg, IFFT.  The
    //    range-compressed image is kept in `out`, which the last pass
    //    overwrites with the focused image.  H_r carries the 1/n_rg; the
    //    pass's workgroup 0 computes it (a row shape that cannot falls back
    //    to a launch of its own).
    KArgs ar{n_az, 1, n_rg, n_rg, 1.0f, 0};
    ar.ref_rows = 1;
    ar.ref_in[0] = reinterpret_cast<const float2 *>(range_ref);
    ar.ref_out[0] = h_rg;
    ar.ref_scale[0] = s_rg;
    ar.ref_flag = flag;
    ar.ref_epoch = next_chain_epoch();
    e = launch_fft(n_rg, vrow, LAYOUT_ROWS, FFT_STORAGE_FP32, inter_storage, 0, EPI_MATCHED, raw, out, tw_rg, h_rg,
                   ar, stream);
    if (e == hipErrorNotSupported) {
        const KArgs aref{1, 1, n_rg, n_rg, s_rg, 0};
        e = launch_fft(n_rg, vrow, LAYOUT_ROWS, 0, 0, 0, EPI_NONE, range_ref, h_rg, tw_rg, nullptr, aref, stream);
        if (e != hipSuccess) return map_hip(e);
        const KArgs ar2{n_az, 1, n_rg, n_rg, 1.0f, 0};
        e = launch_fft(n_rg, vrow, LAYOUT_ROWS, FFT_STORAGE_FP32, inter_storage, 0, EPI_MATCHED, raw, out, tw_rg,
                       h_rg, ar2, stream);
    }
    if (e != hipSuccess) return map_hip(e);
    // 2: azimuth FFT of every range bin (a column), / n_az, written as one row
    //    per range bin (the transposed range-Doppler image)
    KArgs ab{n_rg, n_rg, 1, n_az, (float)(1.0 / (double)n_az), strip_map(n_rg * 8)};
    ab.out_stride = 1;
    //    this pass also fills the tables of the migration pass (one entry per
    //    thread: its n_rg * n_az / P threads cover n_az, n_rg and the rows)
    ab.rd_geo = RdGeometry{g[0], g[1], g[2], g[3], g[4]};
    ab.rd_interp = interp;
    ab.rd_tables = tables;
    ab.clear_flag = flag;  // the range pass has finished: no reader remains
    e = launch_fft(n_az, vcol, LAYOUT_COLS, inter_storage, inter_storage, 0, EPI_SCALE, out, zt, tw_az, nullptr, ab,
                   stream);
    if (e != hipSuccess) return map_hip(e);
    // 3-5: migration correction, azimuth filter and azimuth inverse FFT: reads
    //    rows of the transposed image, writes the columns of the focused image
    KArgs ac{n_rg, 1, n_az, 1, 1.0f, strip_map(n_rg * 8)};
    ac.out_stride = n_rg;
    e = launch_fft(n_az, vrcmc, LAYOUT_RCMC, inter_storage, FFT_STORAGE_FP32, 1, EPI_RCMC, zt, out, tw_az,
                   reinterpret_cast<const float2 *>(tables), ac, stream);
    return map_hip(e);
} catch (const std::bad_alloc &) {
    return FFT_ENOMEM;
} catch (...) {
    return FFT_EHIP;
}

int sar_form_image(const void *raw, const void *range_ref, const void *az_ref, void *out, hipStream_t stream) try {
    if (!raw || !range_ref || !az_ref || !out) return FFT_EINVAL;
    if (fail_alloc_hook()) return FFT_ENOMEM;  // test hook: device allocation fails
    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return map_hip(e);
    void *ws = nullptr;
    {
        std::lock_guard<std::mutex> lock(g_ws_mutex);
        auto it = g_ws.find(device);
        if (it != g_ws.end()) {
            ws = it->second;
        } else {
            e = hipMalloc(&ws, sar_workspace_bytes(4096, 4096, FFT_STORAGE_FP32));
            if (e != hipSuccess) return map_hip(e);
            g_ws[device] = ws;
        }
    }
    return sar_form_image_ex(4096, 4096, FFT_STORAGE_FP32, raw, range_ref, az_ref, out, ws, stream);
} catch (const std::bad_alloc &) {
    return FFT_ENOMEM;
} catch (...) {
    return FFT_EHIP;
}

const char *fft_strerror(int code) {
    switch (code) {
        case FFT_OK: return "success";
        case FFT_EINVAL: return "invalid argument";
        case FFT_EUNSUPPORTED: return "unsupported size or configuration";
        case FFT_ENOMEM: return "out of memory";
        case FFT_EALIGN: return "pointer not aligned to one complex element";
        case FFT_EHIP: return "HIP runtime error";
        default: return "unknown error code";
    }
}

}  // extern "C"
