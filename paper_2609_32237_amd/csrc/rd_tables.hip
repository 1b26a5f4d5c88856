// rd_tables.hip -- per-call tables of the range-Doppler chain (Section X).
//
// For each Doppler bin k (frequency f_k = k prf / n_az, minus prf in the upper
// half) with x = lambda f_k / (2 v) and D = sqrt(1 - x^2):
//   migration    (1/D - 1) / range_bin = x^2 / (D (1 + D)) / range_bin, so the
//                echo of slant range R0 sits R0 times this many bins further
//                out (written without cancellation for small x);
//   filter rate  2 (D - 1) / lambda = -2 x^2 / ((1 + D) lambda) cycles per metre
//                of R0, kept as a float pair hi + lo so that the kernel can
//                form R0 times it to about 1e-7 cycles (Section X's second
//                fix: the phase reaches 1e4 rad at the band edge).
// For each range bin n: R0_n = r_near + n range_bin as a float pair.
// The interpolator rows (computed once per device on the host) are copied in.
#include <hip/hip_runtime.h>

#include "fft_launch.h"

namespace mi355fft {
namespace {

__device__ float2 split(double x) {
    const float hi = (float)x;
    return make_float2(hi, (float)(x - (double)hi));
}

__global__ void rd_tables_kernel(long long n_az, long long n_rg, double wavelength, double speed, double prf,
                                 double range_bin, double r_near, const float2 *interp_src, float4 *rows,
                                 float2 *cols, float2 *interp) {
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n_az) {
        const double f = (double)(i < n_az / 2 ? i : i - n_az) * prf / (double)n_az;
        const double x = wavelength * f / (2.0 * speed), x2 = x * x;
        const double d = sqrt(1.0 - x2);
        const double mig = x2 / (d * (1.0 + d)) / range_bin;
        const float2 rate = split(-2.0 * x2 / ((1.0 + d) * wavelength));
        rows[i] = make_float4((float)mig, rate.x, rate.y, 0.0f);
    }
    if (i < n_rg) cols[i] = split(r_near + (double)i * range_bin);
    if (i < (kRcmcSub + 1) * kRcmcTaps) interp[i] = interp_src[i];
}

}  // namespace

hipError_t launch_rd_tables(long long n_az, long long n_rg, double wavelength, double speed, double prf,
                            double range_bin, double r_near, const float2 *interp_src, void *tables,
                            hipStream_t s) {
    const RdTablesLayout l = rd_tables_layout(n_az, n_rg);
    char *base = reinterpret_cast<char *>(tables);
    long long most = n_az > n_rg ? n_az : n_rg;
    if (most < (kRcmcSub + 1) * kRcmcTaps) most = (kRcmcSub + 1) * kRcmcTaps;
    const unsigned blocks = (unsigned)((most + 255) / 256);
    return launch_kernel(rd_tables_kernel, dim3(blocks), dim3(256), s, n_az, n_rg, wavelength, speed, prf, range_bin,
                         r_near, interp_src, reinterpret_cast<float4 *>(base + l.rows),
                         reinterpret_cast<float2 *>(base + l.cols), reinterpret_cast<float2 *>(base + l.interp));
}

}  // namespace mi355fft
