// rd_tables.hpp -- per-call tables of the range-Doppler chain (Section X),
// one entry per thread, computed by the azimuth-FFT pass before its
// transform (no launch of their own).
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
#pragma once

#include "fft_launch.h"

namespace mi355fft {

__device__ __forceinline__ float2 split_double(double x) {
    const float hi = (float)x;
    return make_float2(hi, (float)(x - (double)hi));
}

// Entry i of every table (entries past a table's end are skipped); the
// tables block is laid out by rd_tables_layout(n_az, n_rg).
__device__ __forceinline__ void rd_table_entry(long long i, long long n_az, long long n_rg, const RdGeometry &g,
                                               const float2 *__restrict__ interp_src, void *__restrict__ tables) {
    const RdTablesLayout l = rd_tables_layout(n_az, n_rg);
    char *base = reinterpret_cast<char *>(tables);
    if (i < n_az) {
        const double f = (double)(i < n_az / 2 ? i : i - n_az) * g.prf / (double)n_az;
        const double x = g.wavelength * f / (2.0 * g.speed), x2 = x * x;
        const double d = sqrt(1.0 - x2);
        const double mig = x2 / (d * (1.0 + d)) / g.range_bin;
        const float2 rate = split_double(-2.0 * x2 / ((1.0 + d) * g.wavelength));
        reinterpret_cast<float4 *>(base + l.rows)[i] = make_float4((float)mig, rate.x, rate.y, 0.0f);
    }
    if (i < n_rg) reinterpret_cast<float2 *>(base + l.cols)[i] = split_double(g.r_near + (double)i * g.range_bin);
    if (i < (kRcmcSub + 1) * kRcmcTaps) reinterpret_cast<float2 *>(base + l.interp)[i] = interp_src[i];
}

}  // namespace mi355fft
