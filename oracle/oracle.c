/*
 * oracle.c -- plain fp64 CPU reference for the batched FFT and the SAR chain.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, calls or
 * includes this file; only the tests, the smoke check and the benchmark's CPU
 * baseline use it.  It shares no source with the HIP path.
 *
 * Arithmetic is IEEE double throughout.  Complex arrays are interleaved
 * (re, im) pairs of doubles.  Element j of transform b lives at complex index
 * b*dist + j*stride (the same advanced layout as the GPU library).
 *
 * Functions and the passages they follow (paper: "Bandwidth, Not FLOPS: FFT
 * Kernels, Matrix Units and SAR Imaging on Apple M6"):
 *
 *   oracle_dft_direct   The DFT by its definition, O(N^2): the transform every
 *                       FFT in the paper computes (Section III, correctness and
 *                       the 5 N log2 N convention).  Any N >= 1.
 *   oracle_fft          The same transform by iterative radix-2 Cooley-Tukey
 *                       (N a power of two).  Reaches the definition exactly up to
 *                       rounding order.  Twiddles come from cos/sin of
 *                       2*pi*m/N with m < N, one call per table entry, never a
 *                       recurrence.
 *   oracle_sar_chain    Section X: range compression along each pulse (FFT,
 *                       multiply by the conjugate reference spectrum, inverse
 *                       FFT) with its 1/N_r scale, then the azimuth FFT along
 *                       each range bin scaled by 1/N_a, the multiply by the
 *                       conjugate azimuth reference spectrum, and the azimuth
 *                       inverse FFT.  Without range-cell migration correction,
 *                       and with the azimuth filter taken as the conjugate
 *                       azimuth chirp spectrum.
 *   oracle_xcorr2d_points
 *                       The plain definition that chain reaches: the 2-D
 *                       circular cross-correlation of the echo with both
 *                       references, evaluated point by point.
 *   oracle_rd_chain     Section X's full range-Doppler chain, in the paper's
 *                       order: range compression; the azimuth FFT along each
 *                       range bin (scaled by 1/N_a); range-cell migration
 *                       correction with an 8-tap interpolator whose table
 *                       rows are blended linearly and whose fractional shift
 *                       comes from the shift alone; the baseband azimuth
 *                       filter exp(+j 4 pi R0 (D - 1) / lambda) with
 *                       D = sqrt(1 - (lambda f_a / 2v)^2), its phase reduced
 *                       in cycles; the azimuth inverse FFT.  Can stop after
 *                       any step so each one can be checked on its own.
 *   oracle_rd_interp_table
 *                       The interpolator's table (Kaiser-windowed sinc,
 *                       8 taps, 129 fractional shifts, unit sum per row).
 *
 * Both directions are unnormalised: forward uses exp(-2 pi i n k / N), inverse
 * exp(+2 pi i n k / N).
 *
 * Return codes: 0 on success, -1 on an invalid argument, -3 on allocation
 * failure.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_OK 0
#define OR_EINVAL (-1)
#define OR_ENOMEM (-3)

static const double OR_TWO_PI = 6.283185307179586476925286766559;

static int is_pow2(int64_t n) { return n > 0 && (n & (n - 1)) == 0; }

/* Table of exp(sign * 2 pi i m / n) for m in [0, n).  m/n is exact in binary
 * for the sizes used, so the angle carries one rounding. */
static double *unit_roots(int64_t n, int sign) {
    double *w = (double *)malloc(sizeof(double) * 2 * (size_t)n);
    if (!w) return NULL;
    for (int64_t m = 0; m < n; ++m) {
        double ang = OR_TWO_PI * ((double)m / (double)n);
        w[2 * m] = cos(ang);
        w[2 * m + 1] = (double)sign * sin(ang);
    }
    return w;
}

/* ---------------------------------------------------------------------- */
/* DFT by definition                                                       */
/* ---------------------------------------------------------------------- */

int oracle_dft_direct(int64_t n, int64_t batch, int64_t stride, int64_t dist, int sign,
                      const double *in, double *out) {
    if (n < 1 || batch < 0 || (sign != -1 && sign != 1) || !in || !out) return OR_EINVAL;
    double *w = unit_roots(n, sign);
    double *acc = (double *)malloc(sizeof(double) * 2 * (size_t)n);
    if (!w || !acc) {
        free(w);
        free(acc);
        return OR_ENOMEM;
    }
    for (int64_t b = 0; b < batch; ++b) {
        for (int64_t k = 0; k < n; ++k) {
            double sr = 0.0, si = 0.0;
            for (int64_t j = 0; j < n; ++j) {
                int64_t m = (j * k) % n; /* exact argument reduction */
                const double *x = in + 2 * (b * dist + j * stride);
                sr += x[0] * w[2 * m] - x[1] * w[2 * m + 1];
                si += x[0] * w[2 * m + 1] + x[1] * w[2 * m];
            }
            acc[2 * k] = sr;
            acc[2 * k + 1] = si;
        }
        for (int64_t k = 0; k < n; ++k) {
            double *y = out + 2 * (b * dist + k * stride);
            y[0] = acc[2 * k];
            y[1] = acc[2 * k + 1];
        }
    }
    free(w);
    free(acc);
    return OR_OK;
}

/* ---------------------------------------------------------------------- */
/* Radix-2 Cooley-Tukey, one contiguous transform in place                */
/* ---------------------------------------------------------------------- */

/* a: n complex values, contiguous.  w: exp(sign 2 pi i m / n), m in [0, n). */
static void fft_inplace(int64_t n, double *a, const double *w) {
    /* bit-reversal permutation */
    for (int64_t i = 1, j = 0; i < n; ++i) {
        int64_t bit = n >> 1;
        for (; j & bit; bit >>= 1) j ^= bit;
        j ^= bit;
        if (i < j) {
            double tr = a[2 * i], ti = a[2 * i + 1];
            a[2 * i] = a[2 * j];
            a[2 * i + 1] = a[2 * j + 1];
            a[2 * j] = tr;
            a[2 * j + 1] = ti;
        }
    }
    /* butterflies: length-len sub-transforms from pairs of length-len/2 ones */
    for (int64_t len = 2; len <= n; len <<= 1) {
        int64_t half = len >> 1;
        int64_t step = n / len; /* exp(sign 2 pi i k / len) = w[k * step] */
        for (int64_t base = 0; base < n; base += len) {
            for (int64_t k = 0; k < half; ++k) {
                const double *tw = w + 2 * (k * step);
                double *u = a + 2 * (base + k);
                double *v = a + 2 * (base + k + half);
                double vr = v[0] * tw[0] - v[1] * tw[1];
                double vi = v[0] * tw[1] + v[1] * tw[0];
                v[0] = u[0] - vr;
                v[1] = u[1] - vi;
                u[0] = u[0] + vr;
                u[1] = u[1] + vi;
            }
        }
    }
}

typedef struct {
    int64_t n, b0, b1, stride, dist;
    const double *in;
    double *out;
    const double *w;
    int status;
} fft_job;

static void *fft_worker(void *arg) {
    fft_job *job = (fft_job *)arg;
    double *buf = (double *)malloc(sizeof(double) * 2 * (size_t)job->n);
    if (!buf) {
        job->status = OR_ENOMEM;
        return NULL;
    }
    for (int64_t b = job->b0; b < job->b1; ++b) {
        for (int64_t j = 0; j < job->n; ++j) {
            const double *x = job->in + 2 * (b * job->dist + j * job->stride);
            buf[2 * j] = x[0];
            buf[2 * j + 1] = x[1];
        }
        fft_inplace(job->n, buf, job->w);
        for (int64_t j = 0; j < job->n; ++j) {
            double *y = job->out + 2 * (b * job->dist + j * job->stride);
            y[0] = buf[2 * j];
            y[1] = buf[2 * j + 1];
        }
    }
    free(buf);
    job->status = OR_OK;
    return NULL;
}

/* Runs fn over jobs[0..nt) on nt threads (the calling thread takes job 0). */
static int run_jobs(void *(*fn)(void *), void *jobs, size_t job_size, int nt) {
    pthread_t *th = (pthread_t *)calloc((size_t)nt, sizeof(pthread_t));
    char *started = (char *)calloc((size_t)nt, 1);
    if (!th || !started) {
        free(th);
        free(started);
        return OR_ENOMEM;
    }
    for (int i = 1; i < nt; ++i)
        started[i] = pthread_create(&th[i], NULL, fn, (char *)jobs + (size_t)i * job_size) == 0;
    fn(jobs);
    for (int i = 1; i < nt; ++i) {
        if (started[i])
            pthread_join(th[i], NULL);
        else
            fn((char *)jobs + (size_t)i * job_size); /* could not spawn: run inline */
    }
    free(th);
    free(started);
    return OR_OK;
}

int oracle_fft(int64_t n, int64_t batch, int64_t stride, int64_t dist, int sign,
               const double *in, double *out, int nthreads) {
    if (!is_pow2(n) || batch < 0 || (sign != -1 && sign != 1) || !in || !out) return OR_EINVAL;
    if (batch == 0) return OR_OK;
    int nt = nthreads < 1 ? 1 : nthreads;
    if (nt > batch) nt = (int)batch;
    double *w = unit_roots(n, sign);
    fft_job *jobs = (fft_job *)calloc((size_t)nt, sizeof(fft_job));
    if (!w || !jobs) {
        free(w);
        free(jobs);
        return OR_ENOMEM;
    }
    for (int i = 0; i < nt; ++i) {
        jobs[i].n = n;
        jobs[i].b0 = batch * i / nt;
        jobs[i].b1 = batch * (i + 1) / nt;
        jobs[i].stride = stride;
        jobs[i].dist = dist;
        jobs[i].in = in;
        jobs[i].out = out;
        jobs[i].w = w;
        jobs[i].status = OR_EINVAL;
    }
    int rc = run_jobs(fft_worker, jobs, sizeof(fft_job), nt);
    for (int i = 0; rc == OR_OK && i < nt; ++i)
        if (jobs[i].status != OR_OK) rc = jobs[i].status;
    free(w);
    free(jobs);
    return rc;
}

/* ---------------------------------------------------------------------- */
/* SAR range-Doppler chain (Section X), without RCMC                       */
/* ---------------------------------------------------------------------- */

typedef struct {
    int64_t n_az, n_rg, i0, i1;
    const double *src;   /* pass 1: raw echo; pass 2: range-compressed image */
    double *dst;
    const double *spec;  /* reference spectrum along the processed axis */
    const double *wf, *wi; /* forward / inverse unit roots for that axis */
    int columns;         /* 0: process rows (range), 1: columns (azimuth) */
    int status;
} sar_job;

static void *sar_worker(void *arg) {
    sar_job *job = (sar_job *)arg;
    int64_t len = job->columns ? job->n_az : job->n_rg;
    double *buf = (double *)malloc(sizeof(double) * 2 * (size_t)len);
    if (!buf) {
        job->status = OR_ENOMEM;
        return NULL;
    }
    double inv_len = 1.0 / (double)len;
    for (int64_t i = job->i0; i < job->i1; ++i) {
        /* gather one line: a pulse (row) or a range bin (column) */
        for (int64_t j = 0; j < len; ++j) {
            int64_t idx = job->columns ? j * job->n_rg + i : i * job->n_rg + j;
            buf[2 * j] = job->src[2 * idx];
            buf[2 * j + 1] = job->src[2 * idx + 1];
        }
        fft_inplace(len, buf, job->wf);
        /* X[k] * conj(H[k]) / len  (1/N_r in range compression; 1/N_a on the
         * azimuth FFT output) */
        for (int64_t k = 0; k < len; ++k) {
            double xr = buf[2 * k] * inv_len, xi = buf[2 * k + 1] * inv_len;
            double hr = job->spec[2 * k], hi = -job->spec[2 * k + 1];
            buf[2 * k] = xr * hr - xi * hi;
            buf[2 * k + 1] = xr * hi + xi * hr;
        }
        fft_inplace(len, buf, job->wi);
        for (int64_t j = 0; j < len; ++j) {
            int64_t idx = job->columns ? j * job->n_rg + i : i * job->n_rg + j;
            job->dst[2 * idx] = buf[2 * j];
            job->dst[2 * idx + 1] = buf[2 * j + 1];
        }
    }
    free(buf);
    job->status = OR_OK;
    return NULL;
}

static int sar_axis(int64_t n_az, int64_t n_rg, int columns, const double *src, double *dst,
                    const double *ref, int nthreads) {
    int64_t len = columns ? n_az : n_rg;
    int64_t lines = columns ? n_rg : n_az;
    int nt = nthreads < 1 ? 1 : nthreads;
    if (nt > lines) nt = (int)lines;
    double *wf = unit_roots(len, -1);
    double *wi = unit_roots(len, +1);
    double *spec = (double *)malloc(sizeof(double) * 2 * (size_t)len);
    sar_job *jobs = (sar_job *)calloc((size_t)nt, sizeof(sar_job));
    int rc = OR_OK;
    if (!wf || !wi || !spec || !jobs) {
        rc = OR_ENOMEM;
        goto done;
    }
    /* reference spectrum H = FFT(ref) */
    memcpy(spec, ref, sizeof(double) * 2 * (size_t)len);
    fft_inplace(len, spec, wf);
    for (int i = 0; i < nt; ++i) {
        jobs[i].n_az = n_az;
        jobs[i].n_rg = n_rg;
        jobs[i].i0 = lines * i / nt;
        jobs[i].i1 = lines * (i + 1) / nt;
        jobs[i].src = src;
        jobs[i].dst = dst;
        jobs[i].spec = spec;
        jobs[i].wf = wf;
        jobs[i].wi = wi;
        jobs[i].columns = columns;
        jobs[i].status = OR_EINVAL;
    }
    rc = run_jobs(sar_worker, jobs, sizeof(sar_job), nt);
    for (int i = 0; rc == OR_OK && i < nt; ++i)
        if (jobs[i].status != OR_OK) rc = jobs[i].status;
done:
    free(wf);
    free(wi);
    free(spec);
    free(jobs);
    return rc;
}

/* raw: n_az x n_rg, rows = pulses.  range_ref: n_rg.  az_ref: n_az.
 * out: n_az x n_rg.  out may not alias raw. */
int oracle_sar_chain(int64_t n_az, int64_t n_rg, const double *raw, const double *range_ref,
                     const double *az_ref, double *out, int nthreads) {
    if (!is_pow2(n_az) || !is_pow2(n_rg) || !raw || !range_ref || !az_ref || !out || raw == out)
        return OR_EINVAL;
    double *mid = (double *)malloc(sizeof(double) * 2 * (size_t)(n_az * n_rg));
    if (!mid) return OR_ENOMEM;
    int rc = sar_axis(n_az, n_rg, 0, raw, mid, range_ref, nthreads);  /* range compression */
    if (rc == OR_OK) rc = sar_axis(n_az, n_rg, 1, mid, out, az_ref, nthreads); /* azimuth */
    free(mid);
    return rc;
}

/* out[p] = sum_{ta, tr} raw[(a_p + ta) mod n_az][(r_p + tr) mod n_rg]
 *                        * conj(az_ref[ta]) * conj(range_ref[tr])
 * Terms whose reference entry is exactly zero contribute nothing and are
 * skipped. */
int oracle_xcorr2d_points(int64_t n_az, int64_t n_rg, const double *raw, const double *range_ref,
                          const double *az_ref, int64_t npts, const int64_t *pa, const int64_t *pr,
                          double *out) {
    if (n_az < 1 || n_rg < 1 || npts < 0 || !raw || !range_ref || !az_ref || !pa || !pr || !out)
        return OR_EINVAL;
    for (int64_t p = 0; p < npts; ++p) {
        if (pa[p] < 0 || pa[p] >= n_az || pr[p] < 0 || pr[p] >= n_rg) return OR_EINVAL;
        double acc_r = 0.0, acc_i = 0.0;
        for (int64_t ta = 0; ta < n_az; ++ta) {
            double har = az_ref[2 * ta], hai = -az_ref[2 * ta + 1];
            if (har == 0.0 && hai == 0.0) continue;
            const double *row = raw + 2 * ((pa[p] + ta) % n_az) * n_rg;
            double sr = 0.0, si = 0.0;
            for (int64_t tr = 0; tr < n_rg; ++tr) {
                double hrr = range_ref[2 * tr], hri = -range_ref[2 * tr + 1];
                if (hrr == 0.0 && hri == 0.0) continue;
                const double *x = row + 2 * ((pr[p] + tr) % n_rg);
                sr += x[0] * hrr - x[1] * hri;
                si += x[0] * hri + x[1] * hrr;
            }
            acc_r += sr * har - si * hai;
            acc_i += sr * hai + si * har;
        }
        out[2 * p] = acc_r;
        out[2 * p + 1] = acc_i;
    }
    return OR_OK;
}

/* ---------------------------------------------------------------------- */
/* The full range-Doppler chain (Section X): range compression, azimuth    */
/* FFT, range-cell migration correction with an 8-tap interpolator, the    */
/* baseband azimuth filter and the azimuth inverse FFT                     */
/* ---------------------------------------------------------------------- */

/* Interpolator: 8-tap sinc weighted by a Kaiser window (beta 2.5) spanning
 * the 8 taps, tabulated at RD_SUB + 1 fractional shifts mu = q / RD_SUB and
 * normalised to unit sum; between table rows the taps are blended linearly
 * (Section X's third numerical fix).  Tap j (0..7) multiplies the sample at
 * offset j - 3 from the integer part of the position. */
#define RD_TAPS 8
#define RD_SUB 128
static const double RD_KAISER_BETA = 2.5;
static const double OR_PI = 3.141592653589793238462643383279;

/* modified Bessel function of the first kind, order 0, by its power series */
static double bessel_i0(double x) {
    double term = 1.0, sum = 1.0, q = 0.25 * x * x;
    for (int k = 1; k < 200; ++k) {
        term *= q / ((double)k * (double)k);
        sum += term;
        if (term < 1e-18 * sum) break;
    }
    return sum;
}

int oracle_rd_interp_table(double *tab) {
    if (!tab) return OR_EINVAL;
    const double norm = 1.0 / bessel_i0(RD_KAISER_BETA);
    for (int q = 0; q <= RD_SUB; ++q) {
        double mu = (double)q / RD_SUB, sum = 0.0;
        for (int j = 0; j < RD_TAPS; ++j) {
            double x = (double)(j - 3) - mu; /* distance from the wanted position */
            double sinc = x == 0.0 ? 1.0 : sin(OR_PI * x) / (OR_PI * x);
            double r = x / 4.0, arg = 1.0 - r * r;
            double win = bessel_i0(RD_KAISER_BETA * sqrt(arg > 0.0 ? arg : 0.0)) * norm;
            tab[q * RD_TAPS + j] = sinc * win;
            sum += sinc * win;
        }
        for (int j = 0; j < RD_TAPS; ++j) tab[q * RD_TAPS + j] /= sum;
    }
    return OR_OK;
}

typedef struct {
    int64_t n_az, n_rg, k0, k1;
    double wavelength, speed, prf, range_bin, r_near;
    int step;            /* 3: RCMC, 4: azimuth filter */
    const double *src;   /* range-Doppler image, rows = Doppler bins */
    double *dst;
    const double *tab;
    int status;
} rd_job;

/* Doppler frequency of azimuth FFT bin k (the upper half is negative). */
static double doppler_hz(int64_t k, int64_t n_az, double prf) {
    return (double)(k < n_az / 2 ? k : k - n_az) * prf / (double)n_az;
}

static void *rd_worker(void *arg) {
    rd_job *job = (rd_job *)arg;
    const int64_t n_rg = job->n_rg;
    for (int64_t k = job->k0; k < job->k1; ++k) {
        /* D = sqrt(1 - (lambda f_a / 2v)^2); D - 1 and 1/D - 1 written so
         * that no cancellation occurs for small f_a */
        double x = job->wavelength * doppler_hz(k, job->n_az, job->prf) / (2.0 * job->speed);
        double d = sqrt(1.0 - x * x);
        double d_minus_1 = -x * x / (1.0 + d);
        double inv_d_minus_1 = x * x / (d * (1.0 + d));
        const double *row = job->src + 2 * k * n_rg;
        double *out = job->dst + 2 * k * n_rg;
        for (int64_t n = 0; n < n_rg; ++n) {
            double r0 = job->r_near + (double)n * job->range_bin; /* range of closest approach */
            if (job->step == 3) {
                /* the echo of range r0 sits at r0 / D in this Doppler bin:
                 * read the image there, dn bins further out */
                double dn = r0 * inv_d_minus_1 / job->range_bin;
                double fl = floor(dn);
                double mu = dn - fl; /* from the shift alone (fourth fix) */
                double qf = mu * RD_SUB;
                int q = (int)floor(qf);
                if (q > RD_SUB - 1) q = RD_SUB - 1;
                double a = qf - (double)q;
                int64_t base = n + (int64_t)fl - 3;
                double sr = 0.0, si = 0.0;
                for (int j = 0; j < RD_TAPS; ++j) {
                    int64_t idx = base + j;
                    if (idx < 0 || idx >= n_rg) continue; /* no data outside the swath */
                    double g = (1.0 - a) * job->tab[q * RD_TAPS + j] + a * job->tab[(q + 1) * RD_TAPS + j];
                    sr += g * row[2 * idx];
                    si += g * row[2 * idx + 1];
                }
                out[2 * n] = sr;
                out[2 * n + 1] = si;
            } else {
                /* exp(+j 4 pi r0 (D - 1) / lambda), the phase taken in cycles
                 * and reduced before the angle is formed */
                double cyc = 2.0 * r0 * d_minus_1 / job->wavelength;
                double ang = OR_TWO_PI * (cyc - nearbyint(cyc));
                double c = cos(ang), s = sin(ang);
                double vr = row[2 * n], vi = row[2 * n + 1];
                out[2 * n] = vr * c - vi * s;
                out[2 * n + 1] = vr * s + vi * c;
            }
        }
    }
    job->status = OR_OK;
    return NULL;
}

static int rd_rows(int64_t n_az, int64_t n_rg, const double *geo, int step, const double *src, double *dst,
                   const double *tab, int nthreads) {
    int nt = nthreads < 1 ? 1 : nthreads;
    if (nt > n_az) nt = (int)n_az;
    rd_job *jobs = (rd_job *)calloc((size_t)nt, sizeof(rd_job));
    if (!jobs) return OR_ENOMEM;
    for (int i = 0; i < nt; ++i) {
        rd_job *j = &jobs[i];
        j->n_az = n_az;
        j->n_rg = n_rg;
        j->k0 = n_az * i / nt;
        j->k1 = n_az * (i + 1) / nt;
        j->wavelength = geo[0];
        j->speed = geo[1];
        j->prf = geo[2];
        j->range_bin = geo[3];
        j->r_near = geo[4];
        j->step = step;
        j->src = src;
        j->dst = dst;
        j->tab = tab;
        j->status = OR_EINVAL;
    }
    int rc = run_jobs(rd_worker, jobs, sizeof(rd_job), nt);
    for (int i = 0; rc == OR_OK && i < nt; ++i)
        if (jobs[i].status != OR_OK) rc = jobs[i].status;
    free(jobs);
    return rc;
}

/* raw: n_az x n_rg echo, rows = pulses.  range_ref: n_rg time-domain pulse
 * replica.  geo = {wavelength [m], platform speed [m/s], PRF [Hz], range bin
 * spacing [m], slant range of bin 0 [m]}.  out: n_az x n_rg, the result after
 * step stop_after:
 *   1  range compression: IFFT(FFT(row) * conj(FFT(range_ref))) / n_rg;
 *   2  azimuth FFT along each range bin, scaled by 1 / n_az;
 *   3  range-cell migration correction;
 *   4  azimuth filter exp(+j 4 pi R0 (D - 1) / lambda);
 *   5  azimuth inverse FFT (unnormalised): the focused image. */
int oracle_rd_chain(int64_t n_az, int64_t n_rg, const double *raw, const double *range_ref, const double *geo,
                    int stop_after, double *out, int nthreads) {
    if (!is_pow2(n_az) || !is_pow2(n_rg) || n_az < 2 || !raw || !range_ref || !geo || !out || raw == out ||
        stop_after < 1 || stop_after > 5)
        return OR_EINVAL;
    if (!(geo[0] > 0.0) || !(geo[1] > 0.0) || !(geo[2] > 0.0) || !(geo[3] > 0.0) || !(geo[4] > 0.0))
        return OR_EINVAL;
    if (geo[0] * geo[2] / (4.0 * geo[1]) >= 1.0) return OR_EINVAL; /* |lambda f_a / 2v| < 1 */
    const size_t n = (size_t)(n_az * n_rg);
    double *a = (double *)malloc(sizeof(double) * 2 * n);
    double *b = (double *)malloc(sizeof(double) * 2 * n);
    double *tab = (double *)malloc(sizeof(double) * (RD_SUB + 1) * RD_TAPS);
    int rc = (a && b && tab) ? OR_OK : OR_ENOMEM;
    if (rc == OR_OK) rc = oracle_rd_interp_table(tab);
    /* 1: range compression */
    if (rc == OR_OK) rc = sar_axis(n_az, n_rg, 0, raw, a, range_ref, nthreads);
    /* 2: azimuth FFT of every range bin (column), scaled by 1 / n_az */
    if (rc == OR_OK && stop_after >= 2) {
        rc = oracle_fft(n_az, n_rg, n_rg, 1, -1, a, b, nthreads);
        const double s = 1.0 / (double)n_az;
        for (size_t i = 0; rc == OR_OK && i < 2 * n; ++i) b[i] *= s;
    }
    /* 3: RCMC, 4: azimuth filter */
    if (rc == OR_OK && stop_after >= 3) rc = rd_rows(n_az, n_rg, geo, 3, b, a, tab, nthreads);
    if (rc == OR_OK && stop_after >= 4) rc = rd_rows(n_az, n_rg, geo, 4, a, b, tab, nthreads);
    /* 5: azimuth inverse FFT */
    if (rc == OR_OK && stop_after >= 5) rc = oracle_fft(n_az, n_rg, n_rg, 1, +1, b, a, nthreads);
    if (rc == OR_OK) {
        const double *res = (stop_after == 2 || stop_after == 4) ? b : a;
        memcpy(out, res, sizeof(double) * 2 * n);
    }
    free(a);
    free(b);
    free(tab);
    return rc;
}
