/*
 * mi355fft.h -- C ABI of the MI355X (gfx950) batched FFT and SAR library.
 *
 * The operations follow "Bandwidth, Not FLOPS: FFT Kernels, Matrix Units and
 * SAR Imaging on Apple M6" (arXiv 2609.32237):
 *   - batched complex-to-complex 1-D FFTs, each transform read once from and
 *     written once to device memory (Section IV, eq. (1); Section VI), with
 *     FP32 or FP16 storage and FP32 arithmetic (Section VII);
 *   - the range-Doppler SAR image of a pulses x range-samples echo: range
 *     compression (FFT, matched filter, inverse FFT, 1/N_r) fused in one pass,
 *     then the azimuth FFT read straight from the columns with its 1/N_a
 *     scale, the azimuth matched filter and the azimuth inverse FFT fused in a
 *     second pass (Section X);
 *   - the paper's full range-Doppler chain with range-cell migration
 *     correction and the baseband azimuth filter (Section X): range
 *     compression, the azimuth FFT, and one fused pass that interpolates,
 *     filters and inverse-transforms each range bin.
 *
 * Conventions shared by every entry point
 *   - Complex values are interleaved (re, im): FP32 storage is two floats
 *     (8 bytes) per value, FP16 storage two IEEE binary16 halves (4 bytes).
 *   - Sizes, strides and distances count complex elements, not bytes.
 *   - Every pointer argument named in/out/raw/ref/workspace is a DEVICE
 *     pointer on the current HIP device; the caller owns it.
 *   - Every call is stream-ordered on the given hipStream_t (0 = the null
 *     stream) and never synchronises.  Argument errors are returned before
 *     any HIP call is made.  A failed launch returns FFT_EHIP; the status is
 *     that of the library's own launch, read from the launch call itself, so
 *     an earlier error the caller left pending is neither reported nor
 *     cleared.  Faults inside a kernel surface at the caller's next
 *     synchronisation.
 *   - Transforms are unnormalised in both directions: forward computes
 *     X[k] = sum_n x[n] exp(-2 pi i n k / N), inverse uses exp(+2 pi i n k / N).
 *     Output is in natural order.
 */
#ifndef MI355FFT_H
#define MI355FFT_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Storage formats (Section VII: FP16 storage halves the bytes per point while
 * the arithmetic stays FP32). */
enum { FFT_STORAGE_FP32 = 0, FFT_STORAGE_FP16 = 1 };

/* Direction = sign of the exponent. */
enum { FFT_FORWARD = -1, FFT_INVERSE = +1 };

/* Return codes. */
enum {
    FFT_OK = 0,
    FFT_EINVAL = -1,       /* invalid argument (NULL, bad enum, overlapping layout) */
    FFT_EUNSUPPORTED = -2, /* valid request this library does not implement (size) */
    FFT_ENOMEM = -3,       /* device or host allocation failed */
    FFT_EALIGN = -4,       /* a pointer is not aligned to one complex element */
    FFT_EHIP = -5          /* the HIP runtime reported an error (or another host-side
                              failure inside the library: no C++ exception crosses
                              this interface) */
};

typedef struct fft_plan fft_plan; /* opaque; immutable once created */

/*
 * fft_plan_create -- plan a batch of `batch` transforms of `n` points.
 *
 * Section III states the problem as B transforms of N points in FP32 (the
 * batch's footprint is its input plus its output); Section VII adds FP16
 * storage.
 *
 *   n        transform length: a power of two in [1024, 2^28], else
 *            FFT_EUNSUPPORTED.  Up to 16384 every transform is one pass
 *            (read once, written once).  Longer transforms use the two-pass
 *            four-step form (Section VI: the transform no longer fits on
 *            chip): n = n1 * n2 with n2 = 2^floor(log2(n) / 2); beyond 2^22
 *            a third pass splits n2 again (n = n1 * na * nb, no factor above
 *            1024, so that every pass reads and writes wide pieces of each
 *            row).  They require stride == 1 (else FFT_EUNSUPPORTED) and
 *            out-of-place execution, and use `out` for the intermediate; the
 *            input is not modified.  Batches of at most 16
 *            contiguous 16384-point transforms executed out of place take the
 *            same split (128 x 128) to spread each transform over more
 *            workgroups (Section VI's advice for small batches); in place
 *            they stay single-pass.
 *   batch    number of transforms, >= 1.
 *   stride   distance between consecutive points of one transform, >= 1.
 *   dist     distance between the first points of consecutive transforms, >= 1.
 *            Point j of transform b is at element b*dist + j*stride of both
 *            the input and the output buffer.
 *            The transforms must not overlap: either they sit in disjoint
 *            blocks (dist >= (n-1)*stride + 1) or they interleave
 *            (stride >= (batch-1)*dist + 1), else FFT_EINVAL.
 *            stride == 1 selects the contiguous-row kernels; stride > 1 the
 *            strided-column kernels (columns of a row-major matrix are
 *            stride = row length, dist = 1).  Columns of 8192 or 16384
 *            points with dist == 1 executed out of place run as two passes
 *            of 128 x 64 or 128 x 128 points (the four-step form along the
 *            columns), using `out` for the intermediate; in place they stay
 *            single-pass.
 *   storage  FFT_STORAGE_FP32 or FFT_STORAGE_FP16 (input and output alike).
 *   dir      FFT_FORWARD or FFT_INVERSE.
 *   plan_out receives the plan; untouched on error.
 *
 * Creates (once per device and size, shared by all plans, kept until the
 * process ends) a device table of the n twiddle factors exp(-2 pi i m / n),
 * computed in double precision on the host and rounded once to FP32; for
 * four-step lengths, the tables of n1 and n2 (n1, na and nb) and two-level
 * tables of the factors exp(-2 pi i m / n) (and, with three passes, of
 * exp(-2 pi i m / (na nb))), each about 2 sqrt(n) entries, W^m formed as the
 * product of two entries.  Uses the current HIP device; the plan must be
 * executed on that device.
 * Returns FFT_OK, FFT_EINVAL, FFT_EUNSUPPORTED, FFT_ENOMEM or FFT_EHIP.
 */
int fft_plan_create(int64_t n, int64_t batch, int64_t stride, int64_t dist, int storage, int dir,
                    fft_plan **plan_out);

/* Plan flags of fft_plan_create_ex. */
enum { FFT_FLAG_FP16_EXCHANGE = 1, FFT_FLAG_MATRIX_UNITS = 2 };

/*
 * fft_plan_create_ex -- fft_plan_create with a fixed-shift output scale and
 * options (Section VII: FFT outputs grow up to N for coherent data, so FP16
 * storage of real signals needs block-floating-point scaling; Section X
 * applies it as fixed power-of-two shifts).
 *
 *   scale_log2  the outputs are multiplied by 2^-scale_log2, in [0, 60], else
 *               FFT_EINVAL.  The product is exact in FP32 (no rounding), so
 *               the caller keeps the block exponent: scale_log2 = log2(n)
 *               bounds every output of a forward transform by the largest
 *               input magnitude, whatever the data.  0 is fft_plan_create.
 *               The split forms (four-step, long columns, small batches)
 *               apply 2^-min(s, log2 n1) in their first pass, and with three
 *               passes 2^-min(rest, log2 na) in the second, the rest in the
 *               last, so that no intermediate stored in `out` grows past the
 *               bound of the final outputs; each factor is exact, so the
 *               results are those of one final scale.
 *   flags       0, or FFT_FLAG_FP16_EXCHANGE: the exchange between stages is
 *               stored as binary16 pairs instead of FP32 (Section VII's
 *               FP16-exchange variant: half the on-chip traffic of the FP32
 *               exchange in one round, about 6 dB less accurate).  Requires
 *               FFT_STORAGE_FP16 (else FFT_EINVAL), stride == 1 and
 *               n <= 16384 (else FFT_EUNSUPPORTED).
 *               FFT_FLAG_MATRIX_UNITS: the radix-16 butterflies run on the
 *               matrix cores (Section VIII: each radix-16 stage as the 32 x 32
 *               real DFT matrix times the data, in binary16 with FP32
 *               accumulation; the twiddles in FP32 between stages).  The data
 *               are rounded to binary16 once per stage (the paper's matrix
 *               kernel measured 66 dB).  Requires FFT_STORAGE_FP16 (else
 *               FFT_EINVAL), stride == 1, n = 4096 or 16384 and scale_log2 = 0
 *               (else FFT_EUNSUPPORTED); exclusive with the FP16 exchange.
 *               Slower than the default kernels on MI355X (1.2x the time at
 *               n = 4096, 1.7x at 16384, from HBM): an experiment, opt-in.
 *               Unknown flags give FFT_EINVAL.
 * Other arguments, tables and errors as fft_plan_create.
 */
int fft_plan_create_ex(int64_t n, int64_t batch, int64_t stride, int64_t dist, int storage, int dir,
                       int scale_log2, unsigned flags, fft_plan **plan_out);

/*
 * fft_execute -- run the planned transforms: out = FFT(in).
 *
 * Every transform is read from `in` once and written to `out` once (Section
 * VI: the whole transform stays on chip between its stages).
 *   in, out  device buffers laid out as the plan says; in == out (in place) is
 *            allowed for n <= 16384 (FFT_EINVAL for longer transforms).
 *            Otherwise the two extents, (batch-1)*dist + (n-1)*stride + 1
 *            elements from each pointer, must be disjoint, else FFT_EINVAL.
 *            Aligned to one complex element (8 bytes FP32, 4 bytes FP16),
 *            else FFT_EALIGN.
 *   stream   HIP stream the kernel is launched on.
 * The current HIP device must be the one the plan was created on (its tables
 * live there), else FFT_EINVAL.
 * Safe to call concurrently on different streams with the same plan.
 * Returns FFT_OK, FFT_EINVAL (NULL plan or buffer, overlapping extents, other
 * device), FFT_EALIGN or FFT_EHIP (the status of the launch itself: an
 * earlier, unrelated HIP error of the calling thread is neither returned nor
 * cleared).
 */
int fft_execute(const fft_plan *plan, const void *in, void *out, hipStream_t stream);

/* fft_plan_destroy -- release a plan (host memory only).  NULL is a no-op.
 * The caller must not destroy a plan while a call using it is being made. */
int fft_plan_destroy(fft_plan *plan);

/*
 * sar_workspace_bytes -- device workspace sar_form_image_ex needs.
 * Holds both reference spectra, a 256-byte slot for the flag with which the
 * range pass publishes the range spectrum to its own workgroups, and the
 * range-compressed intermediate image (n_az * n_rg * 8 bytes for FP32, * 4
 * bytes for FP16 intermediates).
 * Returns 0 for an invalid or unsupported request.
 */
size_t sar_workspace_bytes(int64_t n_az, int64_t n_rg, int inter_storage);

/*
 * sar_form_image_ex -- range-Doppler image of an n_az x n_rg echo (Section X).
 *
 *   n_az, n_rg      pulses (rows) and range samples (columns); each a power of
 *                   two in [1024, 16384], else FFT_EUNSUPPORTED.
 *   inter_storage   FFT_STORAGE_FP32 or FFT_STORAGE_FP16 for the one stored
 *                   intermediate (Section X: FP16 intermediates with the
 *                   fixed-shift scaling 1/N_r in range compression and 1/N_a on
 *                   the azimuth FFT output).
 *   raw             n_az x n_rg complex FP32, row-major, rows = pulses.
 *   range_ref       n_rg complex FP32: the time-domain range reference (the
 *                   transmitted chirp, centred and wrapped to index t mod n_rg).
 *   az_ref          n_az complex FP32: the time-domain azimuth reference.
 *                   Neither reference may overlap the workspace (FFT_EINVAL).
 *   out             n_az x n_rg complex FP32 focused image; must not overlap
 *                   raw or the workspace.
 *   workspace       sar_workspace_bytes(n_az, n_rg, inter_storage) bytes,
 *                   256-byte aligned; contents on entry are ignored.
 *   stream          HIP stream; two kernels are launched on it in order when
 *                   n_az == n_rg: the range pass, whose first workgroups
 *                   compute both reference spectra, and the azimuth pass.
 *                   Otherwise the azimuth reference spectrum takes a launch
 *                   of its own first (three).  For n_az of 8192 or 16384
 *                   with FP32 intermediates the azimuth pass runs as three
 *                   passes of short columns after a launch of both spectra
 *                   (five; `out` then also holds the range-compressed image
 *                   between the passes).
 *
 * Computes, with H_r = FFT(range_ref) and H_a = FFT(az_ref):
 *   y[a, :]   = IFFT( FFT(raw[a, :]) * conj(H_r) ) / n_rg      (pass 1, rows)
 *   out[:, r] = IFFT( FFT(y[:, r]) / n_az * conj(H_a) )        (pass 2, columns)
 * i.e. the 2-D circular cross-correlation of raw with az_ref x range_ref.
 * Returns FFT_OK, FFT_EINVAL, FFT_EUNSUPPORTED, FFT_EALIGN, FFT_ENOMEM or
 * FFT_EHIP.
 */
int sar_form_image_ex(int64_t n_az, int64_t n_rg, int inter_storage, const void *raw,
                      const void *range_ref, const void *az_ref, void *out, void *workspace,
                      hipStream_t stream);

/*
 * sar_form_image -- the 4096 x 4096 image with FP32 intermediates (Section X
 * scene size).  Same as sar_form_image_ex(4096, 4096, FFT_STORAGE_FP32, ...)
 * with a workspace the library allocates on the first call on each device and
 * keeps until the process ends.  Calls that overlap on one device (from
 * several threads or streams) share that workspace and race.
 */
int sar_form_image(const void *raw, const void *range_ref, const void *az_ref, void *out,
                   hipStream_t stream);

/*
 * sar_form_image_noalloc -- sar_form_image_ex without a workspace argument,
 * for callers that cannot allocate device memory: code under HIP graph
 * capture (after the first call on the device), tight serving loops,
 * harnesses that forbid hipMalloc.
 *
 * The workspace (both reference spectra and the intermediate image) and the
 * twiddle tables live in one fixed device array of the library, 129 MiB on
 * each device, held from the loading of the library's device code until the
 * process ends; no call allocates or frees device memory.  The intermediate
 * must fit it: n_az * n_rg * (8 with FP32, 4 with FP16 intermediates) at most
 * 128 MiB (4096 x 4096 with FP32 intermediates, 8192 x 4096 with FP16), else
 * FFT_EUNSUPPORTED, returned before any HIP call.  The first call on a device
 * looks up the array's address there and copies the tables in with a
 * synchronous hipMemcpy (so it must not be made under stream capture); later
 * calls only launch kernels on `stream`.
 * Every call on one device uses that device's one array: calls that overlap in
 * time on one device (from several threads or streams) race.  The array keeps
 * the last call's contents; nothing in it needs to start at zero, since each
 * call writes every part of it that it reads.
 * Other arguments, the computation and the other errors are those of
 * sar_form_image_ex.
 */
int sar_form_image_noalloc(int64_t n_az, int64_t n_rg, int inter_storage, const void *raw,
                           const void *range_ref, const void *az_ref, void *out, hipStream_t stream);

/*
 * Acquisition geometry of a broadside stripmap echo (Section X's scene: an
 * L-band platform flying straight at constant speed, zero squint).
 */
typedef struct sar_geometry {
    double wavelength; /* carrier wavelength lambda [m], > 0 */
    double speed;      /* platform speed v [m/s], > 0 */
    double prf;        /* pulse repetition frequency [Hz], > 0 */
    double range_bin;  /* slant-range spacing of the range samples, c / (2 fs) [m], > 0 */
    double r_near;     /* slant range of range sample 0 [m], > 0 */
} sar_geometry;

/*
 * sar_rd_workspace_bytes -- device workspace sar_rd_form_image needs: the
 * range reference spectrum, a 256-byte flag slot (as in sar_workspace_bytes),
 * the per-Doppler-bin and per-range-bin tables of
 * the migration correction and azimuth filter, the interpolator table and
 * one intermediate image (the range-Doppler image, stored one row per range
 * bin: n_az * n_rg * 8 bytes for FP32, * 4 for FP16), each part 256-byte
 * aligned.  Returns 0 for an invalid or unsupported request.
 */
size_t sar_rd_workspace_bytes(int64_t n_az, int64_t n_rg, int inter_storage);

/*
 * sar_rd_form_image -- focused image of a stripmap echo by the full
 * range-Doppler algorithm of Section X, in three passes over device memory.
 *
 *   n_az, n_rg      pulses (rows) and range samples (columns); each a power of
 *                   two in [1024, 16384] with n_az * n_rg <= 2^27, else
 *                   FFT_EUNSUPPORTED.
 *   inter_storage   FFT_STORAGE_FP32 or FFT_STORAGE_FP16 for the stored
 *                   intermediate (Section X: FP16 with the fixed-shift
 *                   scaling 1/N_r in range compression and 1/N_a on the
 *                   azimuth FFT output).
 *   geo             host pointer to the acquisition geometry; every field
 *                   finite and > 0, and lambda * prf / (4 v) < 1 (the largest
 *                   Doppler frequency, prf / 2, has a real D), else
 *                   FFT_EINVAL.  lambda * prf / (4 v) must also be at most
 *                   1/3, else FFT_EUNSUPPORTED: the migration-correction pass
 *                   shares one window of rows across strips of up to 16
 *                   range bins, whose shifts must then differ by less than a
 *                   bin (the scene of Section X has 0.15).  Read before the
 *                   call returns.
 *   raw             n_az x n_rg complex FP32 echo, row-major, rows = pulses.
 *   range_ref       n_rg complex FP32: the transmitted pulse replica,
 *                   starting at index 0 (zero beyond the pulse); must not
 *                   overlap `out` or the workspace (FFT_EINVAL).
 *   out             n_az x n_rg complex FP32 focused image (rows = pulses,
 *                   columns = range bins); must not overlap raw or the
 *                   workspace.  Also holds the range-compressed image between
 *                   the first two passes.
 *   workspace       sar_rd_workspace_bytes(n_az, n_rg, inter_storage) bytes,
 *                   256-byte aligned; contents on entry are ignored.
 *   stream          HIP stream; three kernels run on it in order: the range
 *                   pass (its workgroup 0 computes the reference spectrum),
 *                   the azimuth FFT (which also fills the migration tables)
 *                   and the migration-correction pass.
 *
 * Computes, in Section X's order:
 *   1. y[a, :] = IFFT( FFT(raw[a, :]) * conj(FFT(range_ref)) ) / n_rg;
 *   2. Z[:, n] = FFT(y[:, n]) / n_az  (Doppler bin k has frequency
 *      f_k = k prf / n_az, minus prf for k >= n_az / 2);
 *   3. range-cell migration correction: with D_k = sqrt(1 - (lambda f_k /
 *      2v)^2), R0_n = r_near + n range_bin and dn = R0_n (1/D_k - 1) /
 *      range_bin, s = floor(dn), mu = dn - s:
 *        Zr[k, n] = sum_{j=0..7} g_j(mu) Z[k, n + s + j - 3]
 *      (samples outside [0, n_rg) count as zero), where g(mu) blends
 *      linearly between the two nearest of 129 rows of an 8-tap
 *      Kaiser-windowed (beta 2.5) sinc table at mu = q / 128, each row
 *      normalised to unit sum;
 *   4. the baseband azimuth filter Zr[k, n] *= exp(+j 4 pi R0_n (D_k - 1) /
 *      lambda), its phase evaluated in cycles;
 *   5. out[:, n] = IFFT(Zr[:, n])  (unnormalised).
 * Returns FFT_OK, FFT_EINVAL, FFT_EUNSUPPORTED, FFT_EALIGN, FFT_ENOMEM or
 * FFT_EHIP.
 */
int sar_rd_form_image(int64_t n_az, int64_t n_rg, int inter_storage, const sar_geometry *geo,
                      const void *raw, const void *range_ref, void *out, void *workspace,
                      hipStream_t stream);

/* fft_strerror -- static description of a return code (never NULL). */
const char *fft_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* MI355FFT_H */
