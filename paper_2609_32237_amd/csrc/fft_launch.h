// fft_launch.h -- host-visible interface between the C ABI runtime and the
// kernel instantiations (one translation unit per transform size).
#pragma once

#include <hip/hip_runtime.h>

#include <tuple>
#include <utility>

namespace mi355fft {

// Launches a kernel and returns the status of this launch alone.  Reading
// hipGetLastError after a triple-chevron launch would also return (and clear)
// an earlier, unrelated error of the calling thread.  The arguments are
// converted to the kernel's parameter types and passed by address.
template <class... Params, class... Args, size_t... I>
hipError_t launch_kernel_impl(void (*kern)(Params...), dim3 grid, dim3 block, hipStream_t s,
                              std::index_sequence<I...>, Args &&...args) {
    std::tuple<Params...> vals(std::forward<Args>(args)...);
    void *ptrs[sizeof...(Params) > 0 ? sizeof...(Params) : 1] = {static_cast<void *>(&std::get<I>(vals))...};
    return hipLaunchKernel(reinterpret_cast<const void *>(kern), grid, block, ptrs, 0, s);
}

template <class... Params, class... Args>
hipError_t launch_kernel(void (*kern)(Params...), dim3 grid, dim3 block, hipStream_t s, Args &&...args) {
    static_assert(sizeof...(Params) == sizeof...(Args), "one argument per kernel parameter");
    return launch_kernel_impl(kern, grid, block, s, std::index_sequence_for<Params...>{},
                              std::forward<Args>(args)...);
}

// Kernel families: contiguous rows, strided column strips, and the
// migration-correction pass (row-mapped kernels over the transposed
// range-Doppler image that write columns of the focused image).
// The row kernels with the binary16 exchange (Section VII's FP16-exchange
// variant: half the LDS of the FP32 exchange in one round, about 6 dB less
// accurate) form a fourth family, for FP16 storage only.
enum { LAYOUT_ROWS = 0, LAYOUT_COLS = 1, LAYOUT_RCMC = 2, LAYOUT_ROWS_HALF = 3 };
// Per-kernel fusions around the transform:
//   EPI_NONE     the plain transform;
//   EPI_MATCHED  forward, X * conj(spec), inverse (range or azimuth
//                compression in one pass; spec carries the 1/N scale);
//   EPI_SCALE    forward, output * scale (the azimuth FFT with its 1/N_a),
//                column strips in, written as rows (out_stride 1);
//   EPI_RCMC     the load stage gathers, interpolates and phase-rotates the
//                transposed range-Doppler image (migration correction and
//                azimuth filter), the inverse transform runs, and the result
//                is written as columns; `spec` points to the range-Doppler
//                tables below.
//   EPI_MATCHED_Y  the middle pass of a matched filter along long columns in
//                four-step form: forward, X[k] * conj(spec[y + (k << spec_shift)]),
//                inverse, then output j times conj(W^(y j)) from tab2
//                (y = blockIdx.y);
//   EPI_TWIDDLE_Y  middle pass of a three-pass transform: plain column strips,
//                output point k of problem blockIdx.y times W^(blockIdx.y k)
//                (the same two-level tables as EPI_TWIDDLE);
//   EPI_TWIDDLE  first pass of a four-step transform of length N = N1 * N2:
//                the column FFT of length N1, point k1 of column n2 times
//                W_N^(n2 k1) (conjugate for the inverse), written as rows;
//                `spec` holds W_N^m for m < S followed by W_N^(S m) for
//                m < N / S, with S = 2^aux.
// Block -> strip maps of column kernels over the 8 XCDs (logical_block).
enum { XCD_NONE = 0, XCD_CONTIG = 1, XCD_GROUPS = 2, XCD_ROWS = 3 };
enum {
    EPI_NONE = 0,
    EPI_MATCHED = 1,
    EPI_SCALE = 2,
    EPI_RCMC = 3,
    EPI_TWIDDLE = 4,
    EPI_TWIDDLE_Y = 5,
    EPI_MATCHED_Y = 6
};

// Range-Doppler tables, one device block in this order (byte offsets from
// rd_tables_layout; the interpolator rows are copied in from `interp_src`):
//   rows   float4[n_az]  {(1/D_k - 1) / range_bin, 2 (D_k - 1) / lambda as a
//                         hi + lo pair of floats, 0}
//   cols   float2[n_rg]  {R0_n as a hi + lo pair}
//   interp float2[(kRcmcSub + 1) * kRcmcTaps]  {g_q[j], g_{q+1}[j] - g_q[j]}
constexpr int kRcmcSub = 128, kRcmcTaps = 8;
struct RdTablesLayout {
    long long rows, cols, interp, bytes;
};
__host__ __device__ constexpr long long round_up_256(long long x) { return (x + 255) & ~255LL; }
__host__ __device__ constexpr RdTablesLayout rd_tables_layout(long long n_az, long long n_rg) {
    return RdTablesLayout{0, round_up_256(n_az * 16), round_up_256(n_az * 16) + round_up_256(n_rg * 8),
                          round_up_256(n_az * 16) + round_up_256(n_rg * 8) +
                              round_up_256((long long)(kRcmcSub + 1) * kRcmcTaps * 8)};
}

// Twiddle tables.  The table of a length n holds W_n^m = exp(-2 pi i m / n)
// for m < n, followed by per-stage tables: for every radix R in
// {2, 4, 8, 16, 32} and every sub-transform length NS = 2, 4, ..., n / R, the
// factors a stage of radix R on sub-transforms of length NS applies,
// W_(NS R)^(k r), stored at [(r - 1) NS + k] for k < NS and 1 <= r < R.  A
// butterfly of that stage then reads its R - 1 factors from R - 1 rows of one
// stage table, and consecutive lanes (consecutive k) read consecutive entries.
constexpr int kStageRadices[5] = {2, 4, 8, 16, 32};
__host__ __device__ constexpr long long stage_table_entries(long long n, int r) {
    return n / r >= 2 ? (long long)(r - 1) * (2 * (n / r) - 2) : 0;
}
// Offset (in entries, from the start of the length-n table) of the stage table
// of radix r and sub-transform length ns (2 <= ns <= n / r).
__host__ __device__ constexpr long long stage_table_offset(long long n, int ns, int r) {
    long long off = n;
    for (int i = 0; i < 5 && kStageRadices[i] < r; ++i) off += stage_table_entries(n, kStageRadices[i]);
    return off + (long long)(r - 1) * (ns - 2);
}
__host__ __device__ constexpr long long twiddle_entries(long long n) {
    long long e = n;
    for (int i = 0; i < 5; ++i) e += stage_table_entries(n, kStageRadices[i]);
    return e;
}

// The allocation-free SAR entry point keeps its tables and workspace in one
// fixed device array per device (noalloc.hip), of kNoallocScratchBytes:
// room for the twiddle tables, both reference spectra and an intermediate
// image of at most kNoallocMaxImageBytes (the 4096 x 4096 image with FP32
// intermediates).  noalloc_scratch returns the current device's copy of it;
// the address is looked up once per device and kept.
constexpr size_t kNoallocMaxImageBytes = size_t(128) << 20;
constexpr size_t kNoallocScratchBytes = kNoallocMaxImageBytes + (size_t(3) << 20);
hipError_t noalloc_scratch(int device, void **ptr);

// Acquisition geometry the range-Doppler tables are computed from (metres,
// Hz, m/s); the tables are filled by the azimuth-FFT pass (rd_tables.hpp) in
// double precision and rounded once to FP32 or split into hi + lo pairs.
struct RdGeometry {
    double wavelength, speed, prf, range_bin, r_near;
};

struct KArgs {
    long long batch;       // transforms
    long long stride;      // elements between points of a transform in the input
    long long in_dist;     // elements between transform starts in the input
    long long out_dist;    // elements between transform starts in the output
    float scale;           // epilogue scale
    int xcd_remap;         // block -> strip map over the XCDs (XCD_NONE / XCD_CONTIG / XCD_GROUPS / XCD_ROWS)
    int wide;              // 1: 64-bit pointer addressing (span or sign does not fit buffer offsets)
    unsigned in_span;      // bytes one workgroup's input occupies (buffer addressing)
    unsigned out_span;     // bytes one workgroup's output occupies
    long long out_stride;  // elements between points of a transform in the output; 0: same as the input
    long long outer_in_dist;   // elements between the problems of blockIdx.y (input)
    long long outer_out_dist;  // elements between the problems of blockIdx.y (output)
    int outer;                 // problems along blockIdx.y (0 or 1: one)
    int outer2;                // problems along blockIdx.z (0 or 1: one), each outer2_dist
    long long outer2_dist;     // elements apart in both input and output
    int aux;                   // EPI_TWIDDLE(_Y): log2 of the low twiddle table's length
    // EPI_TWIDDLE with a row permutation: transform m of the batch is written
    // as row ((m mod 2^perm_b) << perm_a) | (m >> perm_b) (0, 0: row m)
    int perm_a, perm_b;
    // EPI_MATCHED_Y: the spectrum value of point k is spec[blockIdx.y +
    // (k << spec_shift)], and tab2 is the two-level table (log2 split aux) of
    // the outer transform's factors
    int spec_shift;
    const float2 *tab2;
    // EPI_SCALE: when rd_tables is set, thread g = blockIdx.x * THREADS +
    // threadIdx.x first writes entry g of the range-Doppler tables (n_az = the
    // transform length, n_rg = batch) from the geometry and interpolator rows
    RdGeometry rd_geo;
    const float2 *rd_interp;
    void *rd_tables;
    // EPI_MATCHED rows: the chain's reference spectra computed by the first
    // workgroups of the range pass instead of a launch of their own.
    // Reference row r < ref_rows (r = 0 the range reference, whose spectrum
    // is `spec`; r = 1 the azimuth reference) is ref_in[r] (FP32, N points,
    // contiguous), transformed forward, times ref_scale[r], stored to
    // ref_out[r] (FP32).  It belongs to thread (blk, c) with blk * C + c = r;
    // the image rows follow as blocks ref_blocks .. (set by the launcher).
    // Workgroup 0 then stores ref_epoch to *ref_flag (agent-scope release)
    // and each image workgroup waits for that value before it reads `spec`.
    int ref_rows;
    int ref_blocks;
    const float2 *ref_in[2];
    float2 *ref_out[2];
    float ref_scale[2];
    unsigned long long *ref_flag;
    unsigned long long ref_epoch;
    // Any kernel: workgroup 0 first stores 0 to *clear_flag (a pass that
    // runs after the one that waited on it, so no reader remains).
    unsigned long long *clear_flag;
};

// Fills the addressing fields of `a` for workgroups of `c` transforms of `n`
// points with elements of in_bytes / out_bytes.
inline void set_spans(KArgs &a, long long n, long long c, int in_bytes, int out_bytes) {
    const long long lim = 0x7fffffffLL;
    if (a.out_stride == 0) a.out_stride = a.stride;
    const long long cc = c < a.batch ? c : a.batch;
    const long long in_el = (cc - 1) * a.in_dist + (n - 1) * a.stride + 1;
    const long long out_el = (cc - 1) * a.out_dist + (n - 1) * a.out_stride + 1;
    const bool ok = a.in_dist >= 0 && a.out_dist >= 0 && a.stride >= 1 && a.out_stride >= 1 &&
                    in_el * in_bytes <= lim && out_el * out_bytes <= lim;
    a.wide = ok ? 0 : 1;
    a.in_span = ok ? (unsigned)(in_el * in_bytes) : 0u;
    a.out_span = ok ? (unsigned)(out_el * out_bytes) : 0u;
}

// Each returns the launch status (hipErrorInvalidValue for an unsupported
// combination of layout, storages, direction and epilogue, or a variant index
// out of range).  variant < 0 selects the size's default kernel shape.
#define MI355FFT_DECLARE_LAUNCH(N)                                                                       \
    hipError_t launch_fft_n##N(int variant, int layout, int in_st, int out_st, int inv, int epi,        \
                               const void *in, void *out, const float2 *tw, const float2 *spec,         \
                               const KArgs &a, hipStream_t s);                                           \
    int variants_n##N(int layout);
MI355FFT_DECLARE_LAUNCH(64)
MI355FFT_DECLARE_LAUNCH(128)
MI355FFT_DECLARE_LAUNCH(256)
MI355FFT_DECLARE_LAUNCH(512)
MI355FFT_DECLARE_LAUNCH(1024)
MI355FFT_DECLARE_LAUNCH(2048)
MI355FFT_DECLARE_LAUNCH(4096)
MI355FFT_DECLARE_LAUNCH(8192)
MI355FFT_DECLARE_LAUNCH(16384)
#undef MI355FFT_DECLARE_LAUNCH

// FP16-storage rows with the radix-16 butterflies on the matrix cores
// (fft_mfma.hpp): one transform per workgroup, stride 1.
// `amat` is the lane-fragment table of the 16-point DFT matrix (8 KiB, see
// fft_mfma.hpp).
hipError_t launch_fft_mfma_n4096(int inv, const void *in, void *out, const float2 *tw, const void *amat,
                                 const KArgs &a, hipStream_t s);
hipError_t launch_fft_mfma_n16384(int inv, const void *in, void *out, const float2 *tw, const void *amat,
                                  const KArgs &a, hipStream_t s);

}  // namespace mi355fft
