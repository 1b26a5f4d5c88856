// membench.hip -- memory-system ceilings of MI355X for the benchmark (Section
// IV: the paper measures streaming bandwidth against working-set size, and
// eq. (1) bounds an FFT pass by that bandwidth).
//
// Plain data movement only, no FFT arithmetic: it measures what the FFT
// kernels' access patterns can reach, so their throughput can be read against
// a ceiling measured on the same GPU rather than against the 8 TB/s datasheet
// figure alone.  Built into its own library (libmi355membench.so); the FFT
// library neither links nor calls it.
//
// Kinds (mb_run's `kind`):
//   MB_COPY       dst[i] = src[i], one 16-byte access per lane, `reps` passes
//                 over the buffer inside one launch (grid-stride, each pass's
//                 chunks shifted to another workgroup of the same XCD), so
//                 small working sets are timed out of the L2 or the Infinity
//                 Cache rather than as launch latency;
//   MB_READ       read src `reps` times; the sums feed a store to dst (1024
//                 floats) that a positive buffer never takes, so nothing is
//                 optimised away;
//   MB_WRITE      write dst `reps` times;
//   MB_BLOCK      the single-pass row FFT's pattern: a workgroup of `threads`
//                 lanes copies one block of `block` bytes, each lane loading
//                 block / (threads * 8) values of 8 bytes at stride threads * 8
//                 (all loads issued before the first store, as the kernel holds
//                 a whole transform), then storing them in the same pattern;
//                 `lds_kib` of LDS per workgroup sets the occupancy the FFT
//                 kernel has;
//   MB_STRIP      the column FFT's pattern on a 4096-row matrix of 8-byte
//                 elements with rows `width` elements long: a 1024-lane
//                 workgroup takes a strip of C adjacent columns (C * 8-byte
//                 pieces of every row), lanes t*C + c, 4096 / (1024 / C) rows
//                 per lane; `mode` 0 stores the strip back in the same strided
//                 layout, 1 stores it as a contiguous block (strided reads
//                 only), 2 reads a contiguous block and stores it strided
//                 (strided writes only).  Workgroups whose strips share a
//                 128-byte line run on one XCD (dispatch is round-robin over
//                 the 8 XCDs), as the FFT's column kernels arrange.
// flags: bit 0 non-temporal loads, bit 1 non-temporal stores (MB_COPY,
// MB_READ, MB_WRITE, MB_BLOCK); bit 2 (MB_COPY in one pass, MB_BLOCK): the
// workgroups in groups of about 1 MiB of consecutive data per XCD,
// successive groups on successive XCDs (the FFT row kernels' block order).
#include <hip/hip_runtime.h>

#include <tuple>
#include <utility>

namespace {

enum { MB_COPY = 0, MB_READ = 1, MB_WRITE = 2, MB_BLOCK = 3, MB_STRIP = 4 };

typedef float f32x4 __attribute__((ext_vector_type(4)));

template <bool NT>
__device__ __forceinline__ f32x4 ld4(const f32x4 *p) {
    if constexpr (NT) return __builtin_nontemporal_load(p);
    return *p;
}
template <bool NT>
__device__ __forceinline__ void st4(f32x4 *p, f32x4 v) {
    if constexpr (NT) {
        __builtin_nontemporal_store(v, p);
    } else {
        *p = v;
    }
}
template <bool NT>
__device__ __forceinline__ float2 ld2(const float2 *p) {
    if constexpr (NT) return __builtin_bit_cast(float2, __builtin_nontemporal_load(reinterpret_cast<const double *>(p)));
    return *p;
}
template <bool NT>
__device__ __forceinline__ void st2(float2 *p, float2 v) {
    if constexpr (NT) {
        __builtin_nontemporal_store(__builtin_bit_cast(double, v), reinterpret_cast<double *>(p));
    } else {
        *p = v;
    }
}

// The chunk a workgroup takes in pass r: its own shifted by 8 r workgroups, so
// that each pass reads data another workgroup of the same XCD touched before
// (dispatch is round-robin over the 8 XCDs): repeated passes over a small
// working set then measure that XCD's L2 (or the Infinity Cache, or HBM)
// rather than the CU's own L1.
__device__ __forceinline__ long long rotated(int r) { return ((long long)blockIdx.x + 8LL * r) % gridDim.x; }

// Block b in groups of G consecutive blocks per XCD, successive groups on
// successive XCDs; blocks past the last whole round of 8 groups keep their
// index.
__device__ __forceinline__ long long grouped(long long b, long long g, long long G) {
    const long long full = g / (8 * G) * (8 * G);
    if (b >= full) return b;
    const long long xcd = b & 7, local = b >> 3;
    return ((local / G) * 8 + xcd) * G + local % G;
}

template <bool NTL, bool NTS, bool GRP = false>
__global__ __launch_bounds__(256) void copy_kernel(const f32x4 *__restrict__ src, f32x4 *__restrict__ dst,
                                                   long long n4, int reps) {
    const long long stride = (long long)gridDim.x * 256;
    if constexpr (GRP) {  // one pass, one 16-byte access per lane; 4 KiB workgroups, 256 per group
        const long long i = grouped(blockIdx.x, gridDim.x, 256) * 256 + threadIdx.x;
        if (i < n4) st4<NTS>(dst + i, ld4<NTL>(src + i));
        return;
    }
    for (int r = 0; r < reps; ++r)
        for (long long i = rotated(r) * 256 + threadIdx.x; i < n4; i += stride) st4<NTS>(dst + i, ld4<NTL>(src + i));
}

template <bool NTL>
__global__ __launch_bounds__(256) void read_kernel(const f32x4 *__restrict__ src, float *__restrict__ sums,
                                                   long long n4, int reps) {
    const long long stride = (long long)gridDim.x * 256;
    f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int r = 0; r < reps; ++r)
        for (long long i = rotated(r) * 256 + threadIdx.x; i < n4; i += stride) acc += ld4<NTL>(src + i);
    // a store the loads feed but that never happens for the all-ones buffers
    // the benchmark reads (their sums are positive)
    if (acc.x + acc.y + acc.z + acc.w == -1.0f) sums[blockIdx.x & 1023] = 1.0f;
}

template <bool NTS>
__global__ __launch_bounds__(256) void write_kernel(f32x4 *__restrict__ dst, long long n4, int reps) {
    const long long stride = (long long)gridDim.x * 256;
    const f32x4 v = {1.0f, 2.0f, 3.0f, 4.0f};
    for (int r = 0; r < reps; ++r)
        for (long long i = rotated(r) * 256 + threadIdx.x; i < n4; i += stride) st4<NTS>(dst + i, v);
}

// One block of T * P 8-byte values per workgroup: lane t loads t + T*i.
template <int T, int P, bool NTL, bool NTS, bool GRP = false>
__global__ __launch_bounds__(T) void block_kernel(const float2 *__restrict__ src, float2 *__restrict__ dst) {
    extern __shared__ float lds_pad[];  // sized by the host only to set occupancy
    if (threadIdx.x == 0xffffffffu) lds_pad[0] = 0.0f;
    const long long b = GRP ? grouped(blockIdx.x, gridDim.x, (1 << 20) / (T * P * 8)) : (long long)blockIdx.x;
    const long long base = b * (T * P) + threadIdx.x;
    float2 v[P];
#pragma unroll
    for (int i = 0; i < P; ++i) v[i] = ld2<NTL>(src + base + T * i);
#pragma unroll
    for (int i = 0; i < P; ++i) st2<NTS>(dst + base + T * i, v[i]);
}

// Logical strip of block b: the GROUP strips of a 128-byte line on one XCD,
// successive groups on successive XCDs (grid a multiple of 8 * GROUP).
template <int GROUP>
__device__ __forceinline__ long long strip_of(long long b, long long g) {
    if (g % (8 * GROUP) != 0) return b;
    const long long xcd = b & 7, local = b >> 3;
    return ((local / GROUP) * 8 + xcd) * GROUP + local % GROUP;
}

template <int C, int MODE>
__global__ __launch_bounds__(1024) void strip_kernel(const float2 *__restrict__ src, float2 *__restrict__ dst,
                                                     long long width) {
    constexpr int T = 1024 / C, ROWS = 4096, P = ROWS / T, GROUP = 16 / C > 1 ? 16 / C : 1;
    const long long s = strip_of<GROUP>(blockIdx.x, gridDim.x);
    const int c = threadIdx.x % C, t = threadIdx.x / C;
    float2 v[P];
#pragma unroll
    for (int i = 0; i < P; ++i) {
        const long long row = t + (long long)T * i;
        v[i] = MODE == 2 ? src[s * (ROWS * C) + row * C + c] : src[row * width + s * C + c];
    }
#pragma unroll
    for (int i = 0; i < P; ++i) {
        const long long row = t + (long long)T * i;
        if (MODE == 1) {
            dst[s * (ROWS * C) + row * C + c] = v[i];
        } else {
            dst[row * width + s * C + c] = v[i];
        }
    }
}

template <class... Params, class... Args, size_t... I>
hipError_t launch_impl(void (*kern)(Params...), dim3 grid, dim3 block, size_t lds, hipStream_t s,
                       std::index_sequence<I...>, Args &&...args) {
    std::tuple<Params...> vals(std::forward<Args>(args)...);
    void *ptrs[] = {static_cast<void *>(&std::get<I>(vals))...};
    return hipLaunchKernel(reinterpret_cast<const void *>(kern), grid, block, ptrs, lds, s);
}

template <class... Params, class... Args>
hipError_t launch(void (*kern)(Params...), dim3 grid, dim3 block, size_t lds, hipStream_t s, Args &&...args) {
    return launch_impl(kern, grid, block, lds, s, std::index_sequence_for<Params...>{}, std::forward<Args>(args)...);
}

template <int T, int P>
hipError_t run_block(int flags, const void *src, void *dst, long long bytes, int lds_kib, hipStream_t s) {
    const long long blk = (long long)T * P * 8;
    if (bytes % blk != 0 || bytes / blk > 0x7fffffffLL) return hipErrorInvalidValue;
    const dim3 grid((unsigned)(bytes / blk)), block(T);
    const size_t lds = (size_t)lds_kib * 1024;
    const float2 *in = static_cast<const float2 *>(src);
    float2 *out = static_cast<float2 *>(dst);
    switch (flags & 7) {
        case 0: return launch(block_kernel<T, P, false, false>, grid, block, lds, s, in, out);
        case 1: return launch(block_kernel<T, P, true, false>, grid, block, lds, s, in, out);
        case 2: return launch(block_kernel<T, P, false, true>, grid, block, lds, s, in, out);
        case 3: return launch(block_kernel<T, P, true, true>, grid, block, lds, s, in, out);
        case 4: return launch(block_kernel<T, P, false, false, true>, grid, block, lds, s, in, out);
        case 5: return launch(block_kernel<T, P, true, false, true>, grid, block, lds, s, in, out);
        case 6: return launch(block_kernel<T, P, false, true, true>, grid, block, lds, s, in, out);
        default: return launch(block_kernel<T, P, true, true, true>, grid, block, lds, s, in, out);
    }
}

template <int C>
hipError_t run_strip(int mode, const void *src, void *dst, long long bytes, long long width, hipStream_t s) {
    if (width <= 0 || width % C != 0 || bytes != 4096LL * width * 8) return hipErrorInvalidValue;
    const dim3 grid((unsigned)(width / C)), block(1024);
    const float2 *in = static_cast<const float2 *>(src);
    float2 *out = static_cast<float2 *>(dst);
    switch (mode) {
        case 0: return launch(strip_kernel<C, 0>, grid, block, 0, s, in, out, width);
        case 1: return launch(strip_kernel<C, 1>, grid, block, 0, s, in, out, width);
        case 2: return launch(strip_kernel<C, 2>, grid, block, 0, s, in, out, width);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

extern "C" {

// Runs one measurement kernel on `stream`.
//   kind    MB_COPY, MB_READ, MB_WRITE, MB_BLOCK or MB_STRIP (above).
//   src     device buffer of `bytes` (unused by MB_WRITE).
//   dst     device buffer of `bytes` (MB_READ: 1024 floats).
//   bytes   working set; a multiple of 16 (MB_COPY/READ/WRITE), of the
//           block (MB_BLOCK), or 4096 * width * 8 (MB_STRIP).
//   a       MB_COPY/READ/WRITE: passes over the buffer (>= 1); MB_BLOCK:
//           points per lane, 8 or 16 (with 256 lanes: 16 or 32 KiB blocks);
//           MB_STRIP: row length `width` in elements.
//   b       MB_COPY/READ/WRITE: workgroups (0: one 16-byte access per lane,
//           bytes / 4096 workgroups); MB_BLOCK: LDS
//           KiB per workgroup; MB_STRIP: strip width C (4, 8 or 16).
//   flags   MB_COPY/READ/WRITE/BLOCK: bit 0 non-temporal loads, bit 1
//           non-temporal stores; MB_STRIP: the mode 0, 1 or 2.
// Returns 0 on success, else the HIP error code of the launch (an invalid
// combination gives hipErrorInvalidValue before any launch).
int mb_run(int kind, const void *src, void *dst, long long bytes, long long a, long long b, int flags,
           hipStream_t stream) {
    if (bytes <= 0) return (int)hipErrorInvalidValue;
    if (kind == MB_COPY || kind == MB_READ || kind == MB_WRITE) {
        if (bytes % 16 != 0 || a < 1 || a > (1 << 20) || b < 0 || b > (1 << 20)) return (int)hipErrorInvalidValue;
        const long long n4 = bytes / 16;
        // default: one 16-byte access per lane per pass over the whole grid
        long long blocks = b > 0 ? b : (n4 + 255) / 256;
        if (blocks * 256 > n4) blocks = (n4 + 255) / 256;
        if (blocks > 0x7fffffffLL) return (int)hipErrorInvalidValue;
        const dim3 grid((unsigned)blocks), block(256);
        const f32x4 *in = static_cast<const f32x4 *>(src);
        f32x4 *out = static_cast<f32x4 *>(dst);
        const int reps = (int)a;
        if (kind == MB_COPY) {
            if ((flags & 4) && (reps != 1 || blocks * 256 < n4)) return (int)hipErrorInvalidValue;
            switch (flags & 7) {
                case 0: return (int)launch(copy_kernel<false, false>, grid, block, 0, stream, in, out, n4, reps);
                case 1: return (int)launch(copy_kernel<true, false>, grid, block, 0, stream, in, out, n4, reps);
                case 2: return (int)launch(copy_kernel<false, true>, grid, block, 0, stream, in, out, n4, reps);
                case 3: return (int)launch(copy_kernel<true, true>, grid, block, 0, stream, in, out, n4, reps);
                case 4: return (int)launch(copy_kernel<false, false, true>, grid, block, 0, stream, in, out, n4, reps);
                case 5: return (int)launch(copy_kernel<true, false, true>, grid, block, 0, stream, in, out, n4, reps);
                case 6: return (int)launch(copy_kernel<false, true, true>, grid, block, 0, stream, in, out, n4, reps);
                default: return (int)launch(copy_kernel<true, true, true>, grid, block, 0, stream, in, out, n4, reps);
            }
        }
        if (kind == MB_READ) {
            float *sums = static_cast<float *>(dst);
            return (int)((flags & 1) ? launch(read_kernel<true>, grid, block, 0, stream, in, sums, n4, reps)
                                     : launch(read_kernel<false>, grid, block, 0, stream, in, sums, n4, reps));
        }
        return (int)((flags & 2) ? launch(write_kernel<true>, grid, block, 0, stream, out, n4, reps)
                                 : launch(write_kernel<false>, grid, block, 0, stream, out, n4, reps));
    }
    if (kind == MB_BLOCK) {
        if (b < 0 || b > 160) return (int)hipErrorInvalidValue;
        if (a == 16) return (int)run_block<256, 16>(flags, src, dst, bytes, (int)b, stream);
        if (a == 8) return (int)run_block<256, 8>(flags, src, dst, bytes, (int)b, stream);
        return (int)hipErrorInvalidValue;
    }
    if (kind == MB_STRIP) {
        if (b == 4) return (int)run_strip<4>(flags, src, dst, bytes, a, stream);
        if (b == 8) return (int)run_strip<8>(flags, src, dst, bytes, a, stream);
        if (b == 16) return (int)run_strip<16>(flags, src, dst, bytes, a, stream);
        return (int)hipErrorInvalidValue;
    }
    return (int)hipErrorInvalidValue;
}

}  // extern "C"
