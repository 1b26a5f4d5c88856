// fft_kernel.hpp -- the single-pass batched FFT kernel template for gfx950.
//
// A workgroup owns C whole transforms of N points.  Each thread loads P
// points of one transform from HBM exactly once (Section IV, eq. (1): one
// read and one write per point is the whole traffic of a single-pass FFT),
// runs every radix stage in VGPRs with LDS exchanges between stages
// (Section VI: registers plus local memory hold the transform, so 8192 and
// 16384 points need no second pass; gfx950's 160 KiB of LDS per CU replaces
// the 32 KiB buffer the paper worked around), and stores each point once.
//
// Two thread-to-data maps:
//   rows (COLS = false): contiguous transforms (stride 1); thread id =
//     c*T + t, so consecutive lanes read consecutive points.
//   columns (COLS = true): strided transforms whose starts are adjacent in
//     memory (dist 1); thread id = t*C + c, so consecutive lanes read the C
//     neighbouring columns of one row and each row access is a contiguous
//     C-element segment (Section X: reading the columns directly instead of
//     transposing; Section IX's "columns side by side" idea on the CPU).
//
// Variants (all compute the same transform; tests force each one):
//   XCHG   FULL: complex exchange through LDS (N*8 bytes per transform);
//          SPLIT: one real component at a time (N*4 bytes, twice the rounds;
//          the paper's Section VI exchange, here used to double occupancy).
//   TWMODE 0: every inter-stage twiddle read from the table;
//          1: one table read per base-4 digit of the radix, the rest formed
//          by complex products (fewer loads, a few more FP32 operations).
//   PERSIST the workgroup loops over its share of the batch and loads the
//          next transform into a second register array while it computes the
//          current one (the second-array idea of Section VI, used here to
//          overlap HBM latency with arithmetic).
// Twiddles for stage s+1 are requested before stage s's LDS exchange, so
// their latency hides behind the exchange.
//
// Optional fused epilogue (Section X, range compression in one kernel):
// after the forward stages, X[k] <- X[k] * conj(H[k]) * scale, then the
// inverse stages run on the same registers with no trip to memory.
#pragma once

#include <atomic>

#include "fft_device.hpp"
#include "fft_launch.h"

namespace mi355fft {

enum { XCHG_FULL = 0, XCHG_SPLIT = 1 };


template <int... Rs>
struct Radices {};

template <class Rad>
struct RadProd;
template <>
struct RadProd<Radices<>> {
    static constexpr int value = 1;
};
template <int R, int... Rs>
struct RadProd<Radices<R, Rs...>> {
    static constexpr int value = R * RadProd<Radices<Rs...>>::value;
};

template <int N_, int P_, int C_, bool COLS_, int XCHG_, int TWMODE_, bool PERSIST_, class Rad_, bool NTROW_ = true>
struct KCfg {
    static constexpr int N = N_, P = P_, T = N_ / P_, C = C_, THREADS = T * C;
    // rows of the plain transform are stored with the non-temporal hint
    static constexpr bool NTROW = NTROW_;
    static constexpr int LOG_T = ilog2(T), LOG_C = ilog2(C);
    static constexpr bool COLS = COLS_, PERSIST = PERSIST_;
    static constexpr int XCHG = XCHG_, TWMODE = TWMODE_;
    // LDS padding: one spare slot every 16 (8-byte exchange) or 32 (4-byte
    // exchange) elements spreads power-of-two strides over the banks.
    static constexpr int PADSH = XCHG_ == XCHG_FULL ? 4 : 5;
    static constexpr int ROW_SPAN = N_ + (N_ >> PADSH);
    static constexpr int SPAN = COLS_ ? (N_ * C_ + ((N_ * C_) >> PADSH)) : C_ * ROW_SPAN;
    static constexpr int LDS_FLOATS = XCHG_ == XCHG_FULL ? 2 * SPAN : SPAN;
    // Waves per SIMD the LDS allows (a CU has 4 SIMDs and 160 KiB of LDS),
    // capped at 4: asking the compiler for this occupancy keeps it from
    // spending registers the LDS limit would not let other waves use anyway,
    // while leaving every wave at least 128 VGPRs.
    static constexpr int WG_PER_CU_LDS = (160 * 1024) / (LDS_FLOATS * 4);
    static constexpr int WAVES_PER_SIMD = (WG_PER_CU_LDS * THREADS) / 256;
    static constexpr int MIN_WAVES = WAVES_PER_SIMD < 1 ? 1 : (WAVES_PER_SIMD > 4 ? 4 : WAVES_PER_SIMD);
    using Rad = Rad_;
    static_assert(RadProd<Rad_>::value == N_, "radices must multiply to N");
    static_assert((N_ & (N_ - 1)) == 0 && (P_ & (P_ - 1)) == 0 && (C_ & (C_ - 1)) == 0, "powers of two");
    static_assert(THREADS <= 1024, "at most 1024 threads per workgroup");
    static_assert(LDS_FLOATS * 4 <= 160 * 1024, "gfx950 LDS is 160 KiB per workgroup");
};

template <class... Ks>
struct KList {};

// LDS slot of (position, transform c): one spare slot after every 2^PADSH
// elements, pad(x) = x + (x >> PADSH); rows keep one padded span per
// transform, columns interleave the C transforms of the strip.
constexpr int pad_slots(int x, int s) { return x + (x >> s); }

template <class K>
__device__ __forceinline__ int lds_index(int pos, int c) {
    if constexpr (K::COLS) {
        return pad_slots((pos << K::LOG_C) + c, K::PADSH);
    } else {
        return c * K::ROW_SPAN + pad_slots(pos, K::PADSH);
    }
}

// Output position of element r of butterfly j in a stage of radix R whose
// sub-transforms so far have length NS (Stockham autosort).
template <int NS, int R>
__device__ __forceinline__ int out_pos(int j, int r) {
    constexpr int LNS = ilog2(NS), LR = ilog2(R);
    return ((j >> LNS) << (LNS + LR)) + (j & (NS - 1)) + r * NS;
}

// Every LDS address of an exchange splits into a per-thread base plus a
// compile-time offset: with j = t + q*T (NS <= T),
//   out_pos(j, r) = out_pos(t, 0) + (q*T*R + r*NS),
// and the low PADSH bits of the two terms never carry into each other, so the
// padding splits the same way (checked exhaustively for every shape in
// fft_configs.hpp).  The offsets fold into the ds_read/ds_write immediates.
template <class K>
constexpr int lds_offset(int delta) {
    return K::COLS ? pad_slots(delta * K::C, K::PADSH) : pad_slots(delta, K::PADSH);
}

// --------------------------------------------------------------------------
// inter-stage twiddles: u[r] *= W_{NS*R}^{k*r} = tw[k*r*N/(NS*R)], k = j mod NS
// --------------------------------------------------------------------------

constexpr int num_digits4(int r) { return r <= 1 ? 0 : 1 + num_digits4((r + 3) / 4); }
constexpr int pow4(int i) { return i == 0 ? 1 : 4 * pow4(i - 1); }
constexpr int top_digit_part(int r) {  // r's highest base-4 digit times its place value
    int p = 1;
    while (p * 4 <= r) p *= 4;
    return (r / p) * p;
}

template <class K, int NS, int R>
struct TwRegs {
    static constexpr int B = K::P / R;
    static constexpr int LOADS = NS == 1 ? 0 : (K::TWMODE == 0 ? R - 1 : num_digits4(R));
    float2 w[B][LOADS > 0 ? LOADS : 1];
};

// Issue the table reads a stage needs (no arithmetic yet).
template <class K, int NS, int R>
__device__ __forceinline__ void tw_issue(TwRegs<K, NS, R> &tr, int t, const float2 *__restrict__ tw) {
    constexpr int T = K::T, B = K::P / R, STR = K::N / (NS * R);
    if constexpr (TwRegs<K, NS, R>::LOADS > 0) {
        static_for<0, B>([&](auto qc) {
            constexpr int q = decltype(qc)::value;
            const int k = (t + q * T) & (NS - 1);
            if constexpr (K::TWMODE == 0) {
                static_for<1, R>([&](auto rc) {
                    constexpr int r = decltype(rc)::value;
                    tr.w[q][r - 1] = tw[k * (r * STR)];
                });
            } else {
                static_for<0, TwRegs<K, NS, R>::LOADS>([&](auto ic) {
                    constexpr int i = decltype(ic)::value;
                    tr.w[q][i] = tw[k * (pow4(i) * STR)];
                });
            }
        });
    }
}

// Expand the reads of butterfly q into w[r] = W^{k r} for r = 1..R-1.
template <class K, int NS, int R, int q>
__device__ __forceinline__ void tw_expand(const TwRegs<K, NS, R> &tr, float2 (&w)[R]) {
    if constexpr (K::TWMODE == 0) {
        static_for<1, R>([&](auto rc) { w[rc] = tr.w[q][rc - 1]; });
    } else {
        // powers of the digit bases, then products of digit parts
        static_for<1, R>([&](auto rc) {
            constexpr int r = decltype(rc)::value;
            constexpr int top = top_digit_part(r);
            if constexpr (top == r) {
                // r = d * 4^i with d in {1, 2, 3}
                constexpr int i = num_digits4(r + 1) - 1;
                constexpr int base = pow4(i);
                constexpr int d = r / base;
                if constexpr (d == 1) w[r] = tr.w[q][i];
                if constexpr (d == 2) w[r] = cmul(tr.w[q][i], tr.w[q][i]);
                if constexpr (d == 3) w[r] = cmul(w[2 * base], tr.w[q][i]);
            } else {
                w[r] = cmul(w[r - top], w[top]);
            }
        });
    }
}

// --------------------------------------------------------------------------
// LDS exchange after a stage: register (q + r*B) goes to its output position;
// afterwards register i holds canonical position t + T*i.
// --------------------------------------------------------------------------
template <class K, int NS, int R, bool FIRST>
__device__ __forceinline__ void exchange(float2 (&v)[K::P], int t, int c, float *lds) {
    constexpr int P = K::P, T = K::T, B = P / R;
    static_assert(NS <= T, "exchange addressing assumes NS <= T");
    const int wbase = lds_index<K>(out_pos<NS, R>(t, 0), c);
    const int rbase = lds_index<K>(t, c);
    if constexpr (K::XCHG == XCHG_FULL) {
        float2 *L = reinterpret_cast<float2 *>(lds);
        if constexpr (!FIRST) __syncthreads();  // previous reads are done
        static_for<0, B>([&](auto qc) {
            constexpr int q = decltype(qc)::value;
            static_for<0, R>([&](auto rc) {
                constexpr int r = decltype(rc)::value;
                L[wbase + lds_offset<K>(q * T * R + r * NS)] = v[q + r * B];
            });
        });
        __syncthreads();
        static_for<0, P>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            v[i] = L[rbase + lds_offset<K>(T * i)];
        });
    } else {
        // one real component at a time: half the LDS, twice the rounds
        if constexpr (!FIRST) __syncthreads();
        static_for<0, B>([&](auto qc) {
            constexpr int q = decltype(qc)::value;
            static_for<0, R>([&](auto rc) {
                constexpr int r = decltype(rc)::value;
                lds[wbase + lds_offset<K>(q * T * R + r * NS)] = v[q + r * B].x;
            });
        });
        __syncthreads();
        float re[P];
        static_for<0, P>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            re[i] = lds[rbase + lds_offset<K>(T * i)];
        });
        __syncthreads();
        static_for<0, B>([&](auto qc) {
            constexpr int q = decltype(qc)::value;
            static_for<0, R>([&](auto rc) {
                constexpr int r = decltype(rc)::value;
                lds[wbase + lds_offset<K>(q * T * R + r * NS)] = v[q + r * B].y;
            });
        });
        __syncthreads();
        static_for<0, P>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            v[i] = make_float2(re[i], lds[rbase + lds_offset<K>(T * i)]);
        });
    }
}

template <int R1, int... Rs>
struct FirstOf {
    static constexpr int value = R1;
};

// One radix-R stage on sub-transforms of length NS: twiddle, butterfly in
// registers; then (unless last) request the next stage's twiddles and
// exchange through LDS.  With a non-null `pre` the last stage first requests
// pre[t + T*i] into `prev` (the epilogue's reference spectrum), so those reads
// overlap the stage's arithmetic.
template <class K, bool INV, bool FIRST_X, bool PREFETCH, int NS, int R, int... Rest>
__device__ __forceinline__ void run_stages(float2 (&v)[K::P], int t, int c, const float2 *__restrict__ tw,
                                           float *lds, const TwRegs<K, NS, R> &cur,
                                           const float2 *__restrict__ pre, float2 (&prev)[K::P]) {
    constexpr int P = K::P, B = P / R;
    static_assert(P % R == 0, "radix must divide points per thread");
    if constexpr (PREFETCH && sizeof...(Rest) == 0) {
        static_for<0, P>([&](auto ic) { prev[ic] = pre[t + K::T * decltype(ic)::value]; });
    }
    static_for<0, B>([&](auto qc) {
        constexpr int q = decltype(qc)::value;
        float2 u[R];
        static_for<0, R>([&](auto rc) { u[rc] = v[q + rc * B]; });
        if constexpr (NS > 1) {
            float2 w[R];
            tw_expand<K, NS, R, q>(cur, w);
            static_for<1, R>([&](auto rc) {
                constexpr int r = decltype(rc)::value;
                u[r] = INV ? cmulc(u[r], w[r]) : cmul(u[r], w[r]);
            });
        }
        Dft<R, INV>::run(u);
        static_for<0, R>([&](auto rc) { v[q + rc * B] = u[rc]; });
    });
    if constexpr (sizeof...(Rest) > 0) {
        constexpr int NS2 = NS * R, R2 = FirstOf<Rest...>::value;
        TwRegs<K, NS2, R2> nxt;
        tw_issue<K, NS2, R2>(nxt, t, tw);  // in flight during the exchange
        exchange<K, NS, R, FIRST_X>(v, t, c, lds);
        run_stages<K, INV, false, PREFETCH, NS2, Rest...>(v, t, c, tw, lds, nxt, pre, prev);
    }
}

template <class K, bool INV, bool FIRST_X, bool PREFETCH, int R1, int... Rs>
__device__ __forceinline__ void run_fft(Radices<R1, Rs...>, float2 (&v)[K::P], int t, int c,
                                        const float2 *__restrict__ tw, float *lds,
                                        const float2 *__restrict__ pre, float2 (&prev)[K::P]) {
    TwRegs<K, 1, R1> none;  // the first stage has no twiddles
    run_stages<K, INV, FIRST_X, PREFETCH, 1, R1, Rs...>(v, t, c, tw, lds, none, pre, prev);
}

// Blocks are dispatched round-robin over the 8 XCDs.  With xcd_remap the
// logical strip of block i is chosen so that each XCD works through one
// contiguous range of strips: strips that share cache lines then meet in the
// same L2.
__device__ __forceinline__ long long logical_block(int xcd_remap) {
    const long long i = blockIdx.x, g = gridDim.x;
    if (!xcd_remap || g < 8) return i;
    const long long xcd = i & 7, local = i >> 3, per = g >> 3, rem = g & 7;
    return xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

// Global access of the P points of transform c of logical block blk (the
// caller guarantees the block exists).  With buffer addressing the workgroup's
// base is uniform, each lane adds one 32-bit offset and each register a
// scalar one; every access stays inside the resource's span, which the host
// checked fits 31 bits.  Lanes of transforms past the end of the batch read
// transform 0 of their block instead (in bounds, never stored), so the loads
// need no per-lane predication.
template <class K, int ST>
__device__ __forceinline__ void load_points(float2 (&v)[K::P], const void *__restrict__ in, long long blk, int c,
                                            int t, bool valid, const KArgs &a) {
    constexpr int EL = Store<ST>::BYTES;
    const int cl = valid ? c : 0;
    if (!a.wide) {
        const char *base = reinterpret_cast<const char *>(in) + blk * K::C * a.in_dist * EL;
        const rsrc_t r = make_rsrc(base, a.in_span);
        const unsigned lane = (unsigned)((cl * a.in_dist + (long long)t * a.stride) * EL);
        static_for<0, K::P>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            const unsigned soff = (unsigned)((long long)(K::T * i) * a.stride * EL);
            v[i] = Store<ST>::load(r, lane, soff);
        });
    } else {
        using T = typename Store<ST>::T;
        const T *src = reinterpret_cast<const T *>(in) + (blk * K::C + cl) * a.in_dist;
        static_for<0, K::P>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            const long long pos = t + K::T * i;
            v[i] = Store<ST>::load(src + pos * a.stride);
        });
    }
}

template <class K, int ST, bool NT>
__device__ __forceinline__ void store_points(const float2 (&v)[K::P], void *__restrict__ out, long long blk, int c,
                                             int t, const KArgs &a) {
    constexpr int EL = Store<ST>::BYTES;
    if (!a.wide) {
        char *base = reinterpret_cast<char *>(out) + blk * K::C * a.out_dist * EL;
        const rsrc_t r = make_rsrc(base, a.out_span);
        const unsigned lane = (unsigned)((c * a.out_dist + (long long)t * a.stride) * EL);
        static_for<0, K::P>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            const unsigned soff = (unsigned)((long long)(K::T * i) * a.stride * EL);
            Store<ST>::template store<NT>(r, lane, soff, v[i]);
        });
    } else {
        using T = typename Store<ST>::T;
        T *dst = reinterpret_cast<T *>(out) + (blk * K::C + c) * a.out_dist;
        static_for<0, K::P>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            const long long pos = t + K::T * i;
            Store<ST>::template store<NT>(dst + pos * a.stride, v[i]);
        });
    }
}

// The whole on-chip computation of one transform (first exchange of the
// kernel may skip its leading barrier).
template <class K, bool INV, int EPI, bool FIRST_X>
__device__ __forceinline__ void transform(float2 (&v)[K::P], int t, int c, const float2 *__restrict__ tw,
                                          const float2 *__restrict__ spec, float scale, float *lds) {
    constexpr bool MF = EPI == EPI_MATCHED;
    float2 h[K::P];  // reference spectrum (unused without the epilogue)
    run_fft<K, INV, FIRST_X, MF>(typename K::Rad{}, v, t, c, tw, lds, spec, h);
    if constexpr (MF) {
        // X[k] * conj(H[k]) * scale, k = t + T*i, then the inverse transform.
        // The scheduling fences keep the two transforms' register lifetimes
        // apart (interleaving them costs occupancy).
        __builtin_amdgcn_sched_barrier(0);
        static_for<0, K::P>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            const float2 y = cmulc(v[i], h[i]);
            v[i] = make_float2(y.x * scale, y.y * scale);
        });
        __builtin_amdgcn_sched_barrier(0);
        run_fft<K, !INV, false, false>(typename K::Rad{}, v, t, c, tw, lds, spec, h);
    }
}

// Occupancy hint: the LDS-derived minimum, except for kernels that need more
// registers than that leaves (persistent kernels hold a second transform;
// column kernels with the epilogue hold the reference spectrum of a strip).
template <class K, int EPI>
constexpr int occupancy_hint() {
    return (K::PERSIST || (EPI == EPI_MATCHED && K::COLS)) ? 1 : K::MIN_WAVES;
}

template <class K, int IN_ST, int OUT_ST, bool INV, int EPI>
__global__ __launch_bounds__(K::THREADS) __attribute__((amdgpu_waves_per_eu(occupancy_hint<K, EPI>())))
void fft_kernel(const void *__restrict__ in, void *__restrict__ out,
                                                         const float2 *__restrict__ tw,
                                                         const float2 *__restrict__ spec, KArgs a) {
    __shared__ float lds[K::LDS_FLOATS];
    // Streaming (non-temporal) stores only where each workgroup writes whole
    // cache lines: contiguous rows.  A column workgroup writes C-element pieces
    // of each line, which L2 must merge with its neighbours' pieces; and the
    // range-compression pass writes the intermediate the azimuth pass reads
    // next, which should stay cacheable.
    constexpr bool NT = K::NTROW && !K::COLS && EPI == EPI_NONE;
    const int tid = threadIdx.x;
    const int c = K::COLS ? (tid & (K::C - 1)) : (tid >> K::LOG_T);
    const int t = K::COLS ? (tid >> K::LOG_C) : (tid & (K::T - 1));
    float2 v[K::P];
    if constexpr (!K::PERSIST) {
        const long long blk = logical_block(a.xcd_remap);
        const bool valid = blk * K::C + c < a.batch;
        load_points<K, IN_ST>(v, in, blk, c, t, valid, a);
        transform<K, INV, EPI, true>(v, t, c, tw, spec, a.scale, lds);
        if (valid) store_points<K, OUT_ST, NT>(v, out, blk, c, t, a);
    } else {
        // persistent: this workgroup takes blocks blockIdx.x, + gridDim.x, ...
        const long long nblk = (a.batch + K::C - 1) / K::C;
        long long blk = blockIdx.x;
        bool valid = blk * K::C + c < a.batch;
        load_points<K, IN_ST>(v, in, blk, c, t, valid, a);
        for (; blk < nblk; blk += gridDim.x) {
            const long long nblk2 = blk + gridDim.x;
            const bool nvalid = nblk2 * K::C + c < a.batch;
            float2 nv[K::P];
            if (nblk2 < nblk) load_points<K, IN_ST>(nv, in, nblk2, c, t, nvalid, a);  // uniform
            transform<K, INV, EPI, false>(v, t, c, tw, spec, a.scale, lds);
            if (valid) store_points<K, OUT_ST, NT>(v, out, blk, c, t, a);
            static_for<0, K::P>([&](auto ic) { v[ic] = nv[ic]; });
            valid = nvalid;
        }
    }
}

// Host-side launcher for one instantiation.  Persistent kernels get as many
// workgroups as fit on the device at once (never more than there is work).
template <class K, int IN_ST, int OUT_ST, bool INV, int EPI>
hipError_t launch_one(const void *in, void *out, const float2 *tw, const float2 *spec, const KArgs &args,
                      hipStream_t stream) {
    KArgs a = args;
    set_spans(a, K::N, K::C, Store<IN_ST>::BYTES, Store<OUT_ST>::BYTES);
    long long blocks = (a.batch + K::C - 1) / K::C;
    if (blocks <= 0 || blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    auto kern = fft_kernel<K, IN_ST, OUT_ST, INV, EPI>;
    if constexpr (K::PERSIST) {
        static std::atomic<int> resident{0};  // workgroups resident on the whole device
        if (resident.load(std::memory_order_relaxed) == 0) {
            int per_cu = 0, dev = 0, cus = 0;
            hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, K::THREADS, 0);
            if (e != hipSuccess) return e;
            e = hipGetDevice(&dev);
            if (e != hipSuccess) return e;
            e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
            if (e != hipSuccess) return e;
            resident.store((per_cu > 0 ? per_cu : 1) * (cus > 0 ? cus : 1), std::memory_order_relaxed);
        }
        if (blocks > resident.load(std::memory_order_relaxed)) blocks = resident.load(std::memory_order_relaxed);
    }
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(K::THREADS), 0, stream, in, out, tw, spec, a);
    return hipGetLastError();
}

}  // namespace mi355fft
