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
//          the paper's Section VI exchange, here used to double occupancy);
//          HALF: the complex value rounded to a binary16 pair (N*4 bytes, one
//          round; Section VII's FP16 exchange, about 6 dB less accurate, for
//          FP16 storage only).
//          LANE: no LDS: each wave holds one 1024-point transform and every
//          exchange is a register/lane transpose made with cross-lane
//          instructions (fft_lane.hpp).
//   TWMODE 0: every inter-stage twiddle read from the table;
//          1: one table read per base-4 digit of the radix, the rest formed
//          by complex products (fewer loads, a few more FP32 operations);
//          2: every factor read from the stage's own table, laid out so that
//          consecutive lanes read consecutive entries (no products: fewer
//          FP32 operations than 1, more loads, each one coalesced);
//          3: stages whose own table is small (at most kLdsTwEntries
//          factors) read every factor from a copy of that table in LDS, which
//          the workgroup fills once; the other stages work as in mode 1.
//   PERSIST the workgroup loops over its share of the batch and loads the
//          next transform into a second register array while it computes the
//          current one (the second-array idea of Section VI, used here to
//          overlap HBM latency with arithmetic).
// Twiddles for stage s+1 are requested before stage s's LDS exchange, so
// their latency hides behind the exchange.
//
// Optional fused epilogue (Section X, range compression in one kernel):
// after the forward stages, X[k] <- X[k] * conj(H[k]) (H carrying the
// chain's 1/N), then the inverse stages run on the same registers with no
// trip to memory.
#pragma once

#include <atomic>

#include "fft_device.hpp"
#include "fft_launch.h"
#include "rd_tables.hpp"

namespace mi355fft {

enum { XCHG_FULL = 0, XCHG_SPLIT = 1, XCHG_HALF = 2, XCHG_LANE = 3 };


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

// Twiddle mode 3: a stage (NS, R) with NS > 1 takes its factors from LDS
// when its table, (R - 1) * NS factors, has at most kLdsTwEntries of them
// (stage tables exist for radices up to 32).
constexpr int kLdsTwEntries = 1024;
constexpr bool lds_tw_stage(int ns, int r) { return ns > 1 && r <= 32 && (r - 1) * ns <= kLdsTwEntries; }

// Offset (in factors) of stage ns's table in the workgroup's LDS copy, and
// (ns = 0) the total size of the copy, for the radix schedule Rs.
template <int... Rs>
constexpr int lds_tw_offset(Radices<Rs...>, int ns_target) {
    constexpr int rs[] = {Rs...};
    int ns = 1, off = 0;
    for (int i = 0; i < (int)sizeof...(Rs); ++i) {
        if (ns == ns_target) return off;
        if (lds_tw_stage(ns, rs[i])) off += (rs[i] - 1) * ns;
        ns *= rs[i];
    }
    return off;
}

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
    // Rows of a multi-transform workgroup start RSKEW slots apart modulo the
    // 32 banks (64 / C four-byte words, or 16 / C eight-byte slots), so that
    // a read across the C rows of one position (the remapped store below)
    // spreads over distinct banks.
    static constexpr int RSKEW = C_ == 1 ? 0 : (XCHG_ == XCHG_FULL ? 16 : 32) / C_;
    static constexpr int ROW_SPAN = N_ + (N_ >> PADSH) + RSKEW;
    static constexpr int SPAN = COLS_ ? (N_ * C_ + ((N_ * C_) >> PADSH)) : C_ * ROW_SPAN;
    // the cross-lane kernels keep each transform inside one wave: no LDS
    static constexpr int XFLOATS = XCHG_ == XCHG_LANE ? 1 : XCHG_ == XCHG_FULL ? 2 * SPAN : SPAN;
    // twiddle mode 3: the LDS copy of the small stage tables (float2 each),
    // after the exchange area (8-byte aligned)
    static constexpr int TWL_OFF = (XFLOATS + 1) & ~1;
    static constexpr int TWL = TWMODE_ == 3 ? lds_tw_offset(Rad_{}, 0) : 0;
    static constexpr int LDS_FLOATS = TWL > 0 ? TWL_OFF + 2 * TWL : XFLOATS;
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
    static_assert(XCHG_ != XCHG_LANE || (N_ == 1024 && P_ == 16 && !COLS_ && !PERSIST_),
                  "cross-lane exchanges: 1024-point rows, one transform per wave");
    static_assert(TWMODE_ != 3 || (TWL > 0 && XCHG_ != XCHG_LANE && !PERSIST_),
                  "twiddle mode 3: a small stage table, an LDS exchange, one transform per workgroup");
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

// The twiddle mode of stage (NS, R): mode 3 applies to the small stage
// tables and falls back to mode 1 for the others.
template <class K, int NS, int R>
constexpr int stage_twmode() {
    return K::TWMODE != 3 ? K::TWMODE : (lds_tw_stage(NS, R) ? 3 : 1);
}

template <class K, int NS, int R>
struct TwRegs {
    static constexpr int B = K::P / R;
    static constexpr int MODE = stage_twmode<K, NS, R>();
    // With the per-stage tables, the R - 1 factors of every butterfly would
    // all be live across the exchange: 60 VGPRs at radix 16 with two
    // butterflies per thread, 62 at radix 32, either of which spills.  Those
    // stages read each butterfly's factors just before applying them instead.
    static constexpr bool LATE = MODE == 2 && (B > 1 || R >= 32);
    static constexpr int LOADS = NS == 1 || LATE || MODE == 3 ? 0 : (MODE == 1 ? num_digits4(R) : R - 1);
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
            if constexpr (TwRegs<K, NS, R>::MODE == 0) {
                static_for<1, R>([&](auto rc) {
                    constexpr int r = decltype(rc)::value;
                    tr.w[q][r - 1] = tw[k * (r * STR)];
                });
            } else if constexpr (TwRegs<K, NS, R>::MODE == 2) {
                // this stage's own table: row r - 1 holds W_(NS R)^(k r) at
                // column k, so consecutive lanes read consecutive entries
                constexpr long long OFF = stage_table_offset(K::N, NS, R);
                static_for<1, R>([&](auto rc) {
                    constexpr int r = decltype(rc)::value;
                    tr.w[q][r - 1] = tw[OFF + (r - 1) * NS + k];
                });
            } else {
                static_for<0, TwRegs<K, NS, R>::LOADS>([&](auto ic) {
                    constexpr int i = decltype(ic)::value;
                    constexpr int step = pow4(i) * STR;  // folded here, never a device call
                    tr.w[q][i] = tw[k * step];
                });
            }
        });
    }
}

// Multiply u[r] by w[r] = W^{k r} (its conjugate for the inverse), r = 1..R-1.
// With the digit-base reads (TWMODE 1), r = low + 16 h with low < 16:
// w[low] is the product of its two base-4 digit parts and w[r] = w[low] *
// w[16 h].  Each factor is applied as soon as it is formed, so only the digit
// bases and one partial product are live at a time rather than all R - 1
// factors (31 complex values at radix 32, which would spill).  The products
// are the same, in the same order, as forming every factor first.
template <class K, int NS, int R, int q, bool INV>
__device__ __forceinline__ void tw_apply(const TwRegs<K, NS, R> &tr, float2 (&u)[R]) {
    auto mul = [](float2 a, float2 w) { return INV ? cmulc(a, w) : cmul(a, w); };
    if constexpr (TwRegs<K, NS, R>::MODE != 1) {
        static_for<1, R>([&](auto rc) { u[rc] = mul(u[rc], tr.w[q][rc - 1]); });
    } else {
        constexpr int D = TwRegs<K, NS, R>::LOADS;
        float2 b[D][3];  // b[i][d - 1] = W^{k d 4^i}
        static_for<0, D>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            constexpr int base = pow4(i);
            b[i][0] = tr.w[q][i];
            if constexpr (2 * base < R) b[i][1] = cmul(b[i][0], b[i][0]);
            if constexpr (3 * base < R) b[i][2] = cmul(b[i][1], b[i][0]);
        });
        constexpr int LOW = R < 16 ? R : 16;
        static_for<0, LOW>([&](auto lc) {
            constexpr int low = decltype(lc)::value;
            constexpr int d0 = low % 4, d1 = low / 4;
            float2 wl = make_float2(1.0f, 0.0f);
            if constexpr (d0 != 0 && d1 != 0) wl = cmul(b[0][d0 - 1], b[1][d1 - 1]);
            if constexpr (d0 != 0 && d1 == 0) wl = b[0][d0 - 1];
            if constexpr (d0 == 0 && d1 != 0) wl = b[1][d1 - 1];
            if constexpr (low != 0) u[low] = mul(u[low], wl);
            static_for<1, (R + 15) / 16>([&](auto hc) {
                constexpr int r = low + 16 * decltype(hc)::value;
                if constexpr (r < R) {
                    const float2 bh = b[2][decltype(hc)::value - 1];
                    if constexpr (low != 0) {
                        u[r] = mul(u[r], cmul(wl, bh));
                    } else {
                        u[r] = mul(u[r], bh);
                    }
                }
            });
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
    } else if constexpr (K::XCHG == XCHG_HALF) {
        // the complex value as a binary16 pair (round to nearest even)
        unsigned *L = reinterpret_cast<unsigned *>(lds);
        if constexpr (!FIRST) __syncthreads();
        static_for<0, B>([&](auto qc) {
            constexpr int q = decltype(qc)::value;
            static_for<0, R>([&](auto rc) {
                constexpr int r = decltype(rc)::value;
                L[wbase + lds_offset<K>(q * T * R + r * NS)] = Store<1>::narrow(v[q + r * B]);
            });
        });
        __syncthreads();
        static_for<0, P>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            v[i] = Store<1>::widen(L[rbase + lds_offset<K>(T * i)]);
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
        static_assert(K::XCHG == XCHG_SPLIT, "exchange mode");
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
// exchange through LDS.
template <class K, bool INV, bool FIRST_X, int NS, int R, int... Rest>
__device__ __forceinline__ void run_stages(float2 (&v)[K::P], int t, int c, const float2 *__restrict__ tw,
                                           float *lds, const TwRegs<K, NS, R> &cur) {
    constexpr int P = K::P, B = P / R;
    static_assert(P % R == 0, "radix must divide points per thread");
    static_for<0, B>([&](auto qc) {
        constexpr int q = decltype(qc)::value;
        float2 u[R];
        static_for<0, R>([&](auto rc) { u[rc] = v[q + rc * B]; });
        if constexpr (NS > 1 && TwRegs<K, NS, R>::MODE == 3) {
            // this butterfly's factors from the LDS copy of the stage table
            // (row r - 1, column k: consecutive lanes, consecutive entries)
            const float2 *L = reinterpret_cast<const float2 *>(lds + K::TWL_OFF) + lds_tw_offset(typename K::Rad{}, NS);
            const int k = (t + q * K::T) & (NS - 1);
            static_for<1, R>([&](auto rc) {
                constexpr int r = decltype(rc)::value;
                const float2 w = L[(r - 1) * NS + k];
                u[r] = INV ? cmulc(u[r], w) : cmul(u[r], w);
            });
        } else if constexpr (NS > 1 && TwRegs<K, NS, R>::LATE) {
            // this butterfly's factors from the stage table, read now
            constexpr long long OFF = stage_table_offset(K::N, NS, R);
            const int k = (t + q * K::T) & (NS - 1);
            static_for<1, R>([&](auto rc) {
                constexpr int r = decltype(rc)::value;
                const float2 w = tw[OFF + (r - 1) * NS + k];
                u[r] = INV ? cmulc(u[r], w) : cmul(u[r], w);
            });
        } else if constexpr (NS > 1) {
            tw_apply<K, NS, R, q, INV>(cur, u);
        }
        Dft<R, INV>::run(u);
        static_for<0, R>([&](auto rc) { v[q + rc * B] = u[rc]; });
    });
    if constexpr (sizeof...(Rest) > 0) {
        constexpr int NS2 = NS * R, R2 = FirstOf<Rest...>::value;
        TwRegs<K, NS2, R2> nxt;
        tw_issue<K, NS2, R2>(nxt, t, tw);  // in flight during the exchange
        exchange<K, NS, R, FIRST_X>(v, t, c, lds);
        run_stages<K, INV, false, NS2, Rest...>(v, t, c, tw, lds, nxt);
    }
}

// Twiddle mode 3: the workgroup copies the small stage tables into LDS.  Each
// thread loads its share into registers before it issues its data loads and
// writes them to LDS after, so the table reads overlap the data's latency;
// the first reads of the copy come after the first exchange's barrier.
template <class K, int NS, int... Rs>
struct LdsTwFill {
    __device__ __forceinline__ void load(const float2 *__restrict__) {}
    __device__ __forceinline__ void store(float *) const {}
};
template <class K, int NS, int R, int... Rs>
struct LdsTwFill<K, NS, R, Rs...> {
    static constexpr int CNT = lds_tw_stage(NS, R) ? (R - 1) * NS : 0;
    static constexpr int PER = (CNT + K::THREADS - 1) / K::THREADS;
    float2 w[PER > 0 ? PER : 1];
    LdsTwFill<K, NS * R, Rs...> rest;
    __device__ __forceinline__ void load(const float2 *__restrict__ tw) {
        static_for<0, PER>([&](auto pc) {
            const int i = decltype(pc)::value * K::THREADS + (int)threadIdx.x;
            if (i < CNT) w[pc] = tw[stage_table_offset(K::N, NS, R) + i];
        });
        rest.load(tw);
    }
    __device__ __forceinline__ void store(float *lds) const {
        float2 *L = reinterpret_cast<float2 *>(lds + K::TWL_OFF) + lds_tw_offset(typename K::Rad{}, NS);
        static_for<0, PER>([&](auto pc) {
            const int i = decltype(pc)::value * K::THREADS + (int)threadIdx.x;
            if (i < CNT) L[i] = w[pc];
        });
        rest.store(lds);
    }
};
template <class K, class Rad>
struct LdsTwFillOf;
template <class K, int... Rs>
struct LdsTwFillOf<K, Radices<Rs...>> {
    using type = LdsTwFill<K, 1, Rs...>;
};

template <class K, bool INV, bool FIRST_X, int R1, int... Rs>
__device__ __forceinline__ void run_fft(Radices<R1, Rs...>, float2 (&v)[K::P], int t, int c,
                                        const float2 *__restrict__ tw, float *lds) {
    TwRegs<K, 1, R1> none;  // the first stage has no twiddles
    run_stages<K, INV, FIRST_X, 1, R1, Rs...>(v, t, c, tw, lds, none);
}

}  // namespace mi355fft

#include "fft_lane.hpp"

namespace mi355fft {

// Blocks are dispatched round-robin over the 8 XCDs.  Strips whose pieces
// share a 128-byte line should run on one XCD, so the line meets them in one
// L2.  Two block -> strip maps (xcd_remap):
//   XCD_CONTIG  each XCD works through one contiguous range of strips;
//   XCD_GROUPS  the GROUP strips of a line run on one XCD, and successive
//               groups go to successive XCDs, so the strips in flight spread
//               over the whole row and its memory channels.
// Measured on MI355X: with rows of 32 KiB the groups win (strided copies of
// 64-byte pieces 3.37 against 3.06 TB/s; 4096-point columns 79 against
// 86 us); with rows of 8 KiB (the four-step passes at 2^20) the contiguous
// ranges win by 10%.  The host picks by row length.  Grids that are not a
// multiple of 8 * GROUP keep the contiguous ranges.
// Rows (XCD_ROWS): about 1 MiB of consecutive workgroups (ROWGROUP of them)
// per XCD at a time, successive groups on successive XCDs; blocks past the
// last whole round of 8 groups keep their own index, so the map stays a
// permutation of the grid (and block 0 stays block 0).  Measured on MI355X
// against the hardware's round-robin order, same process: 4096-point FP32
// rows 6,271 against 5,955 GB/s flushed and 6,034-6,051 against
// 5,643-5,764 back to back (groups of 8 to 32 rows all gain, 128 and more do
// not); 8192-point FP32 6,025 against 5,799 flushed; 16384-point FP16 5,500
// against 5,264 flushed; 16384-point FP32 within noise, so workgroups of more
// than 64 KiB keep the hardware's order.
template <int GROUP, int ROWGROUP = 1>
__device__ __forceinline__ long long logical_block(int xcd_remap) {
    const long long i = blockIdx.x, g = gridDim.x;
    if (xcd_remap == XCD_NONE || g < 8) return i;
    const long long xcd = i & 7, local = i >> 3;
    if (xcd_remap == XCD_ROWS) {
        const long long full = g / (8 * ROWGROUP) * (8 * ROWGROUP);
        return i < full ? ((local / ROWGROUP) * 8 + xcd) * ROWGROUP + local % ROWGROUP : i;
    }
    if (xcd_remap == XCD_GROUPS && g % (8 * GROUP) == 0) return ((local / GROUP) * 8 + xcd) * GROUP + local % GROUP;
    const long long per = g >> 3, rem = g & 7;
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
        const unsigned lane = (unsigned)((c * a.out_dist + (long long)t * a.out_stride) * EL);
        static_for<0, K::P>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            const unsigned soff = (unsigned)((long long)(K::T * i) * a.out_stride * EL);
            Store<ST>::template store<NT>(r, lane, soff, v[i]);
        });
    } else {
        using T = typename Store<ST>::T;
        T *dst = reinterpret_cast<T *>(out) + (blk * K::C + c) * a.out_dist;
        static_for<0, K::P>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            const long long pos = t + K::T * i;
            Store<ST>::template store<NT>(dst + pos * a.out_stride, v[i]);
        });
    }
}

// Store of a cross-lane 1024-point kernel: register i of lane t holds point
// lane_base_1024(t) + lane_reg_pos_1024<i>() (each register still covers 64
// consecutive points, in another lane order).
template <class K, int ST, bool NT>
__device__ __forceinline__ void store_points_lane(const float2 (&v)[K::P], void *__restrict__ out, long long blk,
                                                  int c, int t, const KArgs &a) {
    constexpr int EL = Store<ST>::BYTES;
    const int base = lane_base_1024(t);
    if (!a.wide) {
        char *b = reinterpret_cast<char *>(out) + blk * K::C * a.out_dist * EL;
        const rsrc_t r = make_rsrc(b, a.out_span);
        const unsigned lane = (unsigned)((c * a.out_dist + (long long)base * a.out_stride) * EL);
        static_for<0, K::P>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            const unsigned soff = (unsigned)((long long)lane_reg_pos_1024<i>() * a.out_stride * EL);
            Store<ST>::template store<NT>(r, lane, soff, v[i]);
        });
    } else {
        using T = typename Store<ST>::T;
        T *dst = reinterpret_cast<T *>(out) + (blk * K::C + c) * a.out_dist;
        static_for<0, K::P>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            const long long pos = base + lane_reg_pos_1024<i>();
            Store<ST>::template store<NT>(dst + pos * a.out_stride, v[i]);
        });
    }
}

// Load stage of the azimuth inverse transform in the range-Doppler chain
// (Section X: migration correction and azimuth filter fused with the inverse
// FFT).  The range-Doppler image arrives transposed, one row per range bin
// (Doppler bin k of range bin m at element m*in_dist + k), so the eight taps
// of a point are eight neighbouring rows of one column (Section X: gathering
// eight neighbouring rows).  Thread (t, c) produces Doppler bins
// k = t + T*i of range bin n = n0 + c (n0 = blk*C) of the corrected,
// filtered image:
//   dn = R0_n * (1/D_k - 1) / range_bin, s = floor(dn), mu = dn - s (the
//   fraction from the shift alone: Section X's fourth fix);
//   taps g_j = row q + alpha * (row q+1 - row q) of the interpolator table,
//   q = floor(128 mu), alpha = 128 mu - q (all exact in FP32);
//   value = sum_j g_j Z[n + s - 3 + j][k];
//   times exp(+j 2 pi R0_n * 2 (D_k - 1) / lambda), whose phase in cycles is
//   formed as an unevaluated float sum: the product of the hi parts plus its
//   exact rounding error (FMA), reduced by its nearest integer (exact), plus
//   the cross terms; the reduced phase is then accurate to about 1e-7 cycles.
//
// The C range bins of the workgroup share their taps: for Doppler bin k the
// rows n0 + s0 - 3 .. n0 + s0 + C + 4 (s0 = floor(dn) of range bin n0, never
// larger than that of the others since dn grows with R0) hold every tap of
// all C points, as long as dn changes by less than one bin across the strip
// (the host guarantees it), so that floor(dn) - s0 is 0 or 1.  The gather
// runs by column: thread tau takes Doppler bins k = tau + THREADS*m and, for
// each, loads that window of C + 8 rows into registers (one row per load
// instruction of the wave: contiguous pieces) and interpolates all C range
// bins from it, each point's eight taps starting 0 or 1 rows further down the
// window than those of the point before; the results go to LDS in natural
// order, half of the Doppler bins at a time (C * N / 2 complex values fit
// where one component of the exchange does), and each thread reads back its
// own points k = t + T*i: 16 bytes of LDS traffic per point and four
// barriers in all.  A kernel with one range bin per workgroup (C = 1) has
// nothing to share, and each point loads its own eight rows.
// The image is addressed through one buffer resource spanning its n_rg rows
// (the host guarantees it fits 31 bits), each row with its own 32-bit offset:
// rows outside [0, n_rg) fall outside the resource (a negative row wraps to an
// offset above 2^31, a row past the end lies past the span), and the
// hardware returns zero for them, which is the value the swath has there.
// The column gather needs two or more Doppler bins per thread (the two
// halves) and a strip of two or more range bins to share the window.
template <class K>
constexpr bool rcmc_column() {
    return K::C >= 2 && K::P / K::C >= 2;
}

// The azimuth filter applied to an interpolated value: acc times
// exp(+j 2 pi cycles), cycles = R0 * rate from their hi/lo parts.
__device__ __forceinline__ float2 rcmc_rotate(float2 acc, float2 r0, float4 rw) {
    const float p = r0.x * rw.y;
    const float e = fmaf(r0.x, rw.y, -p);
    const float frac = (p - rintf(p)) + (e + fmaf(r0.x, rw.z, r0.y * rw.y));
    // |frac| <= 1/2 + 2^-20: the hardware sine and cosine take the angle in
    // revolutions (measured on this range: absolute error below 1.3e-7)
    const float sn = __builtin_amdgcn_sinf(frac), cs = __builtin_amdgcn_cosf(frac);
    return make_float2(acc.x * cs - acc.y * sn, acc.x * sn + acc.y * cs);
}

// Point i of thread (t, c): interpolation of the taps z(j) = Z[n + s - 3 + j]
// with the blended table row, times the azimuth filter.
template <class K, class TapFn>
__device__ __forceinline__ float2 rcmc_point(float dn, float2 r0, float4 rw, const float4 *itab, TapFn &&tap) {
    constexpr int RS = 5;
    const float fd = floorf(dn);
    const float qf = (dn - fd) * (float)kRcmcSub;
    const int q = (int)qf;
    const float al = qf - (float)q;
    float2 acc = make_float2(0.0f, 0.0f);
    static_for<0, 4>([&](auto mc) {
        constexpr int m = decltype(mc)::value;
        const float4 g = itab[q * RS + m];
        const float w0 = fmaf(al, g.y, g.x), w1 = fmaf(al, g.w, g.z);
        const float2 z0 = tap(2 * m), z1 = tap(2 * m + 1);
        acc.x = fmaf(w0, z0.x, acc.x);
        acc.y = fmaf(w0, z0.y, acc.y);
        acc.x = fmaf(w1, z1.x, acc.x);
        acc.y = fmaf(w1, z1.y, acc.y);
    });
    return rcmc_rotate(acc, r0, rw);
}

// The same point from a window of rows held in registers: its taps are
// win[CI + d + j], d = 0 or 1.  Rather than selecting eight taps, the
// weights are shifted: nine weights w'_i = (d ? w_(i-1) : w_i), with
// w_(-1) = w_8 = 0, over win[CI .. CI + 8].
template <int CI, int W>
__device__ __forceinline__ float2 rcmc_point_win(float dn, bool d, float2 r0, float4 rw, const float4 *itab,
                                                 const float2 (&win)[W]) {
    static_assert(CI + 9 <= W, "the window holds every tap");
    constexpr int RS = 5;
    const float fd = floorf(dn);
    const float qf = (dn - fd) * (float)kRcmcSub;
    const int q = (int)qf;
    const float al = qf - (float)q;
    float w[8];
    static_for<0, 4>([&](auto mc) {
        constexpr int m = decltype(mc)::value;
        const float4 g = itab[q * RS + m];
        w[2 * m] = fmaf(al, g.y, g.x);
        w[2 * m + 1] = fmaf(al, g.w, g.z);
    });
    float2 acc = make_float2(0.0f, 0.0f);
    static_for<0, 9>([&](auto ic) {
        constexpr int i = decltype(ic)::value;
        const float lo = i < 8 ? w[i < 8 ? i : 0] : 0.0f, hi = i > 0 ? w[i > 0 ? i - 1 : 0] : 0.0f;
        const float wi = d ? hi : lo;
        acc.x = fmaf(wi, win[CI + i].x, acc.x);
        acc.y = fmaf(wi, win[CI + i].y, acc.y);
    });
    return rcmc_rotate(acc, r0, rw);
}

template <class K, int ST>
__device__ __forceinline__ void rcmc_load(float2 (&v)[K::P], const void *__restrict__ in, long long blk, int c,
                                          int t, bool valid, const KArgs &a, const float2 *__restrict__ tables,
                                          float *lds) {
    static_assert(!K::COLS && !K::PERSIST, "the migration correction reads rows of the transposed image");
    static_assert(kRcmcTaps == 8, "four float4 per table row");
    static_assert(rcmc_column<K>() || K::C == 1, "a strip of range bins takes the column gather");
    constexpr int EL = Store<ST>::BYTES, P = K::P, T = K::T;
    // table row q holds {g_j, dg_j, g_j+1, dg_j+1} for j = 0, 2, 4, 6 in four
    // float4 slots of a five-slot stride: consecutive rows start 20 banks
    // apart, so lanes reading different rows spread over the banks
    constexpr int RS = 5;
    __shared__ float4 itab[(kRcmcSub + 1) * RS];
    const int n_rg = (int)a.batch;
    const float4 *rows = reinterpret_cast<const float4 *>(tables);
    const float2 *cols = reinterpret_cast<const float2 *>(reinterpret_cast<const char *>(tables) +
                                                          rd_tables_layout(K::N, n_rg).cols);
    const float4 *interp = reinterpret_cast<const float4 *>(reinterpret_cast<const char *>(tables) +
                                                            rd_tables_layout(K::N, n_rg).interp);
    for (int e = threadIdx.x; e < (kRcmcSub + 1) * 4; e += K::THREADS) itab[(e >> 2) * RS + (e & 3)] = interp[e];
    const int n0 = (int)(blk * K::C);
    const int n = n0 + (valid ? c : 0);  // lanes past the last column redo the block's first
    const float2 r0 = cols[n];
    const unsigned rb = (unsigned)(a.in_dist * EL);
    const rsrc_t r = make_rsrc(in, (unsigned)((long long)n_rg * a.in_dist * EL));
    // integer part of a shift, kept at most n_rg so that no row offset wraps
    auto shift = [&](float dn) { return (int)fminf(floorf(dn), (float)n_rg); };

    if constexpr (rcmc_column<K>()) {
        constexpr int C = K::C, M = P / C, TH = K::THREADS, WR = C + 8, HN = K::N / 2;
        float2 *X = reinterpret_cast<float2 *>(lds);
        static_assert(C * K::N <= K::LDS_FLOATS, "half of the points fit the exchange buffer");
        // R0 of the strip's range bins (past the last one: the last one's)
        float2 r0s[C];
        static_for<0, C>([&](auto cc) { r0s[cc] = cols[min(n0 + (int)decltype(cc)::value, n_rg - 1)]; });
        const int tau = threadIdx.x;
        auto gather = [&](auto mc) {
            constexpr int m = decltype(mc)::value;
            const int k = tau + TH * m;
            const float4 rw = rows[k];
            const int s0 = shift(r0s[0].x * rw.x);
            const unsigned off = (unsigned)(n0 + s0 - 3) * rb + (unsigned)(k * EL);
            float2 win[WR];
            static_for<0, WR>([&](auto uc) {
                win[uc] = Store<ST>::load(r, off + (unsigned)decltype(uc)::value * rb, 0u);
            });
            float2 *dst = X + (k - (m >= M / 2 ? HN : 0));
            static_for<0, C>([&](auto cc) {
                constexpr int ci = decltype(cc)::value;
                const float dn = r0s[ci].x * rw.x;
                dst[ci * HN] = rcmc_point_win<ci>(dn, shift(dn) != s0, r0s[ci], rw, itab, win);
            });
        };
        __syncthreads();  // itab
        static_for<0, M / 2>(gather);  // Doppler bins [0, N/2)
        __syncthreads();
        static_for<0, P / 2>([&](auto ic) { v[ic] = X[c * HN + t + T * decltype(ic)::value]; });
        __syncthreads();  // the first half is read; the second overwrites it
        static_for<M / 2, M>(gather);  // Doppler bins [N/2, N)
        __syncthreads();
        static_for<P / 2, P>([&](auto ic) { v[ic] = X[c * HN + t + T * decltype(ic)::value - HN]; });
        __syncthreads();  // the transform's first exchange writes over X
    } else {
        // one range bin per workgroup: each point reads its own eight rows
        float4 rw[P];
        static_for<0, P>([&](auto ic) { rw[ic] = rows[t + T * decltype(ic)::value]; });
        __syncthreads();  // itab
        static_for<0, P>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            const float dn = r0.x * rw[i].x;
            const unsigned off = (unsigned)(n + shift(dn) - 3) * rb + (unsigned)((t + T * i) * EL);
            v[i] = rcmc_point<K>(dn, r0, rw[i], itab,
                                 [&](int j) { return Store<ST>::load(r, off + (unsigned)j * rb, 0u); });
        });
    }
}

// Store through LDS in the other thread-to-data map, for kernels whose input
// and output run along different axes: a row-mapped kernel (consecutive
// lanes hold consecutive points) writing strided columns hands each lane a
// point of a neighbouring transform instead (C-element pieces of a row); a
// column-mapped kernel writing contiguous rows hands consecutive lanes
// consecutive points (whole rows).
template <class K, int ST>
__device__ __forceinline__ void store_remapped(float2 (&v)[K::P], void *__restrict__ out, long long blk, int c,
                                               int t, const KArgs &a, float *lds) {
    constexpr int P = K::P, T = K::T;
    const int tid = threadIdx.x;
    const int c2 = K::COLS ? (tid >> K::LOG_T) : (tid & (K::C - 1));
    const int t2 = K::COLS ? (tid & (K::T - 1)) : (tid >> K::LOG_C);
    const int wbase = lds_index<K>(t, c), rbase = lds_index<K>(t2, c2);
    __syncthreads();  // the transform's last LDS reads are done
    if constexpr (K::XCHG == XCHG_FULL) {
        float2 *L = reinterpret_cast<float2 *>(lds);
        static_for<0, P>([&](auto ic) { L[wbase + lds_offset<K>(T * decltype(ic)::value)] = v[ic]; });
        __syncthreads();
        static_for<0, P>([&](auto ic) { v[ic] = L[rbase + lds_offset<K>(T * decltype(ic)::value)]; });
    } else {
        // one real component at a time (also for the FP16-exchange shapes: the
        // remap moves final results, which stay exact)
        static_for<0, P>([&](auto ic) { lds[wbase + lds_offset<K>(T * decltype(ic)::value)] = v[ic].x; });
        __syncthreads();
        float re[P];
        static_for<0, P>([&](auto ic) { re[ic] = lds[rbase + lds_offset<K>(T * decltype(ic)::value)]; });
        __syncthreads();
        static_for<0, P>([&](auto ic) { lds[wbase + lds_offset<K>(T * decltype(ic)::value)] = v[ic].y; });
        __syncthreads();
        static_for<0, P>([&](auto ic) {
            v[ic] = make_float2(re[ic], lds[rbase + lds_offset<K>(T * decltype(ic)::value)]);
        });
    }
    const long long m = blk * K::C + c2;
    if (m >= a.batch) return;
    if (a.perm_b == 0) {
        store_points<K, ST, false>(v, out, blk, c2, t2, a);
    } else {
        // permuted rows: each lands in its own row, so address by pointer
        const long long row = ((m & ((1LL << a.perm_b) - 1)) << a.perm_a) | (m >> a.perm_b);
        using E = typename Store<ST>::T;
        E *dst = reinterpret_cast<E *>(out) + row * a.out_dist;
        static_for<0, P>([&](auto ic) {
            const long long pos = t2 + T * decltype(ic)::value;
            Store<ST>::template store<false>(dst + pos * a.out_stride, v[ic]);
        });
    }
}

// An image row of a range pass whose reference spectrum workgroup 0 of the
// same launch computes waits for it before reading the spectrum.  Workgroup 0
// is dispatched first and waits for nothing, so the flag gets set; the bound
// (2^22 polls, a few seconds at most) only keeps a kernel from spinning
// forever should that ever fail.  One thread polls with agent-scope loads; the barrier then
// orders the workgroup's spectrum reads after the flag was seen.  No cache
// can hold an older copy of the spectrum: the launch starts with L1 and L2
// invalidated, and nothing in it reads the spectrum before it is published,
// so no acquire invalidation (of the whole L2, once per workgroup) is needed.
__device__ __forceinline__ void wait_for_reference(unsigned long long *flag, unsigned long long epoch) {
    if (threadIdx.x == 0) {
        for (int n = 0; n < (1 << 22); ++n) {
            if (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == epoch) break;
            __builtin_amdgcn_s_sleep(8);
        }
    }
    __syncthreads();
}

// The whole on-chip computation of one transform (first exchange of the
// kernel may skip its leading barrier).
// t and c are the caller's lane coordinates; the fused inverse launders them
// in place (below), so the caller keeps one copy of them, not two.
template <class K, bool INV, int EPI, bool FIRST_X>
__device__ __forceinline__ void transform(float2 (&v)[K::P], int &t, int &c, const float2 *__restrict__ tw,
                                          const float2 *__restrict__ spec, float scale, float *lds,
                                          int spec_off = 0, int spec_shift = 0,
                                          unsigned long long *ref_flag = nullptr, unsigned long long ref_epoch = 0) {
    constexpr bool MF = EPI == EPI_MATCHED || EPI == EPI_MATCHED_Y;
    if constexpr (K::XCHG == XCHG_LANE) {
        static_assert(EPI == EPI_NONE, "the cross-lane kernels run plain transforms");
        lane_fft_1024<K, INV>(v, t, tw);
    } else {
        run_fft<K, INV, FIRST_X>(typename K::Rad{}, v, t, c, tw, lds);
    }
    if constexpr (MF) {
        // X[k] * conj(H[k]), k = t + T*i, then the inverse transform.
        // The scheduling fences keep the two transforms' register lifetimes
        // apart (interleaving them costs occupancy); H is read eight values
        // at a time between fences, so it never needs a second register
        // array beside X.
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (EPI == EPI_MATCHED && !K::COLS) {
            // the spectrum is being computed by workgroup 0 of this launch
            if (ref_flag) wait_for_reference(ref_flag, ref_epoch);
        }
        // (the chains fold their power-of-two 1/N into the spectrum, which is
        // exact, so no scale is applied here)
        constexpr int HC = K::P < 8 ? K::P : 8;
        static_for<0, K::P / HC>([&](auto jc) {
            static_for<0, HC>([&](auto ec) {
                constexpr int i = decltype(jc)::value * HC + decltype(ec)::value;
                v[i] = cmulc(v[i], spec[spec_off + ((t + K::T * i) << spec_shift)]);
            });
            __builtin_amdgcn_sched_barrier(0);
        });
        // The inverse reads the same twiddle table at the same per-lane
        // indices as the forward transform.  Seen as equal, the compiler
        // keeps the forward transform's loaded twiddles and index arithmetic
        // alive across the multiply to reuse them (over 100 more VGPRs on the
        // 8-column kernels, which then spill); passing the pointer and the
        // lane coordinates through an empty asm statement hides the equality.
        // The coordinates are laundered in place, and the store that follows
        // uses the laundered copies.
        const float2 *tw2 = tw;
        asm volatile("" : "+s"(tw2), "+v"(t), "+v"(c));
        run_fft<K, !INV, false>(typename K::Rad{}, v, t, c, tw2, lds);
    }
    if constexpr (EPI == EPI_SCALE) {
        static_for<0, K::P>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            v[i] = make_float2(v[i].x * scale, v[i].y * scale);
        });
    }
    if constexpr (EPI == EPI_NONE) {
        // the plan's fixed-shift output scale 2^-s (exact), skipped when 1
        if (scale != 1.0f) {
            static_for<0, K::P>([&](auto ic) {
                constexpr int i = decltype(ic)::value;
                v[i] = make_float2(v[i].x * scale, v[i].y * scale);
            });
        }
    }
}

// The reference spectra of a SAR chain (Section X: H_r and H_a, the range
// and azimuth reference chirps' transforms), computed by the first
// workgroups of its range pass rather than by a launch of their own.  Thread
// (blk, c) transforms reference row r = blk * C + c (lanes past the last row
// transform row 0 again and store nothing).  Workgroup 0 holds row 0, the
// range spectrum that the image rows multiply by: once every thread's stores
// have completed, one thread writes this XCD's L2 back (agent-scope release
// fence), waits for that, and stores the call's epoch to the flag.
template <class K>
__device__ __forceinline__ void reference_rows(float2 (&v)[K::P], long long blk, int c, int t,
                                               const float2 *__restrict__ tw, const KArgs &a, float *lds) {
    const int r = (int)blk * K::C + c;
    const bool mine = r < a.ref_rows;
    const bool second = mine && r == 1;
    const float2 *src = second ? a.ref_in[1] : a.ref_in[0];
    [[maybe_unused]] typename LdsTwFillOf<K, typename K::Rad>::type twl;
    if constexpr (K::TWL > 0) twl.load(tw);
    static_for<0, K::P>([&](auto ic) { v[ic] = src[t + K::T * decltype(ic)::value]; });
    if constexpr (K::TWL > 0) twl.store(lds);
    int tt = t, cc = c;
    transform<K, false, EPI_NONE, true>(v, tt, cc, tw, nullptr, second ? a.ref_scale[1] : a.ref_scale[0], lds);
    if (mine) {
        float2 *dst = second ? a.ref_out[1] : a.ref_out[0];
        static_for<0, K::P>([&](auto ic) { dst[t + K::T * decltype(ic)::value] = v[ic]; });
    }
    if (blk == 0) {
        __builtin_amdgcn_s_waitcnt(0);  // this thread's stores have reached L2
        __syncthreads();
        if (threadIdx.x == 0) {
            // write this XCD's L2 back, wait until that has completed, then
            // publish (the explicit wait keeps the flag from overtaking the
            // write-back)
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
            __builtin_amdgcn_s_waitcnt(0);
            __hip_atomic_store(a.ref_flag, a.ref_epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// Occupancy hint: the LDS-derived minimum, except for persistent kernels,
// which hold a second transform and need more registers than that leaves.
template <class K, int EPI>
constexpr int occupancy_hint() {
    return K::PERSIST ? 1 : K::MIN_WAVES;
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
    // Kernels bound by instruction issue rather than memory (FP16 storage:
    // half the bytes for the same arithmetic) raise the wave's priority while
    // it issues its loads and stores, so that waves entering or leaving a
    // transform get their memory requests out ahead of waves in the middle of
    // one: 2.5-2.8% on the FP16 row transforms, while the memory-bound FP32
    // kernels lose up to 10% with it.
    constexpr bool PRIO = IN_ST == 1 && OUT_ST == 1;
    if (blockIdx.y | blockIdx.z) {  // independent problems along the grid's second and third axes
        const long long in_off = (long long)blockIdx.y * a.outer_in_dist + (long long)blockIdx.z * a.outer2_dist;
        const long long out_off = (long long)blockIdx.y * a.outer_out_dist + (long long)blockIdx.z * a.outer2_dist;
        in = reinterpret_cast<const char *>(in) + in_off * Store<IN_ST>::BYTES;
        out = reinterpret_cast<char *>(out) + out_off * Store<OUT_ST>::BYTES;
    }
    if (a.clear_flag && (blockIdx.x | blockIdx.y | blockIdx.z | threadIdx.x) == 0) *a.clear_flag = 0ull;
    const int tid = threadIdx.x;
    int c = K::COLS ? (tid & (K::C - 1)) : (tid >> K::LOG_T);
    int t = K::COLS ? (tid >> K::LOG_C) : (tid & (K::T - 1));
    float2 v[K::P];
    if constexpr (!K::PERSIST) {
        // strips per 128-byte line, from the narrower of the two sides' pieces;
        // the migration pass keeps groups of at least 8 strips on an XCD, since
        // neighbouring strips also read overlapping windows of rows (with the
        // taps staged in LDS, FETCH_SIZE was 1.3x its input against 2.1x with
        // groups of 2)
        constexpr int PIECE = K::C * (Store<IN_ST>::BYTES < Store<OUT_ST>::BYTES ? Store<IN_ST>::BYTES
                                                                                : Store<OUT_ST>::BYTES);
        constexpr int LINE_GROUP = PIECE >= 128 ? 1 : 128 / PIECE;
        constexpr int GROUP = EPI == EPI_RCMC && LINE_GROUP < 8 ? 8 : LINE_GROUP;
        // rows: workgroups per XCD group, about 1 MiB of input; workgroups of
        // more than 64 KiB keep the hardware's order (16384-point FP32 rows,
        // 128 KiB, measured within noise either way)
        constexpr long long BLOCK_BYTES = (long long)K::C * K::N * Store<IN_ST>::BYTES;
        constexpr int ROWGROUP = BLOCK_BYTES > (64 << 10) ? 1 : (int)((1 << 20) / BLOCK_BYTES);
        long long blk = logical_block<GROUP, ROWGROUP>(a.xcd_remap);
        if constexpr (EPI == EPI_MATCHED && !K::COLS) {
            if (a.ref_blocks > 0) {
                // the chain's reference spectra come first (the launcher
                // keeps blocks in dispatch order for them)
                if (blk < a.ref_blocks) {
                    reference_rows<K>(v, blk, c, t, tw, a, lds);
                    return;
                }
                blk -= a.ref_blocks;
            }
        }
        const bool valid = blk * K::C + c < a.batch;
        static_assert(K::TWL == 0 || EPI != EPI_RCMC, "the migration pass keeps its taps in LDS");
        [[maybe_unused]] typename LdsTwFillOf<K, typename K::Rad>::type twl;
        if constexpr (K::TWL > 0) twl.load(tw);
        if constexpr (EPI == EPI_SCALE) {
            // the range-Doppler chain's tables for the migration pass that follows
            if (a.rd_tables)
                rd_table_entry((long long)blockIdx.x * K::THREADS + threadIdx.x, K::N, a.batch, a.rd_geo,
                               a.rd_interp, a.rd_tables);
        }
        if constexpr (EPI == EPI_RCMC) {
            rcmc_load<K, IN_ST>(v, in, blk, c, t, valid, a, spec, lds);
            transform<K, INV, EPI_NONE, true>(v, t, c, tw, spec, a.scale, lds);
        } else {
            if constexpr (PRIO) __builtin_amdgcn_s_setprio(3);
            load_points<K, IN_ST>(v, in, blk, c, t, valid, a);
            if constexpr (PRIO) __builtin_amdgcn_s_setprio(0);
            if constexpr (K::TWL > 0) twl.store(lds);
            if constexpr (EPI == EPI_MATCHED_Y) {
                transform<K, INV, EPI, true>(v, t, c, tw, spec, a.scale, lds, (int)blockIdx.y, a.spec_shift);
            } else {
                transform<K, INV, EPI, true>(v, t, c, tw, spec, a.scale, lds, 0, 0, a.ref_flag, a.ref_epoch);
            }
        }
        if constexpr (EPI == EPI_TWIDDLE || EPI == EPI_TWIDDLE_Y || EPI == EPI_MATCHED_Y) {
            // four-step: point k1 = t + T*i of column n2 times W_N^(n2 k1).
            // Four factors are looked up exactly (W^m = lo[m mod S] *
            // hi[m div S], m < N): W^(n2 t), W^(n2 T), W^(4 n2 T) and
            // W^(16 n2 T).  With i = i0 + 4 g, the point's factor is
            // c[i0] * H[g], where c[i0] = W^(n2 t) W^(n2 T i0) and H[g] is
            // the product of the powers of the other two for the base-4
            // digits of g: eight table reads per thread instead of two per
            // point, at most six products deep.
            static_assert(K::P % 4 == 0 && K::P <= 32, "four-step columns hold 4 to 32 points per thread");
            // the matched pass keeps its spectrum in spec and the table in tab2
            // and multiplies by the conjugate factor (it ends with an inverse)
            constexpr bool CONJ = INV || EPI == EPI_MATCHED_Y;
            const float2 *tab = EPI == EPI_MATCHED_Y ? a.tab2 : spec;
            const float2 *lo = tab, *hi = tab + (1 << a.aux);
            const int mask = (1 << a.aux) - 1;
            // the column's index, or for the forms keyed by the grid's second
            // axis (EPI_TWIDDLE_Y, EPI_MATCHED_Y) that axis's index
            const int n2 = EPI == EPI_TWIDDLE ? (int)(blk * K::C) + (valid ? c : 0) : (int)blockIdx.y;
            auto look = [&](int m) { return cmul(lo[m & mask], hi[m >> a.aux]); };
            float2 cf[4];
            cf[0] = look(n2 * t);
            if constexpr (EPI != EPI_MATCHED_Y) {
                // this pass's share 2^-s of the plan's output scale, folded
                // into the factors (exact: a power of two)
                cf[0] = make_float2(cf[0].x * a.scale, cf[0].y * a.scale);
            }
            const float2 w1 = look(n2 * K::T);
            const float2 w2 = cmul(w1, w1);
            cf[1] = cmul(cf[0], w1);
            cf[2] = cmul(cf[0], w2);
            cf[3] = cmul(cf[2], w1);
            constexpr int NG = K::P / 4;
            float2 e1[3], e2 = make_float2(1.0f, 0.0f);
            if constexpr (NG > 1) {
                e1[0] = look(n2 * K::T * 4);
                e1[1] = cmul(e1[0], e1[0]);
                e1[2] = cmul(e1[1], e1[0]);
            }
            if constexpr (NG > 4) e2 = look(n2 * K::T * 16);
            static_for<0, NG>([&](auto gc) {
                constexpr int g = decltype(gc)::value, g0 = g % 4, g1 = g / 4;
                float2 h = make_float2(1.0f, 0.0f);
                if constexpr (g0 != 0 && g1 != 0) h = cmul(e1[g0 - 1], e2);
                if constexpr (g0 != 0 && g1 == 0) h = e1[g0 - 1];
                if constexpr (g0 == 0 && g1 != 0) h = e2;
                static_for<0, 4>([&](auto jc) {
                    constexpr int i = 4 * g + decltype(jc)::value;
                    const float2 w = g == 0 ? cf[decltype(jc)::value] : cmul(cf[decltype(jc)::value], h);
                    v[i] = CONJ ? cmulc(v[i], w) : cmul(v[i], w);
                });
            });
        }
        if constexpr (EPI == EPI_RCMC || EPI == EPI_SCALE || EPI == EPI_TWIDDLE) {
            // input and output run along different axes of the image
            store_remapped<K, OUT_ST>(v, out, blk, c, t, a, lds);
        } else {
            if constexpr (PRIO) __builtin_amdgcn_s_setprio(3);
            if constexpr (K::XCHG == XCHG_LANE) {
                if (valid) store_points_lane<K, OUT_ST, NT>(v, out, blk, c, t, a);
            } else {
                if (valid) store_points<K, OUT_ST, NT>(v, out, blk, c, t, a);
            }
            if constexpr (PRIO) __builtin_amdgcn_s_setprio(0);
        }
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
    a.ref_blocks = 0;
    if (a.ref_rows > 0) {
        // reference rows ahead of the image rows: matched rows only, blocks
        // in dispatch order, one problem; hipErrorNotSupported tells the
        // caller to run the reference transforms as a launch of their own
        constexpr bool OK = EPI == EPI_MATCHED && !K::COLS && !K::PERSIST && K::XCHG != XCHG_LANE;
        // (both row maps keep block 0, the publisher, as block 0)
        if (!OK || a.ref_rows > 2 || !a.ref_flag || (a.xcd_remap != XCD_NONE && a.xcd_remap != XCD_ROWS) ||
            a.outer > 1 || a.outer2 > 1)
            return hipErrorNotSupported;
        a.ref_blocks = (a.ref_rows + K::C - 1) / K::C;
        blocks += a.ref_blocks;
    }
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
    const unsigned outer = a.outer > 1 ? (unsigned)a.outer : 1u;
    const unsigned outer2 = a.outer2 > 1 ? (unsigned)a.outer2 : 1u;
    if ((outer > 1 || outer2 > 1) && K::PERSIST) return hipErrorInvalidValue;
    if (outer > 65535 || outer2 > 65535) return hipErrorInvalidValue;
    return launch_kernel(kern, dim3((unsigned)blocks, outer, outer2), dim3(K::THREADS), stream, in, out, tw, spec,
                         a);
}

}  // namespace mi355fft
