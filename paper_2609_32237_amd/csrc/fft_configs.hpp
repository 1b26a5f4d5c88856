// fft_configs.hpp -- per-size kernel shapes and the instantiation dispatcher.
//
// Shapes (points per thread P, transforms per workgroup C, radix sequence,
// exchange mode, twiddle mode, persistence) are chosen for gfx950: wave64,
// 160 KiB LDS per CU, 512 VGPRs per SIMD lane.  Rows keep one transform per
// 256-512 threads; columns keep a strip of C adjacent columns so each row
// access is a C-element segment.  The paper's M6 schedules (Section VI:
// 16-8-8-8 for 8192 and 16-16-8-8 for 16384, 16 values per thread) were
// shaped by a 32 KiB threadgroup buffer; these use larger radices because the
// LDS is five times larger.
//
// Each size lists its variants; index 0 of each list is the default.  Every
// variant computes the same transform, and the tests force each of them.
#pragma once

#include "fft_kernel.hpp"

namespace mi355fft {

template <int N>
struct Configs;

// Each list's defaults are given per storage (FP32, FP16) for the plain
// transform and for the matched-filter (SAR) kernels (storage of the
// intermediate): FP16 storage moves half the bytes per point, so its kernels
// are limited by arithmetic issue and prefer the higher-occupancy split
// exchange; the matched-filter kernels hold two transforms' worth of state and
// prefer the shapes that do not spill.  The TWMODE 0 variants are kept as
// regression cases for the table-read twiddle path.
//                 N     P  C  COLS   XCHG        TW PERSIST radices
// Short transforms serve as the column passes of four-step transforms longer
// than 16384 points (many columns per workgroup, one or two exchanges).
template <>
struct Configs<64> {
    using Rows = KList<KCfg<64, 16, 16, false, XCHG_SPLIT, 1, false, Radices<16, 4>>>;
    using Cols = KList<KCfg<64, 16, 64, true, XCHG_SPLIT, 1, false, Radices<16, 4>>>;
    using Rcmc = Rows;
    using RowsHalf = Rows;
    static constexpr int kRowDefault[2] = {0, 0}, kColDefault[2] = {0, 0};
    static constexpr int kRowMatched[2] = {0, 0}, kColMatched[2] = {0, 0};
};
template <>
struct Configs<128> {
    using Rows = KList<KCfg<128, 16, 16, false, XCHG_SPLIT, 1, false, Radices<16, 8>>>;
    using Cols = KList<KCfg<128, 16, 32, true, XCHG_SPLIT, 1, false, Radices<16, 8>>>;
    using Rcmc = Rows;
    using RowsHalf = Rows;
    static constexpr int kRowDefault[2] = {0, 0}, kColDefault[2] = {0, 0};
    static constexpr int kRowMatched[2] = {0, 0}, kColMatched[2] = {0, 0};
};
template <>
struct Configs<256> {
    using Rows = KList<KCfg<256, 16, 16, false, XCHG_SPLIT, 1, false, Radices<16, 16>>>;
    using Cols = KList<KCfg<256, 16, 16, true, XCHG_SPLIT, 1, false, Radices<16, 16>>>;
    using Rcmc = Rows;
    using RowsHalf = Rows;
    static constexpr int kRowDefault[2] = {0, 0}, kColDefault[2] = {0, 0};
    static constexpr int kRowMatched[2] = {0, 0}, kColMatched[2] = {0, 0};
};
template <>
struct Configs<512> {
    using Rows = KList<KCfg<512, 16, 8, false, XCHG_SPLIT, 1, false, Radices<16, 16, 2>>>;
    // 16-column strips measured 5% faster than 8 in the four-step passes
    using Cols = KList<KCfg<512, 16, 16, true, XCHG_SPLIT, 1, false, Radices<16, 16, 2>>,
                       KCfg<512, 16, 8, true, XCHG_SPLIT, 1, false, Radices<16, 16, 2>>>;
    using Rcmc = Rows;
    using RowsHalf = Rows;
    static constexpr int kRowDefault[2] = {0, 0}, kColDefault[2] = {0, 0};
    static constexpr int kRowMatched[2] = {0, 0}, kColMatched[2] = {0, 0};
};
template <>
struct Configs<1024> {
    using Rows = KList<KCfg<1024, 16, 4, false, XCHG_SPLIT, 1, false, Radices<16, 16, 4>>,
                       KCfg<1024, 16, 4, false, XCHG_FULL, 1, false, Radices<16, 16, 4>>,
                       KCfg<1024, 16, 4, false, XCHG_FULL, 1, true, Radices<16, 16, 4>>,
                       KCfg<1024, 16, 4, false, XCHG_FULL, 0, false, Radices<16, 16, 4>>,
                       KCfg<1024, 16, 1, false, XCHG_FULL, 1, false, Radices<16, 16, 4>>,
                       // every exchange across the lanes of one wave, no LDS:
                       // four transforms (waves) or one per workgroup
                       KCfg<1024, 16, 4, false, XCHG_LANE, 1, false, Radices<16, 16, 4>>,
                       KCfg<1024, 16, 1, false, XCHG_LANE, 1, false, Radices<16, 16, 4>>>;
    using Cols = KList<KCfg<1024, 16, 8, true, XCHG_SPLIT, 1, false, Radices<16, 16, 4>>,
                       KCfg<1024, 16, 8, true, XCHG_FULL, 0, false, Radices<16, 16, 4>>>;
    // 8 range bins per strip: 229 against 256 us for 16 (which held one
    // Doppler bin per thread, too few for the column gather) on a 1024 x 16384
    // range-Doppler chain
    using Rcmc = KList<KCfg<1024, 16, 8, false, XCHG_SPLIT, 1, false, Radices<16, 16, 4>>,
                       KCfg<1024, 16, 4, false, XCHG_SPLIT, 1, false, Radices<16, 16, 4>>>;
    using RowsHalf = KList<KCfg<1024, 16, 4, false, XCHG_HALF, 1, false, Radices<16, 16, 4>>>;
    static constexpr int kRowDefault[2] = {1, 0}, kColDefault[2] = {0, 0};
    static constexpr int kRowMatched[2] = {1, 1}, kColMatched[2] = {0, 0};
};
template <>
struct Configs<2048> {
    using Rows = KList<KCfg<2048, 16, 2, false, XCHG_SPLIT, 1, false, Radices<16, 16, 8>>,
                       KCfg<2048, 16, 2, false, XCHG_FULL, 1, false, Radices<16, 16, 8>>,
                       KCfg<2048, 16, 2, false, XCHG_FULL, 1, true, Radices<16, 16, 8>>,
                       KCfg<2048, 16, 2, false, XCHG_FULL, 0, false, Radices<16, 16, 8>>,
                       KCfg<2048, 16, 1, false, XCHG_FULL, 1, false, Radices<16, 16, 8>>>;
    using Cols = KList<KCfg<2048, 16, 4, true, XCHG_SPLIT, 1, false, Radices<16, 16, 8>>,
                       KCfg<2048, 16, 4, true, XCHG_FULL, 0, false, Radices<16, 16, 8>>>;
    // 32 points per thread: 228 against 241 us (16 points, 8 range bins) and
    // 247 us (16 points, 4 range bins) for a 2048 x 8192 range-Doppler chain
    // with FP32 intermediates, 199 against 197 and 212 us with FP16
    using Rcmc = KList<KCfg<2048, 32, 8, false, XCHG_SPLIT, 1, false, Radices<16, 16, 8>>,
                       KCfg<2048, 16, 8, false, XCHG_SPLIT, 1, false, Radices<16, 16, 8>>>;
    using RowsHalf = KList<KCfg<2048, 16, 2, false, XCHG_HALF, 1, false, Radices<16, 16, 8>>>;
    static constexpr int kRowDefault[2] = {0, 0}, kColDefault[2] = {0, 0};
    static constexpr int kRowMatched[2] = {0, 0}, kColMatched[2] = {0, 0};
};
template <>
struct Configs<4096> {
    // measured in the hardware's block order: the hint cost about 2% on this
    // shape and gained 2-5% on the others (the default is now index 8, below)
    using Rows = KList<KCfg<4096, 16, 1, false, XCHG_FULL, 1, false, Radices<16, 16, 16>, false>,
                       KCfg<4096, 16, 1, false, XCHG_SPLIT, 1, false, Radices<16, 16, 16>>,
                       KCfg<4096, 16, 1, false, XCHG_FULL, 1, true, Radices<16, 16, 16>>,
                       KCfg<4096, 16, 1, false, XCHG_SPLIT, 1, true, Radices<16, 16, 16>>,
                       KCfg<4096, 16, 1, false, XCHG_FULL, 0, false, Radices<16, 16, 16>>,
                       KCfg<4096, 16, 1, false, XCHG_SPLIT, 0, false, Radices<16, 16, 16>>,
                       // every factor from the per-stage tables
                       KCfg<4096, 16, 1, false, XCHG_FULL, 2, false, Radices<16, 16, 16>, false>,
                       KCfg<4096, 16, 1, false, XCHG_SPLIT, 2, false, Radices<16, 16, 16>>,
                       // the complex exchange with streaming row stores
                       KCfg<4096, 16, 1, false, XCHG_FULL, 1, false, Radices<16, 16, 16>, true>,
                       // the second stage's 240 factors from LDS (twiddle mode 3)
                       KCfg<4096, 16, 1, false, XCHG_SPLIT, 3, false, Radices<16, 16, 16>>>;
    using Cols = KList<KCfg<4096, 32, 4, true, XCHG_SPLIT, 1, false, Radices<16, 16, 16>>,
                       KCfg<4096, 32, 4, true, XCHG_SPLIT, 0, false, Radices<16, 16, 16>>,
                       KCfg<4096, 16, 4, true, XCHG_SPLIT, 1, false, Radices<16, 16, 16>>,
                       KCfg<4096, 32, 8, true, XCHG_SPLIT, 1, false, Radices<16, 16, 16>>,
                       KCfg<4096, 32, 8, true, XCHG_SPLIT, 2, false, Radices<16, 16, 16>>,
                       // two radix-64 stages, 64 points per thread: one exchange per
                       // transform instead of two, and fewer VALU instructions per
                       // point (100 against 106 for the matched pass)
                       KCfg<4096, 64, 8, true, XCHG_SPLIT, 1, false, Radices<64, 64>>,
                       KCfg<4096, 64, 4, true, XCHG_SPLIT, 1, false, Radices<64, 64>>>;
    // 8-column strips measured fastest for both column passes: 64-byte row
    // pieces against 32 (plain 82 vs 117 us, matched 88 vs 100 us per 4096^2
    // with 32 points per thread).  Radix 64, 8 columns, 30 interleaved
    // flushed samples per 4096^2 workload: plain 75.2 against 78.8 us (FP32)
    // and 53.8 against 55.0 (FP16); SAR chain 143.1 against 157.1 us (FP32
    // intermediate) and 131.3 against 135.7 (FP16).
    using Rcmc = KList<KCfg<4096, 32, 8, false, XCHG_SPLIT, 1, false, Radices<16, 16, 16>>,
                       KCfg<4096, 16, 4, false, XCHG_SPLIT, 1, false, Radices<16, 16, 16>>,
                       KCfg<4096, 32, 8, false, XCHG_SPLIT, 2, false, Radices<16, 16, 16>>>;
    using RowsHalf = KList<KCfg<4096, 16, 1, false, XCHG_HALF, 1, false, Radices<16, 16, 16>>>;
    // FP32 rows: with the rows' XCD groups, streaming stores win back to back
    // (6,108-6,171 against 6,015-6,027 GB/s, same process; flushed 6,120
    // against 6,298, where a call without them leaves its write-back for later)
    // matched rows with an FP16 intermediate (issue-bound): the LDS factors
    // took the range-Doppler chain 0.4-2.8 us faster in five same-process
    // comparisons on two boxes (181.2 -> 179.0 us on one), and moved the SAR
    // chain by -0.4 to +1.4 us; with an FP32 intermediate they cost the SAR
    // chain 1.6-2.7 us, so those rows keep the computed factors
    // matched columns (the SAR azimuth pass) reading an FP32 intermediate:
    // the 4-column strips, two workgroups per CU, took the chain from
    // 140.9 to 134.8-134.9 us (same process, two runs); with an FP16
    // intermediate (16-byte pieces) they measured 125.5-126.3 against
    // 125.2-126.0 us, so those keep the 8-column strips
    static constexpr int kRowDefault[2] = {8, 1}, kColDefault[2] = {5, 5};
    static constexpr int kRowMatched[2] = {1, 9}, kColMatched[2] = {6, 5};
};
template <>
struct Configs<8192> {
    using Rows = KList<KCfg<8192, 16, 1, false, XCHG_SPLIT, 1, false, Radices<16, 16, 16, 2>>,
                       KCfg<8192, 32, 1, false, XCHG_FULL, 1, false, Radices<32, 16, 16>>,
                       KCfg<8192, 16, 1, false, XCHG_SPLIT, 1, true, Radices<16, 16, 16, 2>>,
                       KCfg<8192, 16, 1, false, XCHG_FULL, 0, false, Radices<16, 16, 16, 2>>,
                       KCfg<8192, 32, 1, false, XCHG_SPLIT, 1, false, Radices<32, 16, 16>>,
                       KCfg<8192, 32, 1, false, XCHG_SPLIT, 2, false, Radices<32, 16, 16>>,
                       KCfg<8192, 16, 1, false, XCHG_SPLIT, 2, false, Radices<16, 16, 16, 2>>,
                       // the second stage's 240 factors from LDS (twiddle mode 3)
                       KCfg<8192, 16, 1, false, XCHG_SPLIT, 3, false, Radices<16, 16, 16, 2>>>;
    using Cols = KList<KCfg<8192, 32, 2, true, XCHG_SPLIT, 1, false, Radices<16, 16, 16, 2>>,
                       KCfg<8192, 32, 2, true, XCHG_SPLIT, 0, false, Radices<16, 16, 16, 2>>>;
    using Rcmc = KList<KCfg<8192, 32, 4, false, XCHG_SPLIT, 1, false, Radices<16, 16, 16, 2>>,
                       KCfg<8192, 16, 2, false, XCHG_SPLIT, 1, false, Radices<16, 16, 16, 2>>>;
    // binary16 exchange: three stages 5.5 TB/s, four stages 4.8
    using RowsHalf = KList<KCfg<8192, 32, 1, false, XCHG_HALF, 1, false, Radices<32, 16, 16>>,
                           KCfg<8192, 16, 1, false, XCHG_HALF, 1, false, Radices<16, 16, 16, 2>>>;
    // FP16: 32 points per thread in three stages, 5.7 vs 4.9 TB/s.  FP32:
    // the second stage's factors from LDS, 5,740 against 5,607 GB/s flushed
    // and 5,700-5,731 against 5,318-5,604 back to back (same box, one run)
    static constexpr int kRowDefault[2] = {7, 4}, kColDefault[2] = {0, 0};
    static constexpr int kRowMatched[2] = {0, 0}, kColMatched[2] = {0, 0};
};
template <>
struct Configs<16384> {
    using Rows = KList<KCfg<16384, 16, 1, false, XCHG_SPLIT, 1, false, Radices<16, 16, 16, 4>>,
                       KCfg<16384, 32, 1, false, XCHG_SPLIT, 1, false, Radices<16, 16, 16, 4>>,
                       KCfg<16384, 32, 1, false, XCHG_SPLIT, 1, true, Radices<16, 16, 16, 4>>,
                       KCfg<16384, 32, 1, false, XCHG_SPLIT, 0, false, Radices<16, 16, 16, 4>>,
                       KCfg<16384, 32, 1, false, XCHG_SPLIT, 1, false, Radices<32, 16, 32>>,
                       KCfg<16384, 32, 1, false, XCHG_SPLIT, 2, false, Radices<32, 16, 32>>,
                       // the second stage's 240 factors from LDS (twiddle mode 3)
                       KCfg<16384, 16, 1, false, XCHG_SPLIT, 3, false, Radices<16, 16, 16, 4>>>;
    using Cols = KList<KCfg<16384, 32, 1, true, XCHG_SPLIT, 0, false, Radices<16, 16, 16, 4>>,
                       KCfg<16384, 32, 1, true, XCHG_SPLIT, 1, false, Radices<16, 16, 16, 4>>>;
    // three stages (32 x 16 x 32) against four: one exchange and one twiddle
    // pass fewer; measured 5.5 vs 5.3 TB/s (FP32) and 4.9 vs 3.8 TB/s (FP16).
    // FP32: four stages with the second stage's factors from LDS beat both,
    // 5,800-5,816 against 5,660-5,693 GB/s flushed and 5,637-5,828 against
    // 5,128-5,722 back to back (two boxes, same process each)
    static constexpr int kRowDefault[2] = {6, 4}, kColDefault[2] = {1, 1};
    using Rcmc = KList<KCfg<16384, 32, 2, false, XCHG_SPLIT, 1, false, Radices<16, 16, 16, 4>>,
                       KCfg<16384, 16, 1, false, XCHG_SPLIT, 1, false, Radices<16, 16, 16, 4>>>;
    // binary16 exchange: three stages fastest (4.8 TB/s), then 32 points per
    // thread in four stages (4.3), then 16 (4.0)
    using RowsHalf = KList<KCfg<16384, 32, 1, false, XCHG_HALF, 1, false, Radices<32, 16, 32>>,
                           KCfg<16384, 32, 1, false, XCHG_HALF, 1, false, Radices<16, 16, 16, 4>>,
                           KCfg<16384, 16, 1, false, XCHG_HALF, 1, false, Radices<16, 16, 16, 4>>>;
    static constexpr int kRowMatched[2] = {4, 4}, kColMatched[2] = {1, 1};
};

// Small batches: a batch that gives the default row shape (several
// transforms per workgroup) fewer workgroups than the chip has CUs runs one
// transform per workgroup instead.  Measured on MI355X for 64 transforms
// (one flushed call): N = 1024 6.7 against 7.7 us, N = 2048 7.3 against
// 8.1 us.
template <int N>
struct SmallRows {
    static constexpr int variant = -1;     // index into Rows, or none
    static constexpr long long below = 0;  // applies to batches below this
};
template <>
struct SmallRows<1024> {
    static constexpr int variant = 4;
    static constexpr long long below = 4 * 256;
};
template <>
struct SmallRows<2048> {
    static constexpr int variant = 4;
    static constexpr long long below = 2 * 256;
};

template <int I, class L>
struct KAt;
template <class K, class... Ks>
struct KAt<0, KList<K, Ks...>> {
    using type = K;
};
template <int I, class K, class... Ks>
struct KAt<I, KList<K, Ks...>> {
    using type = typename KAt<I - 1, KList<Ks...>>::type;
};

// Column shapes for the four-step epilogues (EPI_TWIDDLE, EPI_TWIDDLE_Y,
// EPI_MATCHED_Y), which hold at most 32 points per thread: the size's default
// shapes unless a size names others.
template <int N>
struct FourStepCols {
    static constexpr int plain[2] = {Configs<N>::kColDefault[0], Configs<N>::kColDefault[1]};
    static constexpr int matched = Configs<N>::kColMatched[0];  // (FP32 data only)
};
template <>
struct FourStepCols<4096> {
    static constexpr int plain[2] = {3, 3};
    static constexpr int matched = 3;
};

// The column shape of the scaled transform (EPI_SCALE, the range-Doppler
// chain's azimuth pass).  At 4096 points the 4-column radix-64 strips
// measured 205.7 against 214.3 us (8 columns) per range-Doppler chain with
// FP32 intermediates, 190.7 against 191.9 with FP16 (30 interleaved flushed
// samples each), although 8 columns are faster for the plain transform.
template <int N>
struct ScaleCols {
    static constexpr int v[2] = {Configs<N>::kColDefault[0], Configs<N>::kColDefault[1]};
};
template <>
struct ScaleCols<4096> {
    static constexpr int v[2] = {6, 6};
};

template <class L>
struct KListSize;
template <class... Ks>
struct KListSize<KList<Ks...>> {
    static constexpr int value = sizeof...(Ks);
};

// Calls f(K{}) for the idx-th entry of the list.
template <class F, class K, class... Ks>
hipError_t with_variant(int idx, KList<K, Ks...>, F &&f) {
    if (idx == 0) return f(K{});
    if constexpr (sizeof...(Ks) > 0) {
        return with_variant(idx - 1, KList<Ks...>{}, f);
    } else {
        return hipErrorInvalidValue;
    }
}

// Supported (layout, storage, direction, epilogue) combinations:
//   plain FFT:  rows or columns, input storage == output storage, either direction;
//   matched:    forward, multiply by conj(spec) (spec carries 1/N), inverse:
//               rows read FP32 and write FP32 or FP16 (range compression);
//               columns read FP32 or FP16 and write FP32 (azimuth compression);
//   scaled:     columns, forward, input storage == output storage (the azimuth
//               FFT of the full range-Doppler chain);
//   twiddled:   columns, either direction, input storage == output storage,
//               written as rows (first pass of a four-step transform), or
//               written in place with the factor keyed by the second grid
//               axis (middle pass of a three-pass transform);
//   RCMC:       the Rcmc list (row-mapped, several transforms per workgroup),
//               inverse, read FP32 or FP16, write FP32 columns (migration
//               correction, azimuth filter and azimuth inverse FFT).
template <class K>
hipError_t dispatch_cfg_full(int in_st, int out_st, int inv, int epi, const void *in, void *out, const float2 *tw,
                             const float2 *spec, const KArgs &a, hipStream_t s) {
    if (epi == EPI_NONE) {
        if (in_st != out_st) return hipErrorInvalidValue;
        if (in_st == 0)
            return inv ? launch_one<K, 0, 0, true, EPI_NONE>(in, out, tw, spec, a, s)
                       : launch_one<K, 0, 0, false, EPI_NONE>(in, out, tw, spec, a, s);
        return inv ? launch_one<K, 1, 1, true, EPI_NONE>(in, out, tw, spec, a, s)
                   : launch_one<K, 1, 1, false, EPI_NONE>(in, out, tw, spec, a, s);
    }
    if (epi == EPI_SCALE) {
        if constexpr (K::COLS && !K::PERSIST) {
            if (inv || in_st != out_st) return hipErrorInvalidValue;
            return in_st == 0 ? launch_one<K, 0, 0, false, EPI_SCALE>(in, out, tw, spec, a, s)
                              : launch_one<K, 1, 1, false, EPI_SCALE>(in, out, tw, spec, a, s);
        } else {
            return hipErrorInvalidValue;
        }
    }
    if (epi == EPI_TWIDDLE) {
        if constexpr (K::COLS && !K::PERSIST && K::P <= 32) {
            if (in_st != out_st) return hipErrorInvalidValue;
            if (in_st == 0)
                return inv ? launch_one<K, 0, 0, true, EPI_TWIDDLE>(in, out, tw, spec, a, s)
                           : launch_one<K, 0, 0, false, EPI_TWIDDLE>(in, out, tw, spec, a, s);
            return inv ? launch_one<K, 1, 1, true, EPI_TWIDDLE>(in, out, tw, spec, a, s)
                       : launch_one<K, 1, 1, false, EPI_TWIDDLE>(in, out, tw, spec, a, s);
        } else {
            return hipErrorInvalidValue;
        }
    }
    if (epi == EPI_TWIDDLE_Y) {
        if constexpr (K::COLS && !K::PERSIST && K::P <= 32) {
            if (in_st != out_st) return hipErrorInvalidValue;
            if (in_st == 0)
                return inv ? launch_one<K, 0, 0, true, EPI_TWIDDLE_Y>(in, out, tw, spec, a, s)
                           : launch_one<K, 0, 0, false, EPI_TWIDDLE_Y>(in, out, tw, spec, a, s);
            return inv ? launch_one<K, 1, 1, true, EPI_TWIDDLE_Y>(in, out, tw, spec, a, s)
                       : launch_one<K, 1, 1, false, EPI_TWIDDLE_Y>(in, out, tw, spec, a, s);
        } else {
            return hipErrorInvalidValue;
        }
    }
    if (epi == EPI_MATCHED_Y) {
        if constexpr (K::COLS && !K::PERSIST && K::P <= 32) {
            if (inv || in_st != 0 || out_st != 0) return hipErrorInvalidValue;
            return launch_one<K, 0, 0, false, EPI_MATCHED_Y>(in, out, tw, spec, a, s);
        } else {
            return hipErrorInvalidValue;
        }
    }
    if (epi == EPI_RCMC) return hipErrorInvalidValue;  // only through dispatch_rcmc
    if (epi != EPI_MATCHED || inv) return hipErrorInvalidValue;
    if constexpr (!K::COLS) {
        if (in_st != 0) return hipErrorInvalidValue;
        return out_st == 0 ? launch_one<K, 0, 0, false, EPI_MATCHED>(in, out, tw, spec, a, s)
                           : launch_one<K, 0, 1, false, EPI_MATCHED>(in, out, tw, spec, a, s);
    } else {
        if (out_st != 0) return hipErrorInvalidValue;
        return in_st == 0 ? launch_one<K, 0, 0, false, EPI_MATCHED>(in, out, tw, spec, a, s)
                          : launch_one<K, 1, 0, false, EPI_MATCHED>(in, out, tw, spec, a, s);
    }
}

template <class K>
hipError_t dispatch_cfg(int in_st, int out_st, int inv, int epi, const void *in, void *out, const float2 *tw,
                        const float2 *spec, const KArgs &a, hipStream_t s) {
    if constexpr (K::XCHG == XCHG_LANE) {
        // the cross-lane exchange: plain row transforms, either storage
        if (epi != EPI_NONE || in_st != out_st) return hipErrorInvalidValue;
        if (in_st == 0)
            return inv ? launch_one<K, 0, 0, true, EPI_NONE>(in, out, tw, spec, a, s)
                       : launch_one<K, 0, 0, false, EPI_NONE>(in, out, tw, spec, a, s);
        return inv ? launch_one<K, 1, 1, true, EPI_NONE>(in, out, tw, spec, a, s)
                   : launch_one<K, 1, 1, false, EPI_NONE>(in, out, tw, spec, a, s);
    } else if constexpr (K::XCHG == XCHG_HALF) {
        // the binary16 exchange: FP16 storage, plain transforms only
        if (epi != EPI_NONE || in_st != 1 || out_st != 1) return hipErrorInvalidValue;
        return inv ? launch_one<K, 1, 1, true, EPI_NONE>(in, out, tw, spec, a, s)
                   : launch_one<K, 1, 1, false, EPI_NONE>(in, out, tw, spec, a, s);
    } else {
        return dispatch_cfg_full<K>(in_st, out_st, inv, epi, in, out, tw, spec, a, s);
    }
}

template <class K>
hipError_t dispatch_rcmc(int in_st, int out_st, int inv, const void *in, void *out, const float2 *tw,
                         const float2 *spec, const KArgs &a, hipStream_t s) {
    if (!inv || out_st != 0) return hipErrorInvalidValue;
    return in_st == 0 ? launch_one<K, 0, 0, true, EPI_RCMC>(in, out, tw, spec, a, s)
                      : launch_one<K, 1, 0, true, EPI_RCMC>(in, out, tw, spec, a, s);
}

template <int N>
hipError_t dispatch(int variant, int layout, int in_st, int out_st, int inv, int epi, const void *in, void *out,
                    const float2 *tw, const float2 *spec, const KArgs &a, hipStream_t s) {
    auto f = [&](auto k) { return dispatch_cfg<decltype(k)>(in_st, out_st, inv, epi, in, out, tw, spec, a, s); };
    if (layout == LAYOUT_ROWS_HALF) {
        if constexpr (N >= 1024) {
            return with_variant(variant >= 0 ? variant : 0, typename Configs<N>::RowsHalf{}, f);
        } else {
            return hipErrorInvalidValue;
        }
    }
    if (layout == LAYOUT_RCMC) {
        if constexpr (N >= 1024) {
            if (epi != EPI_RCMC) return hipErrorInvalidValue;
            auto g = [&](auto k) { return dispatch_rcmc<decltype(k)>(in_st, out_st, inv, in, out, tw, spec, a, s); };
            return with_variant(variant >= 0 ? variant : 0, typename Configs<N>::Rcmc{}, g);
        } else {
            return hipErrorInvalidValue;
        }
    }
    const int half = (in_st | out_st) != 0;  // any FP16 storage involved
    const bool mf = epi == EPI_MATCHED || epi == EPI_MATCHED_Y;
    if (layout == LAYOUT_ROWS) {
        int v = variant >= 0 ? variant : mf ? Configs<N>::kRowMatched[half] : Configs<N>::kRowDefault[half];
        if (variant < 0 && !mf && epi == EPI_NONE && a.batch < SmallRows<N>::below) v = SmallRows<N>::variant;
        return with_variant(v, typename Configs<N>::Rows{}, f);
    }
    using Cols = typename Configs<N>::Cols;
    static_assert(KAt<FourStepCols<N>::plain[0], Cols>::type::P <= 32 &&
                      KAt<FourStepCols<N>::plain[1], Cols>::type::P <= 32 &&
                      KAt<FourStepCols<N>::matched, Cols>::type::P <= 32,
                  "the four-step epilogues hold at most 32 points per thread");
    const bool four_step = epi == EPI_TWIDDLE || epi == EPI_TWIDDLE_Y || epi == EPI_MATCHED_Y;
    int v = variant;
    if (v < 0) {
        if (four_step) {
            v = mf ? FourStepCols<N>::matched : FourStepCols<N>::plain[half];
        } else if (epi == EPI_SCALE) {
            v = ScaleCols<N>::v[half];
        } else {
            v = mf ? Configs<N>::kColMatched[half] : Configs<N>::kColDefault[half];
        }
    }
    return with_variant(v, Cols{}, f);
}

template <int N>
int variant_count(int layout) {
    return layout == LAYOUT_ROWS   ? KListSize<typename Configs<N>::Rows>::value
           : layout == LAYOUT_COLS ? KListSize<typename Configs<N>::Cols>::value
           : layout == LAYOUT_RCMC ? KListSize<typename Configs<N>::Rcmc>::value
                                   : KListSize<typename Configs<N>::RowsHalf>::value;
}

}  // namespace mi355fft
