// fft_mfma.hpp -- FP16-storage FFT whose radix-16 butterflies run on the
// matrix cores (Section VIII: a radix-r stage as a dense DFT matrix times the
// data, the twiddles applied per column between stages).
//
// A radix-16 stage over N/16 butterflies is the real 32 x 32 matrix of the
// 16-point DFT (rows 2k'+{re,im} of the outputs, columns 2r+{re,im} of the
// inputs) times a 32 x (N/16) data matrix.  One v_mfma_f32_32x32x16_f16 takes
// 32 butterflies (a tile) and half of the 32 input rows, so a tile is four
// instructions: the two halves of the inputs, each against the matrix split
// into a binary16 high part and the binary16 rounding of the rest (their sum
// is the FP32 matrix to about 2^-22, so the matrix adds no error of its own).
// The data enter each stage as binary16 (the one rounding per stage of this
// form; the paper's matrix-unit kernel measured 66 dB) and leave it in FP32,
// where the next stage's twiddles are applied before rounding again.
//
// Section VIII's bound: a dense radix-r block pays only when the unit's rate
// exceeds the vector units' by 8r / (5 log2 r), 6.4x at r = 16.  MI355X's
// dense FP16 matrix rate (2.5 PFLOP/s) is about 32x its unpacked FP32 vector
// rate, so the bound passes; and the FP16-storage transforms are bound by
// vector issue, not by memory (their vector kernels issue 53-63 instructions
// per point), so moving the butterflies to the matrix cores is what could pay.
// Measured, it does not: with 1 GiB batches from HBM this kernel takes 1.1x
// (N = 4096) and 1.6x (N = 16384) the time of the vector kernels.  The
// matrix form removes only 5-16% of the vector instructions per transform,
// because the operand packing (FP32 -> binary16 fragments), the twiddles and
// the Stockham moves through LDS stay on the vector units; the matrix cores
// are busy about a fifth of the time.  It is kept as an opt-in plan flag.
//
// Operand layouts of v_mfma_f32_32x32x16_f16 (wave64, checked on the device):
// lane l holds A[l % 32][8 (l / 32) + e] and B[8 (l / 32) + e][l % 32] for
// e = 0..7, and C register j holds row 8 (j / 4) + 4 (l / 32) + j % 4 of
// column l % 32.  So lane l of a tile works on butterfly j = 32 tile + l % 32:
// it supplies inputs r = 4h..4h+3 (first instruction pair) and 8+4h..8+4h+3
// (second pair), h = l / 32, and receives outputs k' = 4q + 2h + {0, 1},
// q = 0..3 (registers 4q .. 4q+3 as (re, im, re, im)).
//
// Stockham order as in the vector kernels: butterfly j of a stage with
// sub-transforms of length NS reads positions j + r N/16 and writes output k'
// to ((j / NS) NS + ... ) = (j / NS) 16 NS + j % NS + k' NS; the first stage
// reads the input directly, and the last writes natural order directly.  An
// optional final stage of radix 2, 4 or 8 runs on the vector units.
#pragma once

#include "fft_kernel.hpp"

namespace mi355fft {

typedef _Float16 mf_half8 __attribute__((ext_vector_type(8)));
typedef float mf_float16 __attribute__((ext_vector_type(16)));

// The lane fragments of the 32 x 32 real DFT matrix come from a table the
// host computes once per device (double precision, split into binary16 hi and
// lo parts): for direction d (0 forward, 1 inverse), lane l and input half s,
// entries [((d * 64 + l) * 2 + s) * 2 + {0 hi, 1 lo}] hold A[l % 32][16 s +
// 8 (l / 32) + e], e = 0..7, as eight binary16 values.  Row 2k' + co, column
// 2r + ci of the forward matrix: c = cos(2 pi k' r / 16), s = sin(...):
// [c, s; -s, c] (y = (c - i s) x); the inverse flips the sign of s.
constexpr int kMfmaMatrixHalf8 = 2 * 64 * 2 * 2;  // mf_half8 entries

template <int N_, int R0_, int WAVES_>
struct MfmaCfg {
    static constexpr int N = N_, R0 = R0_, WAVES = WAVES_, THREADS = 64 * WAVES_;
    static constexpr int NB = N_ / 16;  // butterflies of a radix-16 stage
    static constexpr int S16 = ilog2(N_ / R0_) / 4;  // radix-16 stages
    static constexpr int TILES = NB / 32;
    static_assert((1 << (4 * S16)) * R0_ == N_, "N = 16^S16 * R0");
    static_assert(TILES % WAVES_ == 0, "tiles split evenly over the waves");
    static constexpr int LDS_SLOTS = N_ + (N_ >> 4);  // complex FP32, one pad slot per 16
};

__device__ __forceinline__ int mf_pad(int p) { return p + (p >> 4); }

// W_{16 NS}^{jm r} for this lane's eight inputs r = 4h + e and 8 + 4h + e
// (e = 0..3), jm = j mod NS, from two table reads (W^jm, W^4jm) and products.
template <int N, int NS, bool INV>
__device__ __forceinline__ void stage_twiddles(const float2 *__restrict__ tw, int jm, int h, float2 (&w)[8]) {
    constexpr int STR = N / (16 * NS);
    const float2 a = tw[jm * STR], b = tw[4 * jm * STR];
    const float2 a2 = cmul(a, a), a3 = cmul(a2, a), b2 = cmul(b, b);
    const float2 bh = h ? b : make_float2(1.0f, 0.0f);
    const float2 bh2 = cmul(b2, bh);
    w[0] = bh;
    w[1] = cmul(bh, a);
    w[2] = cmul(bh, a2);
    w[3] = cmul(bh, a3);
    w[4] = bh2;
    w[5] = cmul(bh2, a);
    w[6] = cmul(bh2, a2);
    w[7] = cmul(bh2, a3);
    if constexpr (INV) {
        static_for<0, 8>([&](auto ic) { w[ic].y = -w[ic].y; });
    }
}

__device__ __forceinline__ unsigned pack_half2(float2 v) { return Store<1>::narrow(v); }

// One radix-16 stage (NS = 16^s) on the matrix cores.  FIRST reads the FP16
// input, LAST writes the FP16 output; otherwise LDS (FP32) to LDS, in place:
// every wave first turns all its tiles' inputs into binary16 B fragments
// (eight registers per tile), then a barrier, then the products and the
// writes, so no write lands on a position another wave has still to read.
template <class M, int NS, bool INV, bool FIRST, bool LAST>
__device__ __forceinline__ void mfma_stage(const mf_half8 (&ahi)[2], const mf_half8 (&alo)[2], int lane, int wave,
                                           const rsrc_t &rin, const rsrc_t &rout, const float2 *__restrict__ tw,
                                           float2 *L) {
    constexpr int NB = M::NB, TPW = M::TILES / M::WAVES;
    const int h = lane >> 5;
    mf_half8 b0[TPW], b1[TPW];
    static_for<0, TPW>([&](auto tc) {
        constexpr int ti = decltype(tc)::value;
        const int j = 32 * (wave * TPW + ti) + (lane & 31);
        typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
        if constexpr (FIRST) {
            // inputs r = 4h + e and 8 + 4h + e of butterfly j, straight from
            // memory: the stored binary16 pairs are the operand as they are
            const unsigned v0 = (unsigned)((j + 4 * h * NB) * 4), v1 = (unsigned)((j + (8 + 4 * h) * NB) * 4);
            u32x4 p0, p1;
            static_for<0, 4>([&](auto ec) {
                constexpr int e = decltype(ec)::value;
                p0[e] = __builtin_amdgcn_raw_buffer_load_b32(rin, v0, (unsigned)(e * NB * 4), 0);
                p1[e] = __builtin_amdgcn_raw_buffer_load_b32(rin, v1, (unsigned)(e * NB * 4), 0);
            });
            b0[ti] = __builtin_bit_cast(mf_half8, p0);
            b1[ti] = __builtin_bit_cast(mf_half8, p1);
        } else {
            float2 x[8];
            static_for<0, 4>([&](auto ec) {
                constexpr int e = decltype(ec)::value;
                x[e] = L[mf_pad(j + (4 * h + e) * NB)];
                x[4 + e] = L[mf_pad(j + (8 + 4 * h + e) * NB)];
            });
            float2 w[8];
            stage_twiddles<M::N, NS, INV>(tw, j & (NS - 1), h, w);
            static_for<0, 8>([&](auto ic) { x[ic] = cmul(x[ic], w[ic]); });
            // each complex value becomes one packed binary16 pair (one conversion)
            const u32x4 p0 = {pack_half2(x[0]), pack_half2(x[1]), pack_half2(x[2]), pack_half2(x[3])};
            const u32x4 p1 = {pack_half2(x[4]), pack_half2(x[5]), pack_half2(x[6]), pack_half2(x[7])};
            b0[ti] = __builtin_bit_cast(mf_half8, p0);
            b1[ti] = __builtin_bit_cast(mf_half8, p1);
        }
    });
    if constexpr (!FIRST && !LAST) __syncthreads();  // every input of this stage read
    static_for<0, TPW>([&](auto tc) {
        constexpr int ti = decltype(tc)::value;
        const int j = 32 * (wave * TPW + ti) + (lane & 31);
        mf_float16 acc = {};
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(ahi[0], b0[ti], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(alo[0], b0[ti], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(ahi[1], b1[ti], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(alo[1], b1[ti], acc, 0, 0, 0);
        const int base = (j / NS) * 16 * NS + (j & (NS - 1));
        static_for<0, 8>([&](auto qc) {
            constexpr int q = decltype(qc)::value;  // output k' = 4 (q / 2) + 2h + q % 2
            const int kp = 4 * (q / 2) + 2 * h + (q % 2);
            const float2 y = make_float2(acc[2 * q], acc[2 * q + 1]);
            if constexpr (LAST) {
                Store<1>::template store<false>(rout, (unsigned)((base + kp * NS) * 4), 0u, y);
            } else {
                L[mf_pad(base + kp * NS)] = y;
            }
        });
    });
}

template <class M, bool INV, int NS, int S>
__device__ __forceinline__ void mfma_stages(const mf_half8 (&ahi)[2], const mf_half8 (&alo)[2], int lane, int wave,
                                            const rsrc_t &rin, const rsrc_t &rout, const float2 *__restrict__ tw,
                                            float2 *L) {
    constexpr bool FIRST = NS == 1, LAST = S == M::S16 - 1 && M::R0 == 1;
    mfma_stage<M, NS, INV, FIRST, LAST>(ahi, alo, lane, wave, rin, rout, tw, L);
    if constexpr (S + 1 < M::S16) {
        __syncthreads();
        mfma_stages<M, INV, NS * 16, S + 1>(ahi, alo, lane, wave, rin, rout, tw, L);
    }
}

// The final radix-R0 stage on the vector units (NS = N / R0): butterfly j
// reads j + r N/R0, multiplies by W_N^{j r}, and writes natural order.
template <class M, bool INV>
__device__ __forceinline__ void vector_last_stage(int tid, const rsrc_t &rout, const float2 *__restrict__ tw,
                                                  const float2 *L) {
    constexpr int R = M::R0, NS = M::N / R;
    for (int j = tid; j < NS; j += M::THREADS) {
        float2 u[R];
        static_for<0, R>([&](auto rc) {
            constexpr int r = decltype(rc)::value;
            u[r] = L[mf_pad(j + r * NS)];
            if constexpr (r > 0) {
                const float2 w = tw[j * r];
                u[r] = INV ? cmulc(u[r], w) : cmul(u[r], w);
            }
        });
        Dft<R, INV>::run(u);
        static_for<0, R>([&](auto rc) {
            constexpr int r = decltype(rc)::value;
            Store<1>::template store<false>(rout, (unsigned)((j + r * NS) * 4), 0u, u[r]);
        });
    }
}

// One FP16 transform per workgroup, rows (stride 1, distance a.in_dist).
template <class M, bool INV>
__global__ __launch_bounds__(M::THREADS) void fft_mfma_kernel(const void *__restrict__ in, void *__restrict__ out,
                                                              const float2 *__restrict__ tw,
                                                              const mf_half8 *__restrict__ amat, KArgs a) {
    __shared__ float2 L[M::LDS_SLOTS];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const long long b = blockIdx.x;
    const rsrc_t rin = make_rsrc(reinterpret_cast<const char *>(in) + b * a.in_dist * 4, (unsigned)(M::N * 4));
    const rsrc_t rout = make_rsrc(reinterpret_cast<char *>(out) + b * a.out_dist * 4, (unsigned)(M::N * 4));
    const mf_half8 *am = amat + (((INV ? 1 : 0) * 64 + lane) * 2) * 2;
    const mf_half8 ahi[2] = {am[0], am[2]}, alo[2] = {am[1], am[3]};
    mfma_stages<M, INV, 1, 0>(ahi, alo, lane, wave, rin, rout, tw, L);
    if constexpr (M::R0 > 1) {
        __syncthreads();
        vector_last_stage<M, INV>(tid, rout, tw, L);
    }
}

template <class M>
hipError_t launch_mfma(int inv, const void *in, void *out, const float2 *tw, const void *amat, const KArgs &a,
                       hipStream_t s) {
    const mf_half8 *am = reinterpret_cast<const mf_half8 *>(amat);
    if (a.batch <= 0 || a.batch > 0x7fffffffLL || a.stride != 1) return hipErrorInvalidValue;
    if (a.in_dist < M::N || a.out_dist < M::N) return hipErrorInvalidValue;
    return launch_kernel(inv ? fft_mfma_kernel<M, true> : fft_mfma_kernel<M, false>, dim3((unsigned)a.batch),
                         dim3(M::THREADS), s, in, out, tw, am, a);
}

}  // namespace mi355fft
