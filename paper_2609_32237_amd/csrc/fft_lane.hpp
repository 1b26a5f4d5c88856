// fft_lane.hpp -- the 1024-point transform held by one wavefront, with every
// exchange between stages made across the 64 lanes instead of through LDS.
//
// Section VI exchanges data between radix stages through threadgroup memory,
// with a barrier per exchange.  When one 64-lane wave holds a whole transform
// (1024 points, 16 per lane) every exchange stays inside the wave, and each
// one is a transpose of index bits between the register number and the lane
// number:
//   lane bit 5 or 4  v_permlane32_swap / v_permlane16_swap: one instruction
//                    swaps the upper half of one register with the lower half
//                    of another (1 VALU instruction per point and bit);
//   lane bit 3 or 2  a DPP row shift by 8 or 4 lanes whose bank mask enables
//                    only the lanes that receive (2 per point and bit);
//   lane bit 1 or 0  a DPP quad permutation and a select (2 to 4 per point
//                    and bit).
// There is no LDS traffic and no barrier, at the cost of these VALU moves.
//
// Index bookkeeping (p = position 0..1023, L = lane, i = register):
//   load      register i of lane L holds p = L + 64 i (canonical);
//   stage 1   radix 16 on sub-transforms of length 1: butterfly L, outputs
//             p = 16 L + r in register r;
//   exchange  register bits 0..3 <-> lane bits 2..5: register i then holds
//             p with bits 6..9 = i, bits 0..3 = L >> 2, bits 4..5 = L & 3;
//   stage 2   radix 16 on sub-transforms of length 16: butterfly
//             j = (L >> 2) + 16 (L & 3), outputs (j >> 4) 256 + (j & 15) + 16 r;
//   exchange  register bits 0..1 <-> lane bits 0..1: register r + 4 q then
//             holds p = (L >> 2) + 16 (L & 3) + 64 q + 256 r;
//   stage 3   radix 4 on sub-transforms of length 256: four butterflies
//             j = (L >> 2) + 16 (L & 3) + 64 q, outputs j + 256 r in register
//             r + 4 q: the natural-order result, in that lane order (each
//             register still covers 64 consecutive points, so the store stays
//             one contiguous 512-byte piece per register).
#pragma once

#include "fft_device.hpp"

namespace mi355fft {

// Transpose register bit RB with lane bit LB across the wave: for every
// register pair (i, i + 2^RB) with register bit RB clear, the lanes whose bit
// LB is set exchange their value of register i with their partner lane's
// value of register i + 2^RB.  Afterwards register i' of lane L' holds what
// register (i' with bit RB := bit LB of L') of lane (L' with bit LB := bit RB
// of i') held.
__device__ __forceinline__ unsigned fbits(float x) { return __builtin_bit_cast(unsigned, x); }
__device__ __forceinline__ float ffloat(unsigned x) { return __builtin_bit_cast(float, x); }

template <int LB>
__device__ __forceinline__ void lane_swap_pair(float &x, float &y, int lane) {
    if constexpr (LB == 5 || LB == 4) {
        // v_permlaneN_swap(x, y): x keeps its lower lanes and takes y's lower
        // lanes into its upper ones; y takes x's upper lanes into its lower ones
        const auto r = LB == 5 ? __builtin_amdgcn_permlane32_swap(fbits(x), fbits(y), false, false)
                               : __builtin_amdgcn_permlane16_swap(fbits(x), fbits(y), false, false);
        x = ffloat(r[0]);
        y = ffloat(r[1]);
    } else if constexpr (LB == 3 || LB == 2) {
        // row_shr:n (lane l reads lane l - n) into the lanes with the bit set,
        // row_shl:n (lane l reads lane l + n) into the lanes with it clear;
        // the bank mask (four-lane banks of each 16-lane row) leaves the other
        // lanes holding their old value
        constexpr int SHR = LB == 3 ? 0x118 : 0x114, SHL = LB == 3 ? 0x108 : 0x104;
        constexpr int HI = LB == 3 ? 0xC : 0xA, LO = LB == 3 ? 0x3 : 0x5;
        const int nx = __builtin_amdgcn_update_dpp((int)fbits(x), (int)fbits(y), SHR, 0xF, HI, false);
        const int ny = __builtin_amdgcn_update_dpp((int)fbits(y), (int)fbits(x), SHL, 0xF, LO, false);
        x = ffloat((unsigned)nx);
        y = ffloat((unsigned)ny);
    } else {
        static_assert(LB == 1 || LB == 0, "lane bits 0..5");
        // quad permutation l ^ 2^LB, then keep the old value where it stays
        constexpr int QP = LB == 0 ? 0xB1 : 0x4E;  // [1,0,3,2] or [2,3,0,1]
        const float px = ffloat((unsigned)__builtin_amdgcn_mov_dpp((int)fbits(x), QP, 0xF, 0xF, false));
        const float py = ffloat((unsigned)__builtin_amdgcn_mov_dpp((int)fbits(y), QP, 0xF, 0xF, false));
        const bool set = (lane >> LB) & 1;
        x = set ? py : x;
        y = set ? y : px;
    }
}

template <int RB, int LB, int P>
__device__ __forceinline__ void lane_transpose_bit(float2 (&v)[P], int lane) {
    static_for<0, P>([&](auto ic) {
        constexpr int i = decltype(ic)::value;
        if constexpr (((i >> RB) & 1) == 0) {
            constexpr int j = i | (1 << RB);
            lane_swap_pair<LB>(v[i].x, v[j].x, lane);
            lane_swap_pair<LB>(v[i].y, v[j].y, lane);
        }
    });
}

// The 1024-point transform of one wave (layout above), forward or inverse.
// tw is the 1024-entry twiddle table; K supplies the twiddle mode.
template <class K, bool INV>
__device__ __forceinline__ void lane_fft_1024(float2 (&v)[16], int lane, const float2 *__restrict__ tw) {
    static_assert(K::N == 1024 && K::P == 16 && K::T == 64, "one wave holds one 1024-point transform");
    // stage 2's twiddles W_256^(k r), k = L >> 2: requested before stage 1
    const int j2 = (lane >> 2) + ((lane & 3) << 4);
    TwRegs<K, 16, 16> tw2;
    tw_issue<K, 16, 16>(tw2, j2, tw);
    // stage 1: radix 16, no twiddles
    Dft<16, INV>::run(v);
    // exchange: register bits 0..3 <-> lane bits 2..5
    lane_transpose_bit<0, 2>(v, lane);
    lane_transpose_bit<1, 3>(v, lane);
    lane_transpose_bit<2, 4>(v, lane);
    lane_transpose_bit<3, 5>(v, lane);
    // stage 3's twiddles W_1024^(j r), j = base + 64 q (base < 64 = T)
    const int base = j2;
    TwRegs<K, 256, 4> tw3;
    tw_issue<K, 256, 4>(tw3, base, tw);
    // stage 2: radix 16 on sub-transforms of length 16
    tw_apply<K, 16, 16, 0, INV>(tw2, v);
    Dft<16, INV>::run(v);
    // exchange: register bits 0..1 <-> lane bits 0..1
    lane_transpose_bit<0, 0>(v, lane);
    lane_transpose_bit<1, 1>(v, lane);
    // stage 3: radix 4, butterfly q on registers 4q .. 4q + 3
    static_for<0, 4>([&](auto qc) {
        constexpr int q = decltype(qc)::value;
        float2 u[4];
        static_for<0, 4>([&](auto rc) { u[rc] = v[4 * q + rc]; });
        tw_apply<K, 256, 4, q, INV>(tw3, u);
        Dft<4, INV>::run(u);
        static_for<0, 4>([&](auto rc) { v[4 * q + rc] = u[rc]; });
    });
}

// Position of register i of lane L after lane_fft_1024.
__device__ __forceinline__ int lane_base_1024(int lane) { return (lane >> 2) + ((lane & 3) << 4); }
template <int I>
constexpr int lane_reg_pos_1024() {
    return 64 * (I >> 2) + 256 * (I & 3);
}

}  // namespace mi355fft
