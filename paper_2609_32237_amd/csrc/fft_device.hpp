// fft_device.hpp -- device building blocks of the single-pass FFT kernels.
//
// One workgroup owns whole transforms (Section VI: one threadgroup per
// transform, every point read once and written once).  Each thread keeps P
// complex FP32 values in VGPRs; a stage of radix R runs P/R register
// butterflies per thread, multiplies by the inter-stage twiddles, and the
// stages exchange data through LDS.  The formulation is the Stockham
// autosort one, so results come out in natural order with no reordering pass.
//
// Canonical register layout: thread t of a transform holds position t + T*i
// in register i (T = N/P threads per transform).  Every stage reads its
// butterfly inputs from that layout, and the last stage's outputs land in it
// again, so the global load, the global store and a fused inverse transform
// (which starts from the same layout) need no reshuffle.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <type_traits>
#include <utility>

namespace mi355fft {

// --------------------------------------------------------------------------
// compile-time helpers
// --------------------------------------------------------------------------

template <int I, int E, class F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (I < E) {
        f(std::integral_constant<int, I>{});
        static_for<I + 1, E>(f);
    }
}

constexpr int ilog2(int x) { return x <= 1 ? 0 : 1 + ilog2(x >> 1); }

// cos(2 pi j / 64) for j = 0..16 (first quadrant of the 64th roots of unity).
constexpr float kCos64[17] = {
    1.0f,
    0.99518472667219688624f,
    0.98078528040323044913f,
    0.95694033573220886494f,
    0.92387953251128675613f,
    0.88192126434835502971f,
    0.83146961230254523708f,
    0.77301045336273696081f,
    0.70710678118654752440f,
    0.63439328416364549822f,
    0.55557023301960222474f,
    0.47139673682599764856f,
    0.38268343236508977173f,
    0.29028467725446236764f,
    0.19509032201612826785f,
    0.098017140329560601994f,
    0.0f,
};

constexpr float cos64(int j) {
    j &= 63;
    return j <= 16 ? kCos64[j] : j <= 32 ? -kCos64[32 - j] : j <= 48 ? -kCos64[j - 32] : kCos64[64 - j];
}
constexpr float sin64(int j) { return cos64(j - 16); }

// --------------------------------------------------------------------------
// complex FP32 arithmetic on float2 = (re, im)
// --------------------------------------------------------------------------

__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float2 cmul(float2 a, float2 w) {
    return make_float2(a.x * w.x - a.y * w.y, a.x * w.y + a.y * w.x);
}
// a * conj(w)
__device__ __forceinline__ float2 cmulc(float2 a, float2 w) {
    return make_float2(a.x * w.x + a.y * w.y, a.y * w.x - a.x * w.y);
}

// a * W_R^M with W_R = exp(-2 pi i / R) (forward) or its conjugate (inverse).
// Multiples of pi/4 are special-cased so the unit factors cost no multiply.
template <int R, int M, bool INV>
__device__ __forceinline__ float2 twiddle_const(float2 a) {
    constexpr int m = ((M % R) + R) % R;
    if constexpr (m == 0) {
        return a;
    } else if constexpr ((8 * m) % R == 0) {
        constexpr int e = (8 * m) / R;  // angle = -e * pi / 4 (forward)
        constexpr float h = 0.70710678118654752440f;
        // forward factor exp(-i e pi/4); inverse uses +e
        constexpr int ee = INV ? (8 - e) % 8 : e;
        if constexpr (ee == 2) return make_float2(a.y, -a.x);   // * -i
        if constexpr (ee == 4) return make_float2(-a.x, -a.y);  // * -1
        if constexpr (ee == 6) return make_float2(-a.y, a.x);   // * +i
        if constexpr (ee == 1) return make_float2((a.x + a.y) * h, (a.y - a.x) * h);    // (1-i)/sqrt2
        if constexpr (ee == 3) return make_float2((a.y - a.x) * h, -(a.x + a.y) * h);   // (-1-i)/sqrt2
        if constexpr (ee == 5) return make_float2(-(a.x + a.y) * h, (a.x - a.y) * h);   // (-1+i)/sqrt2
        if constexpr (ee == 7) return make_float2((a.x - a.y) * h, (a.x + a.y) * h);    // (1+i)/sqrt2
    } else {
        static_assert(64 % R == 0, "constant twiddles cover radices dividing 64");
        constexpr int j = m * (64 / R);
        constexpr float c = cos64(j);
        constexpr float s = INV ? sin64(j) : -sin64(j);
        return make_float2(a.x * c - a.y * s, a.x * s + a.y * c);
    }
}

// --------------------------------------------------------------------------
// small DFTs in registers: X[k] = sum_n x[n] W_R^{nk}, in place
// --------------------------------------------------------------------------

template <int R, bool INV>
struct Dft;

template <bool INV>
struct Dft<2, INV> {
    __device__ __forceinline__ static void run(float2 *v) {
        float2 a = v[0], b = v[1];
        v[0] = cadd(a, b);
        v[1] = csub(a, b);
    }
};

template <bool INV>
struct Dft<4, INV> {
    __device__ __forceinline__ static void run(float2 *v) {
        float2 t0 = cadd(v[0], v[2]), t1 = csub(v[0], v[2]);
        float2 t2 = cadd(v[1], v[3]), t3 = twiddle_const<4, 1, INV>(csub(v[1], v[3]));
        v[0] = cadd(t0, t2);
        v[2] = csub(t0, t2);
        v[1] = cadd(t1, t3);
        v[3] = csub(t1, t3);
    }
};

// Composite R = R1 * R2: n = R2*n1 + n2, k = k1 + R1*k2.
//   Y[n2][k1] = DFT_R1 over n1 of x[R2*n1 + n2], times W_R^{n2*k1};
//   X[k1 + R1*k2] = DFT_R2 over n2 of Y[n2][k1].
template <int R>
struct DftSplit {
    static constexpr int R1 = R == 8 ? 2 : R == 16 ? 4 : R == 32 ? 4 : 8;
    static constexpr int R2 = R / R1;
};

template <int R, bool INV>
struct Dft {
    static_assert(R == 8 || R == 16 || R == 32 || R == 64, "unsupported radix");
    __device__ __forceinline__ static void run(float2 *v) {
        constexpr int R1 = DftSplit<R>::R1, R2 = DftSplit<R>::R2;
        float2 y[R];
        static_for<0, R2>([&](auto n2c) {
            constexpr int n2 = decltype(n2c)::value;
            float2 u[R1];
            static_for<0, R1>([&](auto n1c) { u[n1c] = v[R2 * n1c + n2]; });
            Dft<R1, INV>::run(u);
            static_for<0, R1>([&](auto k1c) {
                constexpr int k1 = decltype(k1c)::value;
                y[n2 * R1 + k1] = twiddle_const<R, n2 * k1, INV>(u[k1]);
            });
        });
        static_for<0, R1>([&](auto k1c) {
            constexpr int k1 = decltype(k1c)::value;
            float2 u[R2];
            static_for<0, R2>([&](auto n2c) { u[n2c] = y[n2c * R1 + k1]; });
            Dft<R2, INV>::run(u);
            static_for<0, R2>([&](auto k2c) { v[k1 + R1 * k2c] = u[k2c]; });
        });
    }
};

// --------------------------------------------------------------------------
// storage conversions
// --------------------------------------------------------------------------

// Every point is read once and written once.  Final results are stored with
// the non-temporal hint (measured faster for outputs far larger than the
// caches); intermediates that the next kernel reads soon are stored normally
// so they can stay in the 256 MiB Infinity Cache.  Loads carry no hint (the
// hint measured slower on loads).
//
// Two addressing forms: raw buffer accesses (a per-workgroup resource built
// from a uniform base, one 32-bit lane offset, and a scalar offset per
// register: no per-access vector address arithmetic), and plain 64-bit
// pointers for layouts whose per-workgroup span does not fit 31 bits.
using rsrc_t = __amdgpu_buffer_rsrc_t;
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
constexpr int kBufferFlags = 0x00020000;  // raw buffer, 32-bit data format
constexpr int kNtAux = 2;                 // cache-policy bit of the non-temporal hint

__device__ __forceinline__ rsrc_t make_rsrc(const void *base, unsigned bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, kBufferFlags);
}

template <int STORAGE>
struct Store;

template <>
struct Store<0> {  // complex FP32, 8 bytes
    using T = float2;
    static constexpr int BYTES = 8;
    __device__ __forceinline__ static float2 load(const T *p) { return *p; }
    __device__ __forceinline__ static float2 load(rsrc_t r, unsigned voff, unsigned soff) {
        return __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
    }
    template <bool NT>
    __device__ __forceinline__ static void store(T *p, float2 v) {
        if constexpr (NT) {
            __builtin_nontemporal_store(__builtin_bit_cast(unsigned long long, v),
                                        reinterpret_cast<unsigned long long *>(p));
        } else {
            *p = v;
        }
    }
    template <bool NT>
    __device__ __forceinline__ static void store(rsrc_t r, unsigned voff, unsigned soff, float2 v) {
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2_t, v), r, voff, soff, NT ? kNtAux : 0);
    }
};

template <>
struct Store<1> {  // complex FP16 (binary16 pair), 4 bytes; FP32 arithmetic
    using T = __half2;
    static constexpr int BYTES = 4;
    __device__ __forceinline__ static float2 widen(unsigned int bits) {
        const f32x2_t f = __builtin_convertvector(__builtin_bit_cast(f16x2_t, bits), f32x2_t);
        return make_float2(f.x, f.y);
    }
    // round to nearest even (the conversion's default rounding mode)
    __device__ __forceinline__ static unsigned int narrow(float2 v) {
        return __builtin_bit_cast(unsigned int, __builtin_convertvector((f32x2_t){v.x, v.y}, f16x2_t));
    }
    __device__ __forceinline__ static float2 load(const T *p) { return widen(*reinterpret_cast<const unsigned *>(p)); }
    __device__ __forceinline__ static float2 load(rsrc_t r, unsigned voff, unsigned soff) {
        return widen(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
    }
    template <bool NT>
    __device__ __forceinline__ static void store(T *p, float2 v) {
        if constexpr (NT) {
            __builtin_nontemporal_store(narrow(v), reinterpret_cast<unsigned int *>(p));
        } else {
            *reinterpret_cast<unsigned int *>(p) = narrow(v);
        }
    }
    template <bool NT>
    __device__ __forceinline__ static void store(rsrc_t r, unsigned voff, unsigned soff, float2 v) {
        __builtin_amdgcn_raw_buffer_store_b32(narrow(v), r, voff, soff, NT ? kNtAux : 0);
    }
};

}  // namespace mi355fft
