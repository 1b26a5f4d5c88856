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
template <int STORAGE>
struct Store;

template <>
struct Store<0> {  // complex FP32, 8 bytes
    using T = float2;
    __device__ __forceinline__ static float2 load(const T *p) { return *p; }
    template <bool NT>
    __device__ __forceinline__ static void store(T *p, float2 v) {
        if constexpr (NT) {
            __builtin_nontemporal_store(__builtin_bit_cast(unsigned long long, v),
                                        reinterpret_cast<unsigned long long *>(p));
        } else {
            *p = v;
        }
    }
};

template <>
struct Store<1> {  // complex FP16 (binary16 pair), 4 bytes; FP32 arithmetic
    using T = __half2;
    __device__ __forceinline__ static float2 load(const T *p) {
        const unsigned int bits = *reinterpret_cast<const unsigned int *>(p);
        const _Float16 lo = __builtin_bit_cast(_Float16, (unsigned short)(bits & 0xffffu));
        const _Float16 hi = __builtin_bit_cast(_Float16, (unsigned short)(bits >> 16));
        return make_float2((float)lo, (float)hi);
    }
    template <bool NT>
    __device__ __forceinline__ static void store(T *p, float2 v) {
        // round to nearest even (the conversion's default rounding mode)
        const unsigned short lo = __builtin_bit_cast(unsigned short, (_Float16)v.x);
        const unsigned short hi = __builtin_bit_cast(unsigned short, (_Float16)v.y);
        const unsigned int bits = (unsigned int)lo | ((unsigned int)hi << 16);
        if constexpr (NT) {
            __builtin_nontemporal_store(bits, reinterpret_cast<unsigned int *>(p));
        } else {
            *reinterpret_cast<unsigned int *>(p) = bits;
        }
    }
};

}  // namespace mi355fft
