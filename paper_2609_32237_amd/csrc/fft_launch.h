// fft_launch.h -- host-visible interface between the C ABI runtime and the
// kernel instantiations (one translation unit per transform size).
#pragma once

#include <hip/hip_runtime.h>

namespace mi355fft {

enum { LAYOUT_ROWS = 0, LAYOUT_COLS = 1 };
enum { EPI_NONE = 0, EPI_MATCHED = 1 };

struct KArgs {
    long long batch;     // transforms
    long long stride;    // elements between points of a transform (input and output)
    long long in_dist;   // elements between transform starts in the input
    long long out_dist;  // elements between transform starts in the output
    float scale;         // epilogue scale
    int xcd_remap;       // 1: map blocks so consecutive strips share an XCD
    int wide;            // 1: 64-bit pointer addressing (span or sign does not fit buffer offsets)
    unsigned in_span;    // bytes one workgroup's input occupies (buffer addressing)
    unsigned out_span;   // bytes one workgroup's output occupies
};

// Fills the addressing fields of `a` for workgroups of `c` transforms of `n`
// points with elements of in_bytes / out_bytes.
inline void set_spans(KArgs &a, long long n, long long c, int in_bytes, int out_bytes) {
    const long long lim = 0x7fffffffLL;
    const long long cc = c < a.batch ? c : a.batch;
    const long long in_el = (cc - 1) * a.in_dist + (n - 1) * a.stride + 1;
    const long long out_el = (cc - 1) * a.out_dist + (n - 1) * a.stride + 1;
    const bool ok = a.in_dist >= 0 && a.out_dist >= 0 && a.stride >= 1 && in_el * in_bytes <= lim &&
                    out_el * out_bytes <= lim;
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
MI355FFT_DECLARE_LAUNCH(1024)
MI355FFT_DECLARE_LAUNCH(2048)
MI355FFT_DECLARE_LAUNCH(4096)
MI355FFT_DECLARE_LAUNCH(8192)
MI355FFT_DECLARE_LAUNCH(16384)
#undef MI355FFT_DECLARE_LAUNCH

}  // namespace mi355fft
