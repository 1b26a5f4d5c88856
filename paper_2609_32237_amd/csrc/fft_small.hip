// fft_small.hip -- instantiations for N = 64 ... 512, the column passes of
// four-step transforms longer than 16384 points.
#include "fft_configs.hpp"

namespace mi355fft {

#define MI355FFT_DEFINE_LAUNCH(N)                                                                          \
    hipError_t launch_fft_n##N(int variant, int layout, int in_st, int out_st, int inv, int epi,           \
                               const void *in, void *out, const float2 *tw, const float2 *spec,            \
                               const KArgs &a, hipStream_t s) {                                            \
        return dispatch<N>(variant, layout, in_st, out_st, inv, epi, in, out, tw, spec, a, s);             \
    }                                                                                                      \
    int variants_n##N(int layout) { return variant_count<N>(layout); }
MI355FFT_DEFINE_LAUNCH(64)
MI355FFT_DEFINE_LAUNCH(128)
MI355FFT_DEFINE_LAUNCH(256)
MI355FFT_DEFINE_LAUNCH(512)
#undef MI355FFT_DEFINE_LAUNCH

}  // namespace mi355fft
