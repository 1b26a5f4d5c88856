// fft_n2048.hip -- instantiations of the single-pass kernels for N = 2048.
#include "fft_configs.hpp"

namespace mi355fft {

hipError_t launch_fft_n2048(int variant, int layout, int in_st, int out_st, int inv, int epi, const void *in,
                          void *out, const float2 *tw, const float2 *spec, const KArgs &a, hipStream_t s) {
    return dispatch<2048>(variant, layout, in_st, out_st, inv, epi, in, out, tw, spec, a, s);
}

int variants_n2048(int layout) { return variant_count<2048>(layout); }

}  // namespace mi355fft
