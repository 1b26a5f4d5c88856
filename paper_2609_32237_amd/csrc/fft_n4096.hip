// fft_n4096.hip -- instantiations of the single-pass kernels for N = 4096.
#include "fft_configs.hpp"
#include "fft_mfma.hpp"

namespace mi355fft {

hipError_t launch_fft_n4096(int variant, int layout, int in_st, int out_st, int inv, int epi, const void *in,
                          void *out, const float2 *tw, const float2 *spec, const KArgs &a, hipStream_t s) {
    return dispatch<4096>(variant, layout, in_st, out_st, inv, epi, in, out, tw, spec, a, s);
}

int variants_n4096(int layout) { return variant_count<4096>(layout); }

hipError_t launch_fft_mfma_n4096(int inv, const void *in, void *out, const float2 *tw, const void *amat,
                               const KArgs &a, hipStream_t s) {
    return launch_mfma<MfmaCfg<4096, 1, 4>>(inv, in, out, tw, amat, a, s);
}

}  // namespace mi355fft
