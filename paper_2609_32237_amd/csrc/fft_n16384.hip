// fft_n16384.hip -- instantiations of the single-pass kernels for N = 16384.
#include "fft_configs.hpp"
#include "fft_mfma.hpp"

namespace mi355fft {

hipError_t launch_fft_n16384(int variant, int layout, int in_st, int out_st, int inv, int epi, const void *in,
                          void *out, const float2 *tw, const float2 *spec, const KArgs &a, hipStream_t s) {
    return dispatch<16384>(variant, layout, in_st, out_st, inv, epi, in, out, tw, spec, a, s);
}

int variants_n16384(int layout) { return variant_count<16384>(layout); }

hipError_t launch_fft_mfma_n16384(int inv, const void *in, void *out, const float2 *tw, const void *amat,
                               const KArgs &a, hipStream_t s) {
    return launch_mfma<MfmaCfg<16384, 4, 8>>(inv, in, out, tw, amat, a, s);
}

}  // namespace mi355fft
