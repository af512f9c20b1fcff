// Matrix-core dispatch of the fused FFT convolution for 16-bit I/O (Sec. 4.1:
// kernel fusion + block FFT): the one-wave kernel at L = 2048, the four-wave
// kernel at L = 8192 and the eight-wave kernel at L = 16384, each computing
// the kernel spectrum from k itself.
#include "common.h"
#include "internal.h"

namespace h3 {

bool fftconv_mfma_supported(int L, int dtype) {
    return fftconv_wave_supported(L, dtype) || fftconv_wave16k_supported(L, dtype) ||
           fftconv_wave32k_supported(L, dtype);
}

// hipErrorInvalidValue for any other shape.  An output gate is supported at L = 2048 only.
hipError_t launch_fftconv_mfma(const ConvArgs &a, const float *k, hipStream_t s) {
    if (fftconv_wave_supported(a.L, a.dtype)) return launch_fftconv_wave(a, k, s);
    if (a.gate) return hipErrorInvalidValue;
    if (fftconv_wave16k_supported(a.L, a.dtype)) return launch_fftconv_wave16k(a, k, s);
    if (fftconv_wave32k_supported(a.L, a.dtype)) return launch_fftconv_wave32k(a, k, s);
    return hipErrorInvalidValue;
}

}  // namespace h3
