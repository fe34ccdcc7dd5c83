// Convolution input gradient kernels, float32 storage.
#include "kconv.hpp"

namespace lrcnn {

int launch_conv_f32_dgrad(const ConvArgs &a, hipStream_t s) { return conv_dispatch<float, true>(a, s); }

}  // namespace lrcnn
