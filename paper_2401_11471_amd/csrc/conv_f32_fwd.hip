// Convolution forward kernels, float32 storage.
#include "kconv.hpp"

namespace lrcnn {

int launch_conv_f32_fwd(const ConvArgs &a, hipStream_t s) { return conv_dispatch<float, false>(a, s); }

}  // namespace lrcnn
