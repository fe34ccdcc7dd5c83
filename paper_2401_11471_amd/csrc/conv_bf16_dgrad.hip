// Convolution input gradient kernels, bfloat16 storage.
#include "kconv.hpp"

namespace lrcnn {

int launch_conv_bf16_dgrad(const ConvArgs &a, hipStream_t s) { return conv_dispatch<bf16, true>(a, s); }

}  // namespace lrcnn
