// Convolution forward kernels, bfloat16 storage.
#include "kconv.hpp"

namespace lrcnn {

int launch_conv_bf16_fwd(const ConvArgs &a, hipStream_t s) { return conv_dispatch<bf16, false>(a, s); }

}  // namespace lrcnn
