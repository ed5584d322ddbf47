// Instantiates the attention kernels for head_dim 128, f32 inputs.
#include "attn_kernels.hpp"

namespace splice_dev {
AttnKernels attn_kernels_d128_f32(int G) { return pick_g<128, false>(G); }
}  // namespace splice_dev
