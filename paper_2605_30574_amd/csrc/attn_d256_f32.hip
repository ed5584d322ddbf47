// Instantiates the attention kernels for head_dim 256, f32 inputs.
#include "attn_kernels.hpp"

namespace splice_dev {
AttnKernels attn_kernels_d256_f32(int G) { return pick_g<256, false>(G); }
}  // namespace splice_dev
