// Instantiates the attention kernels for head_dim 64, f32 inputs.
#include "attn_kernels.hpp"

namespace splice_dev {
AttnKernels attn_kernels_d64_f32(int G) { return pick_g<64, false>(G); }
}  // namespace splice_dev
