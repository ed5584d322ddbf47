// Instantiates the attention kernels for head_dim 64, bf16 inputs.
#include "attn_kernels.hpp"

namespace splice_dev {
AttnKernels attn_kernels_d64_bf16(int G) { return pick_g<64, true>(G); }
}  // namespace splice_dev
