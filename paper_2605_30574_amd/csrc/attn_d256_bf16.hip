// Instantiates the attention kernels for head_dim 256, bf16 inputs.
#include "attn_kernels.hpp"

namespace splice_dev {
AttnKernels attn_kernels_d256_bf16(int G) { return pick_g<256, true>(G); }
}  // namespace splice_dev
