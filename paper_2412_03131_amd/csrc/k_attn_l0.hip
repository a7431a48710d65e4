// k_attn_l0.hip -- the attention and significance kernels for page layout 0
// (see kLayoutFmts), one translation unit per layout so they build in parallel.
#include "attn_kernels.hpp"

namespace dkv {
const void* attn_kernel_l0(int gq, int which) { return attn_kernel_of<0>(gq, which); }
}  // namespace dkv
