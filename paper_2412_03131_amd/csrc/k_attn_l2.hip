// k_attn_l2.hip -- the attention and significance kernels for page layout 2
// (see kLayoutFmts), one translation unit per layout so they build in parallel.
#include "attn_kernels.hpp"

namespace dkv {
const void* attn_kernel_l2(int gq, int which) { return attn_kernel_of<2>(gq, which); }
}  // namespace dkv
