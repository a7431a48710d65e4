// k_attn_l1.hip -- the attention and significance kernels for page layout 1
// (see kLayoutFmts), one translation unit per layout so they build in parallel.
#include "attn_kernels.hpp"

namespace dkv {
const void* attn_kernel_l1(int gq, int which) { return attn_kernel_of<1>(gq, which); }
}  // namespace dkv
