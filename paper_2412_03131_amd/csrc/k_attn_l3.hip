// k_attn_l3.hip -- the attention and significance kernels for page layout 3
// (see kLayoutFmts), one translation unit per layout so they build in parallel.
#include "attn_kernels.hpp"

namespace dkv {
const void* attn_kernel_l3(int gq, int which) { return attn_kernel_of<3>(gq, which); }
}  // namespace dkv
