// attn_common.hpp -- constants shared by the attention kernels and their
// host-side launchers.
#pragma once

#include "internal.hpp"

namespace dkv {

constexpr int kAttnWaves = 8;  // single page buffer: GQ <= 6 fits two workgroups per CU
constexpr int kAttnThreads = kAttnWaves * kWave;
// Workgroups of attn_decode<GQ, LI> each CU holds at once; the launch bounds
// make the compiler fit that residency (at most 128 VGPRs for two eight-wave
// workgroups).  GQ 7-8 need more registers: four waves per SIMD there spilled
// and measured slower, so they run one workgroup per CU.  Layouts with 8-bit
// values stage two value rows per lane, which leaves LDS for two workgroups
// per CU only up to GQ 5.
constexpr bool layout_wide_values(int li)
{
    return 2 * kLayoutFmts[li].hi.T * kLayoutFmts[li].hi.vb / 8 > 16 ||
           2 * kLayoutFmts[li].lo.T * kLayoutFmts[li].lo.vb / 8 > 16;
}
constexpr int attn_blocks_per_cu(int gq, int li) { return gq <= (layout_wide_values(li) ? 5 : 6) ? 2 : 1; }
constexpr int kPartStride = kD + 2;
constexpr int kSigWaves = 4;
constexpr int kSigPages = 16;  // pages per workgroup of attn_significance

// Kernel entry points of layout n (k_attn_l<n>.hip): which = 0 attn_decode,
// 1 attn_significance; nullptr for an unknown gq.
const void* attn_kernel_l0(int gq, int which);
const void* attn_kernel_l1(int gq, int which);
const void* attn_kernel_l2(int gq, int which);
const void* attn_kernel_l3(int gq, int which);

}  // namespace dkv
