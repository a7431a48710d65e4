// attn_common.hpp -- constants shared by the attention kernels and their
// host-side launchers.
#pragma once

#include "internal.hpp"

namespace dkv {

// Workgroups of attn_decode<GQ, LI> each CU holds at once: two eight-wave
// workgroups (four waves per SIMD, at most 128 VGPRs) up to GQ 5; from GQ 6
// the kernel needs more registers (129-153), and one twelve-wave workgroup per
// CU keeps three waves per SIMD.  Layouts with 8-bit values stage two value
// rows per lane (more LDS per wave).
constexpr bool layout_wide_values(int li)
{
    return 2 * kLayoutFmts[li].hi.T * kLayoutFmts[li].hi.vb / 8 > 16 ||
           2 * kLayoutFmts[li].lo.T * kLayoutFmts[li].lo.vb / 8 > 16;
}
constexpr int attn_blocks_per_cu(int gq, int li) { return gq <= 5 ? 2 : 1; }
// Waves per workgroup: eight (two per SIMD) where two workgroups share a CU,
// twelve (three per SIMD) where one workgroup has the CU: the registers of
// the larger group sizes (at most 168 VGPRs) allow three waves per SIMD, and
// the page loops need the waves to cover each other's waits.
constexpr int attn_waves(int gq, int li) { return attn_blocks_per_cu(gq, li) == 2 ? 8 : 12; }
// The paired-table kernel: sixteen waves, one workgroup per CU, up to GQ 5
// (at most 128 VGPRs, four waves per SIMD).
constexpr int kPairWaves = 16;
constexpr int kPairMaxGq = 5;
constexpr int kModePair = -2;  // launch mode of attn_pair (internal; never a caller's num_splits)
constexpr int kPartStride = kD + 2;
constexpr int kSigWaves = 4;
constexpr int kSigPages = 16;  // pages per workgroup of attn_significance

// Kernel entry points of layout n (k_attn_l<n>.hip): which = 0 attn_decode,
// 1 attn_significance, 2 attn_pair; nullptr for an unknown gq (and for
// attn_pair above kPairMaxGq).
const void* attn_kernel_l0(int gq, int which);
const void* attn_kernel_l1(int gq, int which);
const void* attn_kernel_l2(int gq, int which);
const void* attn_kernel_l3(int gq, int which);

}  // namespace dkv
