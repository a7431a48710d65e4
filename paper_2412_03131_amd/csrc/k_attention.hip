// k_attention.hip -- host side of the decode attention and significance
// kernels (attn_kernels.hpp, instantiated per page layout in k_attn_l<n>.hip):
// the launch mode, the balanced mode's share count, the launches, and the
// device scratch of the no-allocation entry point.
#include <atomic>

#include "attn_common.hpp"

namespace dkv {

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
// Kernel entry points of layout li: which = 0 decode, 1 significance, 2 paired tables.
static const void* attn_kernel_ptr(int li, int gq, int which)
{
    switch (li) {
    case 0: return attn_kernel_l0(gq, which);
    case 1: return attn_kernel_l1(gq, which);
    case 2: return attn_kernel_l2(gq, which);
    case 3: return attn_kernel_l3(gq, which);
    default: return nullptr;
    }
}

// Workgroups of attn_decode<gq> the device holds at once (the balanced mode's
// share count): the residency the launch bounds guarantee times the CU count of
// the current device, at most kAttnMaxWorkers.  A third workgroup per CU (three
// waves per SIMD, where the registers allow it) measured slower: the page loop
// is bound by VALU issue, and more shares only split more tables.  Nothing is
// cached between calls.
static hipError_t balanced_workers(int gq, int li, int* workers)
{
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    const int w = attn_blocks_per_cu(gq, li) * (cus > 0 ? cus : 1);
    *workers = w < kAttnMaxWorkers ? w : kAttnMaxWorkers;
    return hipSuccess;
}

hipError_t attention_mode(int gq, int li, long long T, int splits, int* mode, int* workers)
{
    hipError_t e = balanced_workers(gq, li, workers);
    if (e != hipSuccess) return e;
    // automatic: when the tables alone fill the device, no table is split --
    // pairs of tables (a long one with a short one) per sixteen-wave workgroup
    // up to GQ 5, one workgroup per table above (their spread is absorbed by
    // wave priorities and by the hardware dispatching further workgroups as
    // others finish); balanced shares when there are fewer tables than
    // resident workgroups
    *mode = splits != 0 ? splits : (T >= *workers ? (gq <= kPairMaxGq ? kModePair : 1) : -1);
    return hipSuccess;
}

// The no-allocation entry point's scratch: arrival words and split partial
// states of one attention call.  In host code `scratch` names a host-side
// stand-in, so its device address is looked up once per device (with that
// device current) and only that address is handed to kernels.
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

hipError_t noalloc_scratch(void** ptr)
{
    constexpr int kDevs = 64;
    static std::atomic<void*> addr[kDevs];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kDevs) return hipErrorInvalidDevice;
    void* p = addr[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        addr[dev].store(p, std::memory_order_release);
    }
    *ptr = p;
    return hipSuccess;
}

hipError_t launch_attention(AttnArgs a, hipStream_t st)
{
    const int gq = a.Hq / a.Hkv;
    const void* kern = attn_kernel_ptr(a.layout, gq, 0);
    if (!kern) return hipErrorInvalidValue;
    const long long T = (long long)a.B * a.Hkv;
    int workers = 0;
    hipError_t e = attention_mode(gq, a.layout, T, a.splits, &a.splits, &workers);
    if (e != hipSuccess) return e;
    void* args[] = {&a};
    if (a.splits == kModePair) {
        const void* pair = attn_kernel_ptr(a.layout, gq, 2);
        if (!pair) return hipErrorInvalidValue;
        const long long pgrid = (T + 1) / 2;
        if (pgrid < 1 || pgrid > INT32_MAX) return hipErrorInvalidValue;
        return hipLaunchKernel(pair, dim3((unsigned)pgrid), dim3((unsigned)(kPairWaves * kWave)), args, 0, st);
    }
    const long long grid = a.splits > 0 ? T * a.splits : workers;
    if (grid < 1 || grid > INT32_MAX) return hipErrorInvalidValue;
    return hipLaunchKernel(kern, dim3((unsigned)grid), dim3((unsigned)(attn_waves(gq, a.layout) * kWave)), args, 0, st);
}


hipError_t launch_significance(const SigArgs& a, hipStream_t st)
{
    const int gq = a.Hq / a.Hkv;
    const void* kern = attn_kernel_ptr(a.layout, gq, 1);
    if (!kern) return hipErrorInvalidValue;
    const long long T = (long long)a.B * a.Hkv;
    const long long grid = T * ((a.p_max + kSigPages - 1) / kSigPages);
    if (T < 1 || grid > INT32_MAX) return hipErrorInvalidValue;
    void* args[] = {const_cast<SigArgs*>(&a)};
    return hipLaunchKernel(kern, dim3((unsigned)grid), dim3(kSigWaves * kWave), args, 0, st);
}

}  // namespace dkv
