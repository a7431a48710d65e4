// common.hpp -- shared device helpers of the gfx950 DiffKV kernels.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "diffkv.h"

namespace dkv {

// Shapes the append and attention kernels implement (checked by the API).
constexpr int kD = 128;        // head_dim
constexpr int kG = 32;         // quantization group
constexpr int kNG = kD / kG;   // groups per vector
constexpr int kTHi = 16;       // tokens per high-precision page of layout 0 (K8V4)
constexpr int kTLo = 32;       // tokens per low-precision page of layout 0 (K4V2)
constexpr int kWave = 64;

// ---- page formats the kernels implement -------------------------------------
// A section's format: key bits, value bits, tokens per page.  The layouts (high
// section format, low section format) the append, attention and significance
// kernels implement, head_dim 128 and group 32 throughout:
//   0  K8V4 / K4V2, 16 / 32 tokens  (the paper's two levels, Sec. 4)
//   1  K8V8 / K4V2, 16 / 32         (K8V8 for the important tokens)
//   2  K8V2 / K4V1, 16 / 32         (the skewed variants of Sec. 7.2)
//   3  K8V4 / K4V2, 16 / 16         (as 0 with 16 tokens per low page)
// The generation-phase policy implements layout 0 only.
struct KvFmt {
    int kb, vb, T;
};
struct LayoutFmt {
    KvFmt hi, lo;
};
constexpr int kNumLayouts = 4;
constexpr LayoutFmt kLayoutFmts[kNumLayouts] = {
    {{8, 4, 16}, {4, 2, 32}}, {{8, 8, 16}, {4, 2, 32}}, {{8, 2, 16}, {4, 1, 32}}, {{8, 4, 16}, {4, 2, 16}}};

// Segment offsets of one section's page, as diffkv_layout_init lays them out:
// K codes, K meta, V codes, V meta, scores, positions, each 64-byte aligned.
struct SecOffsets {
    int kc, km, vc, vm, sc, pos, used;
};
constexpr int align64c(int x) { return (x + 63) & ~63; }
constexpr SecOffsets sec_offsets(KvFmt f)
{
    const int km = align64c((kD * f.kb / 128) * f.T * 16);
    const int vc = align64c(km + f.T * kNG * 4);
    const int vm = align64c(vc + kD * (f.T * f.vb / 8));
    const int sc = align64c(vm + kNG * f.T * 4);
    const int pos = align64c(sc + f.T * 4);
    return {0, km, vc, vm, sc, pos, align64c(pos + f.T * 4)};
}
constexpr int layout_page_bytes(int li)
{
    return sec_offsets(kLayoutFmts[li].hi).used > sec_offsets(kLayoutFmts[li].lo).used
               ? sec_offsets(kLayoutFmts[li].hi).used
               : sec_offsets(kLayoutFmts[li].lo).used;
}
static_assert(layout_page_bytes(0) == 4352 && sec_offsets(kLayoutFmts[0].lo).vc == 2560, "layout 0");

// Per-call device flags kept at the start of every workspace.
// Every field is written by the call's planning kernel before any later
// kernel of the same call reads it, so the block never needs clearing.
struct CallFlags {
    int32_t ok;         // 1 when the planning kernel accepted the call
    int32_t njobs;      // quantize jobs (append)
    int64_t head_old;   // ring head before this call
    int64_t tail_old;   // ring tail before this call
    unsigned long long arrive;  // arrival word of the one-token append (arrive_claim, arrive_count)
    unsigned long long arrive_group[16];  // its first level: one word per group of workgroups
};
static_assert(sizeof(CallFlags) <= 256, "call flags fit the 256 B every workspace reserves for them");

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// ---- wave reductions -------------------------------------------------------
template <int W>
__device__ __forceinline__ int wave_isum_w(int x)
{
#pragma unroll
    for (int o = W / 2; o > 0; o >>= 1) x += __shfl_xor(x, o, W);
    return x;
}

// Inclusive prefix sum over a full 64-lane wave with DPP: shifts of 1, 2, 4
// and 8 inside each 16-lane row, then row_bcast:15 and row_bcast:31 carry the
// row totals upward (lanes without a source read 0).
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROWS, 0xF, true);
}
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t x)
{
    x += dpp_u32<0x111, 0xF>(x);  // row_shr:1
    x += dpp_u32<0x112, 0xF>(x);  // row_shr:2
    x += dpp_u32<0x114, 0xF>(x);  // row_shr:4
    x += dpp_u32<0x118, 0xF>(x);  // row_shr:8
    x += dpp_u32<0x142, 0xA>(x);  // row_bcast:15 into rows 1 and 3
    x += dpp_u32<0x143, 0xC>(x);  // row_bcast:31 into rows 2 and 3
    return x;
}
__device__ __forceinline__ int wave_incl_scan(int x) { return (int)wave_incl_scan_u32((uint32_t)x); }
// two independent 32-bit counters packed in one 64-bit value
__device__ __forceinline__ long long wave_incl_scan64(long long x)
{
    const uint32_t lo = wave_incl_scan_u32((uint32_t)x);
    const uint32_t hi = wave_incl_scan_u32((uint32_t)((unsigned long long)x >> 32));
    return (long long)(((unsigned long long)hi << 32) | lo);
}

// Inclusive OR over a full wave, same DPP pattern as the prefix sum.
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_or_step(uint32_t x)
{
    return x | dpp_u32<CTRL, ROWS>(x);
}
__device__ __forceinline__ uint32_t wave_or_u32(uint32_t x)  // result in lane 63
{
    x = dpp_or_step<0x111, 0xF>(x);
    x = dpp_or_step<0x112, 0xF>(x);
    x = dpp_or_step<0x114, 0xF>(x);
    x = dpp_or_step<0x118, 0xF>(x);
    x = dpp_or_step<0x142, 0xA>(x);
    x = dpp_or_step<0x143, 0xC>(x);
    return (uint32_t)__builtin_amdgcn_readlane((int)x, kWave - 1);
}

// Makes one wave's LDS writes visible to its other lanes' later reads (the
// wave's LDS operations execute in order; this keeps the compiler from
// reordering them and states the synchronisation).
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int wave_index() { return __builtin_amdgcn_readfirstlane(threadIdx.x / kWave); }

template <typename TInt>
__device__ __forceinline__ TInt wave_incl_scan_t(TInt x)
{
    if constexpr (sizeof(TInt) == 8) return (TInt)wave_incl_scan64((long long)x);
    else return (TInt)wave_incl_scan((int)x);
}
template <typename TInt>
__device__ __forceinline__ TInt read_lane(TInt x, int l)  // l uniform
{
    if constexpr (sizeof(TInt) == 8) {
        const unsigned long long u = (unsigned long long)x;
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
        const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
        return (TInt)(((unsigned long long)hi << 32) | lo);
    } else {
        return (TInt)__builtin_amdgcn_readlane((int)x, l);
    }
}

// Exclusive block scan of one value per thread (blockDim.x multiple of 64,
// at most 1024).  Returns the exclusive prefix; *total gets the block sum.
// `lds` must hold blockDim.x/64 entries.  64-bit values are two independent
// 32-bit counters (no carry between the halves).  Every wave scans the wave
// totals itself, so there is one barrier plus one that frees `lds` for reuse.
// With `bits`, *bits_out also gets the OR of every thread's bits (`lds_bits`
// then holds blockDim.x/64 entries).
template <typename TInt>
__device__ __forceinline__ TInt block_excl_scan(TInt x, TInt* lds, TInt* total, uint32_t bits = 0,
                                                uint32_t* lds_bits = nullptr, uint32_t* bits_out = nullptr)
{
    const int l = lane_id();
    const int w = wave_index();
    const int nw = blockDim.x / kWave;
    const TInt inc = wave_incl_scan_t<TInt>(x);
    if (lds_bits) bits = wave_or_u32(bits);
    if (l == kWave - 1) {
        lds[w] = inc;
        if (lds_bits) lds_bits[w] = bits;
    }
    __syncthreads();
    const TInt tv = l < nw ? lds[l] : (TInt)0;
    const TInt tinc = wave_incl_scan_t<TInt>(tv);
    if (lds_bits) *bits_out = wave_or_u32(l < nw ? lds_bits[l] : 0u);
    const TInt below = read_lane<TInt>(tinc - tv, w);
    *total = read_lane<TInt>(tinc, nw - 1);
    __syncthreads();
    return below + inc - x;
}

// ---- arrival words --------------------------------------------------------
// Workgroups of one launch that must find out which of them comes last count
// themselves in a 64-bit word of the caller's workspace: a 44-bit call tag
// above a 20-bit count.  A word whose tag is not this call's counts as zero,
// so the workspace needs no clearing and what an earlier call left there is
// never taken for this one's.  The tag is the dispatch's packet index in its
// hardware queue (32 bits) with 12 bits of the queue's address (queues count
// their packets separately).
extern "C" __device__ unsigned long long dkv_dispatch_id() __asm("llvm.amdgcn.dispatch.id");

__device__ __forceinline__ unsigned long long call_tag()
{
    const unsigned long long q = (unsigned long long)(size_t)__builtin_amdgcn_queue_ptr();
    return (dkv_dispatch_id() & 0xffffffffull) | ((((q >> 12) ^ (q >> 24)) & 0xfffull) << 32);
}

constexpr int kArriveCountBits = 20;

// The count before this arrival once the add that returned `old` has landed on
// another call's word (where it counts nothing): the word is taken over by
// compare-and-swap (tag, 1), or, once another arrival has done that, counted in
// by compare-and-swap as well.
__device__ __forceinline__ unsigned long long arrive_takeover(unsigned long long* w, unsigned long long old,
                                                              unsigned long long tag)
{
    constexpr unsigned long long kCount = (1ull << kArriveCountBits) - 1;
    unsigned long long cnt;
    old += 1;
    for (;;) {
        cnt = (old >> kArriveCountBits) == tag ? (old & kCount) : 0ull;
        const unsigned long long nw = (tag << kArriveCountBits) | (cnt + 1);
        if (__hip_atomic_compare_exchange_strong(w, &old, nw, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT))
            return cnt;
    }
}

// Count one arrival of the call tagged `tag` in word w (agent-scope atomics);
// returns the count including it (1 .. 2^20 - 1).  One add counts the arrival
// when the word already carries this call's tag (every arrival but, normally,
// the first); otherwise arrive_takeover.
__device__ __forceinline__ unsigned long long arrive_count(unsigned long long* w, unsigned long long tag)
{
    constexpr unsigned long long kCount = (1ull << kArriveCountBits) - 1;
    const unsigned long long old = __hip_atomic_fetch_add(w, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return ((old >> kArriveCountBits) == tag ? (old & kCount) : arrive_takeover(w, old, tag)) + 1;
}

// Put this call's tag on word w with count 0 unless it already carries it.
// Done by one workgroup as a call starts, long before the arrivals of a word
// that many workgroups share: they then find the tag and count with one add
// each instead of taking the word over together (one compare-and-swap retry
// per concurrent arrival).  An arrival that still comes first takes the word
// over itself (arrive_takeover), and the claim never replaces a word that
// already carries the tag, so no counted arrival is lost.
__device__ __forceinline__ void arrive_claim(unsigned long long* w, unsigned long long tag)
{
    unsigned long long old = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    while ((old >> kArriveCountBits) != tag) {
        if (__hip_atomic_compare_exchange_strong(w, &old, tag << kArriveCountBits, __ATOMIC_RELAXED,
                                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
            break;
    }
}

// Block-wide sum of a true 64-bit value and OR of flag bits (all threads get
// the result).  `lds` must hold blockDim.x/64 + 1 entries.
__device__ __forceinline__ long long block_sum_or(long long x, uint32_t bits, long long* lds,
                                                  uint32_t* bits_out)
{
    const int w = threadIdx.x / kWave;
    const int nw = blockDim.x / kWave;
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        x += __shfl_xor(x, o, kWave);
        bits |= (uint32_t)__shfl_xor((int)bits, o, kWave);
    }
    __shared__ uint32_t s_bits;
    if (threadIdx.x == 0) s_bits = 0;
    __syncthreads();
    if (lane_id() == 0) {
        lds[w] = x;
        atomicOr(&s_bits, bits);
    }
    __syncthreads();
    long long t = 0;
    for (int i = 0; i < nw; ++i) t += lds[i];
    *bits_out = s_bits;
    __syncthreads();
    return t;
}

// ---- fp16 helpers ----------------------------------------------------------
__device__ __forceinline__ float h2f(uint32_t bits16)
{
    return __half2float(__ushort_as_half((unsigned short)bits16));
}
// fp32 -> fp16, round to nearest even (v_cvt_f16_f32 under the default mode)
__device__ __forceinline__ uint32_t f2h_rne(float f)
{
    return (uint32_t)__half_as_ushort(__float2half_rn(f));
}

// ---- host: launches ---------------------------------------------------------
// Enqueue one launch of a kernel taking one argument block and return the
// status of that launch itself (hipLaunchKernel's), never an error that an
// earlier, unrelated runtime call left on the calling thread.
template <typename A>
inline hipError_t launch1(void (*kern)(A), unsigned grid, unsigned block, hipStream_t st, const A& a,
                          size_t lds_bytes = 0)
{
    void* args[] = {const_cast<A*>(&a)};
    return hipLaunchKernel(reinterpret_cast<const void*>(kern), dim3(grid), dim3(block), args, lds_bytes, st);
}

}  // namespace dkv
