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
constexpr int kTHi = 16;       // tokens per high-precision page (K8V4)
constexpr int kTLo = 32;       // tokens per low-precision page (K4V2)
constexpr int kWave = 64;

// Per-call device flags kept at the start of every workspace.
// Every field is written by the call's planning kernel before any later
// kernel of the same call reads it, so the block never needs clearing.
struct CallFlags {
    int32_t ok;         // 1 when the planning kernel accepted the call
    int32_t njobs;      // quantize jobs (append)
    int64_t head_old;   // ring head before this call
    int64_t tail_old;   // ring tail before this call
};

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// ---- wave reductions -------------------------------------------------------
template <int W>
__device__ __forceinline__ float wave_sum_w(float x)
{
#pragma unroll
    for (int o = W / 2; o > 0; o >>= 1) x += __shfl_xor(x, o, W);
    return x;
}
template <int W>
__device__ __forceinline__ float wave_max_w(float x)
{
#pragma unroll
    for (int o = W / 2; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, W));
    return x;
}
template <int W>
__device__ __forceinline__ float wave_min_w(float x)
{
#pragma unroll
    for (int o = W / 2; o > 0; o >>= 1) x = fminf(x, __shfl_xor(x, o, W));
    return x;
}
template <int W>
__device__ __forceinline__ int wave_isum_w(int x)
{
#pragma unroll
    for (int o = W / 2; o > 0; o >>= 1) x += __shfl_xor(x, o, W);
    return x;
}

// Inclusive prefix sum over a full 64-lane wave.
__device__ __forceinline__ int wave_incl_scan(int x)
{
    const int l = lane_id();
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        int y = __shfl_up(x, o, kWave);
        if (l >= o) x += y;
    }
    return x;
}
__device__ __forceinline__ long long wave_incl_scan64(long long x)
{
    const int l = lane_id();
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        long long y = __shfl_up(x, o, kWave);
        if (l >= o) x += y;
    }
    return x;
}

// Exclusive block scan of one value per thread (blockDim.x multiple of 64,
// at most 1024).  Returns the exclusive prefix; *total gets the block sum.
// `lds` must hold blockDim.x/64 + 1 entries.
template <typename TInt>
__device__ __forceinline__ TInt block_excl_scan(TInt x, TInt* lds, TInt* total)
{
    const int l = lane_id();
    const int w = threadIdx.x / kWave;
    const int nw = blockDim.x / kWave;
    TInt inc;
    if constexpr (sizeof(TInt) == 8) inc = (TInt)wave_incl_scan64((long long)x);
    else inc = (TInt)wave_incl_scan((int)x);
    if (l == kWave - 1) lds[w] = inc;
    __syncthreads();
    if (threadIdx.x == 0) {
        TInt run = 0;
        for (int i = 0; i < nw; ++i) {
            TInt t = lds[i];
            lds[i] = run;
            run += t;
        }
        lds[nw] = run;
    }
    __syncthreads();
    TInt r = lds[w] + inc - x;
    *total = lds[nw];
    __syncthreads();
    return r;
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

}  // namespace dkv
