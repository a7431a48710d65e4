// k_attention.hip -- decode attention over the differentiated paged KV cache
// for gfx950 (DiffKV Eq. (1) of Sec. 2.1, kernel structure of Sec. 6.2).
//
// Grid (splits, Hkv, B); a workgroup of four waves owns one table (one
// sequence, one KV head) -- or one page range of it when the sequence is
// split -- and all GQ query heads that read it.  Each wave walks its share of
// the table's pages, high-precision pages first, then low-precision pages.
//
// Lane mapping inside a wave (64 lanes = 4 rows of 16):
//   key phase    lane = grp*16 + j: token j (and j+16 on 32-token pages),
//                32-dim group grp; the lane holds q of its group as fp16
//                pairs and computes sum(q*code) with v_dot2_f32_f16, then
//                s*sum + z*sum(q) (scale and zero factored out of the dot
//                product); the four groups of a token are summed across rows.
//   softmax      online, base 2, per query head; page max by row reduction.
//   value phase  lane owns dims 2*lane, 2*lane+1 (group = its row): the
//                weights p*s_v of the row's tokens are broadcast inside the
//                row (DPP row_newbcast) and multiplied into fp32 accumulators;
//                the zero-point term sum(p*z_v) is accumulated per lane and
//                added once at the end.
// Partial states of the four waves merge through LDS; with splits > 1 the
// per-range (max, sum, acc) states go to the workspace and attn_merge
// combines them.
#include "internal.hpp"

namespace dkv {

constexpr int kAttnWaves = 4;
constexpr int kAttnThreads = kAttnWaves * kWave;
constexpr int kPartStride = kD + 2;

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

template <int J>
__device__ __forceinline__ float row_bcast(float x)
{
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x150 + J, 0xF, 0xF, true));
}

// four K8 codes (one dword) -> two fp16 pairs holding the codes exactly
__device__ __forceinline__ void k8_pairs(uint32_t w, half2_t& x01, half2_t& x23)
{
    const half2_t off = {(_Float16)-1024.0f, (_Float16)-1024.0f};
    uint32_t a = __builtin_amdgcn_perm(0x64646464u, w, 0x04010400u);  // 0x64 b1 0x64 b0
    uint32_t b = __builtin_amdgcn_perm(0x64646464u, w, 0x04030402u);  // 0x64 b3 0x64 b2
    x01 = __builtin_bit_cast(half2_t, a) + off;
    x23 = __builtin_bit_cast(half2_t, b) + off;
}

// eight K4 codes (one dword, dims 2m in the low nibble of byte m) -> four pairs
__device__ __forceinline__ void k4_pairs(uint32_t w, half2_t x[4])
{
    const half2_t mul = {(_Float16)1.0f, (_Float16)0.0625f};
    const half2_t off = {(_Float16)-1024.0f, (_Float16)-64.0f};
    const uint32_t sel[4] = {0x04000400u, 0x04010401u, 0x04020402u, 0x04030403u};
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        uint32_t y = __builtin_amdgcn_perm(0x64646464u, w, sel[m]) & 0xFFF0FF0Fu;
        x[m] = __builtin_bit_cast(half2_t, y) * mul + off;
    }
}

__device__ __forceinline__ float dot2(half2_t a, half2_t b, float c)
{
    return __builtin_amdgcn_fdot2(a, b, c, false);
}

template <int GQ>
struct WaveState {
    float m[GQ];      // running max (log2 domain), wave-uniform
    float l[GQ];      // this lane's share of the running sum
    float z[GQ];      // this lane's share of sum(p * z_v) for its row's group
    float acc[GQ][2]; // dims 2*lane, 2*lane+1
};

// Process the logits of up to two tokens per lane; returns p and updates state.
template <int GQ, int NT>
__device__ __forceinline__ void online_softmax(WaveState<GQ>& st, float (&lg)[NT][GQ],
                                               float (&p)[NT][GQ])
{
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh) {
        float mx = lg[0][hh];
        if (NT > 1) mx = fmaxf(mx, lg[NT - 1][hh]);
        mx = wave_max_w<16>(mx);
        const float mnew = fmaxf(st.m[hh], mx);
        const float alpha = __builtin_amdgcn_exp2f(st.m[hh] - mnew);
        st.m[hh] = mnew;
        float psum = 0.f;
#pragma unroll
        for (int i = 0; i < NT; ++i) {
            p[i][hh] = __builtin_amdgcn_exp2f(lg[i][hh] - mnew);
            psum += p[i][hh];
        }
        st.l[hh] = st.l[hh] * alpha + psum;
        st.z[hh] *= alpha;
        st.acc[hh][0] *= alpha;
        st.acc[hh][1] *= alpha;
    }
}

template <int GQ, int J>
__device__ __forceinline__ void pv_hi_step(WaveState<GQ>& st, const float (&cf)[GQ], uint32_t w0,
                                           uint32_t w1)
{
    // token J of a 16-token page: nibble J of each dim row (rows are 64 bits;
    // w0/w1 hold the dword that contains token J for dims 2*lane and 2*lane+1)
    const float c0 = (float)((w0 >> (4 * (J & 7))) & 15u);
    const float c1 = (float)((w1 >> (4 * (J & 7))) & 15u);
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh) {
        const float b = row_bcast<J>(cf[hh]);
        st.acc[hh][0] = fmaf(b, c0, st.acc[hh][0]);
        st.acc[hh][1] = fmaf(b, c1, st.acc[hh][1]);
    }
}

template <int GQ, int J>
__device__ __forceinline__ void pv_hi_all(WaveState<GQ>& st, const float (&cf)[GQ], const uint4& vr)
{
    if constexpr (J < 16) {
        const uint32_t w0 = (J < 8) ? vr.x : vr.y;
        const uint32_t w1 = (J < 8) ? vr.z : vr.w;
        pv_hi_step<GQ, J>(st, cf, w0, w1);
        pv_hi_all<GQ, J + 1>(st, cf, vr);
    }
}

template <int GQ, int J>
__device__ __forceinline__ void pv_lo_all(WaveState<GQ>& st, const float (&cfA)[GQ],
                                          const float (&cfB)[GQ], const uint4& vr)
{
    if constexpr (J < 16) {
        // token J sits in the first dword of each 64-bit row, token J+16 in the second
        const float a0 = (float)((vr.x >> (2 * J)) & 3u), a1 = (float)((vr.z >> (2 * J)) & 3u);
        const float b0 = (float)((vr.y >> (2 * J)) & 3u), b1 = (float)((vr.w >> (2 * J)) & 3u);
#pragma unroll
        for (int hh = 0; hh < GQ; ++hh) {
            const float ba = row_bcast<J>(cfA[hh]);
            const float bb = row_bcast<J>(cfB[hh]);
            st.acc[hh][0] = fmaf(ba, a0, fmaf(bb, b0, st.acc[hh][0]));
            st.acc[hh][1] = fmaf(ba, a1, fmaf(bb, b1, st.acc[hh][1]));
        }
        pv_lo_all<GQ, J + 1>(st, cfA, cfB, vr);
    }
}

template <int GQ>
__global__ __launch_bounds__(kAttnThreads) void attn_decode(AttnArgs a)
{
    const int split = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int t = b * a.Hkv + h;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int grp = lane >> 4;
    const int jl = lane & 15;
    const int len_hi = a.len[2 * t], len_lo = a.len[2 * t + 1];
    // page counts from the section lengths, clamped to the table width
    int ph = (len_hi + kTHi - 1) / kTHi;
    int pl = (len_lo + kTLo - 1) / kTLo;
    ph = ph < 0 ? 0 : (ph > a.p_max ? a.p_max : ph);
    pl = pl < 0 ? 0 : (pl > a.p_max - ph ? a.p_max - ph : pl);
    const int P = ph + pl;
    const int p0 = (int)(((long long)split * P) / a.splits);
    const int p1 = (int)(((long long)(split + 1) * P) / a.splits);

    // q of this lane's group, as fp16 pairs, and its sum
    half2_t q2[GQ][16];
    float qsum[GQ];
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh) {
        const uint4* qp = reinterpret_cast<const uint4*>(
            a.q + ((long long)b * a.Hq + h * GQ + hh) * kD + grp * kG);
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint4 v = qp[i];
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                q2[hh][4 * i + k] = __builtin_bit_cast(half2_t, w[k]);
                s += (float)q2[hh][4 * i + k].x + (float)q2[hh][4 * i + k].y;
            }
        }
        qsum[hh] = s;
    }

    WaveState<GQ> st;
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh) {
        st.m[hh] = -INFINITY;
        st.l[hh] = 0.f;
        st.z[hh] = 0.f;
        st.acc[hh][0] = st.acc[hh][1] = 0.f;
    }
    const float sl2 = a.scale_log2;
    const int32_t* trow = a.page_table + (long long)t * a.p_max;

    for (int pp = p0 + wave; pp < p1; pp += kAttnWaves) {
        const int p = __builtin_amdgcn_readfirstlane(pp);
        const bool hi = p < ph;
        const int kpg = hi ? p : p - ph;
        const int id = trow[hi ? kpg : a.p_max - 1 - kpg];
        if ((unsigned)id >= (unsigned)a.num_pages) continue;  // never read outside the pool
        const uint8_t* pg = a.pool + (long long)id * a.page_bytes;
        if (hi) {
            const uint8_t* kc = pg + a.off_kcode[0];
            const uint4 ka = *reinterpret_cast<const uint4*>(kc + ((2 * grp) * kTHi + jl) * 16);
            const uint4 kb = *reinterpret_cast<const uint4*>(kc + ((2 * grp + 1) * kTHi + jl) * 16);
            const uint32_t km = *reinterpret_cast<const uint32_t*>(pg + a.off_kmeta[0] + (jl * kNG + grp) * 4);
            const uint32_t vm = *reinterpret_cast<const uint32_t*>(pg + a.off_vmeta[0] + (grp * kTHi + jl) * 4);
            const uint4 vr = *reinterpret_cast<const uint4*>(pg + a.off_vcode[0] + lane * 16);
            half2_t x[16];
            k8_pairs(ka.x, x[0], x[1]);
            k8_pairs(ka.y, x[2], x[3]);
            k8_pairs(ka.z, x[4], x[5]);
            k8_pairs(ka.w, x[6], x[7]);
            k8_pairs(kb.x, x[8], x[9]);
            k8_pairs(kb.y, x[10], x[11]);
            k8_pairs(kb.z, x[12], x[13]);
            k8_pairs(kb.w, x[14], x[15]);
            const float ks = h2f(km & 0xffffu), kz = h2f(km >> 16);
            const bool valid = kpg * kTHi + jl < len_hi;
            float lg[1][GQ];
#pragma unroll
            for (int hh = 0; hh < GQ; ++hh) {
                float d = 0.f;
#pragma unroll
                for (int m = 0; m < 16; ++m) d = dot2(q2[hh][m], x[m], d);
                float part = fmaf(ks, d, kz * qsum[hh]);
                part += __shfl_xor(part, 16);
                part += __shfl_xor(part, 32);
                lg[0][hh] = valid ? part * sl2 : -INFINITY;
            }
            float p_[1][GQ];
            online_softmax<GQ, 1>(st, lg, p_);
            const float vs = h2f(vm & 0xffffu), vz = h2f(vm >> 16);
            float cf[GQ];
#pragma unroll
            for (int hh = 0; hh < GQ; ++hh) {
                cf[hh] = p_[0][hh] * vs;
                st.z[hh] = fmaf(p_[0][hh], vz, st.z[hh]);
            }
            pv_hi_all<GQ, 0>(st, cf, vr);
        } else {
            const uint8_t* kc = pg + a.off_kcode[1];
            const uint4 kA = *reinterpret_cast<const uint4*>(kc + (grp * kTLo + jl) * 16);
            const uint4 kB = *reinterpret_cast<const uint4*>(kc + (grp * kTLo + jl + 16) * 16);
            const uint32_t kmA = *reinterpret_cast<const uint32_t*>(pg + a.off_kmeta[1] + (jl * kNG + grp) * 4);
            const uint32_t kmB = *reinterpret_cast<const uint32_t*>(pg + a.off_kmeta[1] + ((jl + 16) * kNG + grp) * 4);
            const uint32_t vmA = *reinterpret_cast<const uint32_t*>(pg + a.off_vmeta[1] + (grp * kTLo + jl) * 4);
            const uint32_t vmB = *reinterpret_cast<const uint32_t*>(pg + a.off_vmeta[1] + (grp * kTLo + jl + 16) * 4);
            const uint4 vr = *reinterpret_cast<const uint4*>(pg + a.off_vcode[1] + lane * 16);
            float lg[2][GQ];
#pragma unroll
            for (int tk = 0; tk < 2; ++tk) {
                const uint4 kk = tk ? kB : kA;
                const uint32_t km = tk ? kmB : kmA;
                half2_t x[16];
                k4_pairs(kk.x, &x[0]);
                k4_pairs(kk.y, &x[4]);
                k4_pairs(kk.z, &x[8]);
                k4_pairs(kk.w, &x[12]);
                const float ks = h2f(km & 0xffffu), kz = h2f(km >> 16);
                const bool valid = kpg * kTLo + jl + 16 * tk < len_lo;
#pragma unroll
                for (int hh = 0; hh < GQ; ++hh) {
                    float d = 0.f;
#pragma unroll
                    for (int m = 0; m < 16; ++m) d = dot2(q2[hh][m], x[m], d);
                    float part = fmaf(ks, d, kz * qsum[hh]);
                    part += __shfl_xor(part, 16);
                    part += __shfl_xor(part, 32);
                    lg[tk][hh] = valid ? part * sl2 : -INFINITY;
                }
            }
            float p_[2][GQ];
            online_softmax<GQ, 2>(st, lg, p_);
            const float vsA = h2f(vmA & 0xffffu), vzA = h2f(vmA >> 16);
            const float vsB = h2f(vmB & 0xffffu), vzB = h2f(vmB >> 16);
            float cfA[GQ], cfB[GQ];
#pragma unroll
            for (int hh = 0; hh < GQ; ++hh) {
                cfA[hh] = p_[0][hh] * vsA;
                cfB[hh] = p_[1][hh] * vsB;
                st.z[hh] = fmaf(p_[0][hh], vzA, fmaf(p_[1][hh], vzB, st.z[hh]));
            }
            pv_lo_all<GQ, 0>(st, cfA, cfB, vr);
        }
    }

    // ---- finish the wave: row sums of l and of the zero-point term ----------
    __shared__ float s_m[kAttnWaves][8];
    __shared__ float s_l[kAttnWaves][8];
    __shared__ float s_acc[kAttnWaves][8][kD];
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh) {
        const float l = wave_sum_w<16>(st.l[hh]);
        const float z = wave_sum_w<16>(st.z[hh]);
        if (lane == 0) {
            s_m[wave][hh] = st.m[hh];
            s_l[wave][hh] = l;
        }
        s_acc[wave][hh][2 * lane] = st.acc[hh][0] + z;
        s_acc[wave][hh][2 * lane + 1] = st.acc[hh][1] + z;
    }
    __syncthreads();
    // ---- merge the waves ----------------------------------------------------
    for (int i = threadIdx.x; i < GQ * kD; i += kAttnThreads) {
        const int hh = i / kD, d = i - hh * kD;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kAttnWaves; ++w) M = fmaxf(M, s_m[w][hh]);
        float L = 0.f, O = 0.f;
        if (M != -INFINITY) {
#pragma unroll
            for (int w = 0; w < kAttnWaves; ++w) {
                const float f = __builtin_amdgcn_exp2f(s_m[w][hh] - M);
                L = fmaf(s_l[w][hh], f, L);
                O = fmaf(s_acc[w][hh][d], f, O);
            }
        }
        const int hq = h * GQ + hh;
        if (a.splits == 1) {
            a.out[((long long)b * a.Hq + hq) * kD + d] = (L > 0.f) ? O / L : 0.f;
            if (d == 0 && a.lse)
                a.lse[(long long)b * a.Hq + hq] = (L > 0.f) ? (M + __log2f(L)) * 0.69314718055994530942f : -INFINITY;
        } else {
            float* pr = a.part + (((long long)split * a.B + b) * a.Hq + hq) * kPartStride;
            pr[2 + d] = O;
            if (d == 0) {
                pr[0] = M;
                pr[1] = L;
            }
        }
    }
}

__global__ __launch_bounds__(kD) void attn_merge(AttnArgs a)
{
    const int hq = blockIdx.x, b = blockIdx.y;
    const int d = threadIdx.x;
    const long long stride = (long long)a.B * a.Hq * kPartStride;
    const float* pr = a.part + ((long long)b * a.Hq + hq) * kPartStride;
    float M = -INFINITY;
    for (int s = 0; s < a.splits; ++s) M = fmaxf(M, pr[s * stride]);
    float L = 0.f, O = 0.f;
    if (M != -INFINITY) {
        for (int s = 0; s < a.splits; ++s) {
            const float* q = pr + s * stride;
            const float f = __builtin_amdgcn_exp2f(q[0] - M);
            L = fmaf(q[1], f, L);
            O = fmaf(q[2 + d], f, O);
        }
    }
    a.out[((long long)b * a.Hq + hq) * kD + d] = (L > 0.f) ? O / L : 0.f;
    if (d == 0 && a.lse)
        a.lse[(long long)b * a.Hq + hq] = (L > 0.f) ? (M + __log2f(L)) * 0.69314718055994530942f : -INFINITY;
}

template <int GQ>
static void launch_gq(const AttnArgs& a, hipStream_t st)
{
    hipLaunchKernelGGL(attn_decode<GQ>, dim3(a.splits, a.Hkv, a.B), dim3(kAttnThreads), 0, st, a);
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t st)
{
    const int gq = a.Hq / a.Hkv;
    switch (gq) {
    case 1: launch_gq<1>(a, st); break;
    case 2: launch_gq<2>(a, st); break;
    case 3: launch_gq<3>(a, st); break;
    case 4: launch_gq<4>(a, st); break;
    case 5: launch_gq<5>(a, st); break;
    case 6: launch_gq<6>(a, st); break;
    case 7: launch_gq<7>(a, st); break;
    case 8: launch_gq<8>(a, st); break;
    default: return hipErrorInvalidValue;
    }
    if (a.splits > 1) hipLaunchKernelGGL(attn_merge, dim3(a.Hq, a.B), dim3(kD), 0, st, a);
    return hipGetLastError();
}

}  // namespace dkv
