// k_attention.hip -- decode attention over the differentiated paged KV cache
// for gfx950 (DiffKV Eq. (1) of Sec. 2.1, kernel structure of Sec. 6.2).
//
// Grid (splits, Hkv, B); a workgroup of four waves owns one table (one
// sequence, one KV head) -- or one page range of it when the sequence is
// split -- and all GQ query heads that read it.  Each wave walks its share of
// the table's pages, high-precision pages first, then low-precision pages,
// and loads page i+1 into registers while it computes page i.  The wave's
// page IDs are fetched 64 at a time into one VGPR and read back with
// v_readlane, so a page's loads wait on nothing but the previous page.
//
// Lane mapping inside a wave (64 lanes = 4 rows of 16):
//   key phase    lane = grp*16 + j: token j (and j+16 on 32-token pages),
//                32-dim group grp.  The lane holds q of its group as fp16
//                pairs and computes sum(q*code) with v_dot2_f32_f16 on codes
//                turned into fp16 denormals (exact, one v_perm or AND per two
//                codes), then s*sum + z*sum(q) (scale and zero factored out of
//                the dot product); the four groups of a token are summed with
//                v_permlane16/32_swap.
//   softmax      online, base 2, per query head, with a lazily raised max: the
//                page max (DPP row ops) is only taken when a logit exceeds
//                the running max by more than 2^8.
//   value phase  lane owns dims 2*lane, 2*lane+1 (its row's group).  The
//                weights p*s_v (fp32) of the row's tokens go through LDS (one
//                broadcast read per token for all heads) into fp32 FMAs with
//                the codes; the zero-point term sum(p*z_v) is accumulated per
//                lane and added once at the end.  (fp16 weights with v_dot2
//                would halve these FMAs but miss the 2e-3 bound when one
//                token dominates.)
// The four waves' (max, sum, acc) states merge through LDS; with splits > 1
// the per-range states go to the workspace and attn_merge combines them.
#include "internal.hpp"

namespace dkv {

constexpr int kAttnWaves = 4;
constexpr int kAttnThreads = kAttnWaves * kWave;
constexpr int kPartStride = kD + 2;

// Byte offsets of the supported page layout (checked by the API against the
// caller's diffkv_layout).
constexpr int kOffKcHi = 0, kOffKmHi = 2048, kOffVcHi = 2304, kOffVmHi = 3328;
constexpr int kOffKcLo = 0, kOffKmLo = 2048, kOffVcLo = 2560, kOffVmLo = 3584;

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

// ---- cross-lane helpers ------------------------------------------------------
// sum of the four rows (lanes l, l^16, l^32, l^48), result in every lane
__device__ __forceinline__ float rows_sum4(float x)
{
    auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

template <int CTRL>
__device__ __forceinline__ float dpp(float x)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float fmax_sel(float a, float b) { return a > b ? a : b; }

// max over the 16 lanes of each row, result in every lane of the row
__device__ __forceinline__ float row_max16(float x)
{
    x = fmax_sel(x, dpp<0x128>(x));  // row_ror:8
    x = fmax_sel(x, dpp<0x124>(x));  // row_ror:4
    x = fmax_sel(x, dpp<0x122>(x));  // row_ror:2
    x = fmax_sel(x, dpp<0x121>(x));  // row_ror:1
    return x;
}
__device__ __forceinline__ float row_sum16(float x)
{
    x += dpp<0x128>(x);
    x += dpp<0x124>(x);
    x += dpp<0x122>(x);
    x += dpp<0x121>(x);
    return x;
}

// ---- code conversions ---------------------------------------------------------
// Key codes become fp16 *denormals* (bit pattern = code, value = code * 2^-24):
// one v_perm or one AND per two codes, exact, and exact again in
// v_dot2_f32_f16 (its fp16 products are exact in fp32).  The 2^24 is folded
// into the key scale.  Pairs hold dims (d, d+4) of each 8-dim block, the
// pairing the q registers use.
__device__ __forceinline__ uint32_t perm_pair(uint32_t w_hi, uint32_t w_lo, int a)
{
    // bytes: [w_lo.byte a, 0, w_hi.byte a, 0]
    return __builtin_amdgcn_perm(w_hi, w_lo, 0x0C000C00u | ((uint32_t)(4 + a) << 16) | (uint32_t)a);
}

__device__ __forceinline__ float dot2(half2_t a, uint32_t b, float c)
{
    return __builtin_amdgcn_fdot2(a, __builtin_bit_cast(half2_t, b), c, false);
}

constexpr float kTwo24 = 16777216.0f;

// Raw bytes of one page as one lane needs them.
struct PageRaw {
    uint4 k0, k1;  // high: K8 chunks 2g, 2g+1 of token j; low: K4 chunk g of tokens j, j+16
    uint4 vr;      // V code rows of dims 2*lane, 2*lane+1
    uint32_t m0, m1, m2, m3;  // high: kmeta, vmeta; low: kmeta j, kmeta j+16, vmeta j, vmeta j+16
};

__device__ __forceinline__ uint4 ld16(const uint8_t* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ uint32_t ld4(const uint8_t* p) { return *reinterpret_cast<const uint32_t*>(p); }

__device__ __forceinline__ void load_page(PageRaw& r, const uint8_t* pg, bool hi, int lane)
{
    const int grp = lane >> 4, jl = lane & 15;
    if (hi) {
        r.k0 = ld16(pg + kOffKcHi + ((2 * grp) * kTHi + jl) * 16);
        r.k1 = ld16(pg + kOffKcHi + ((2 * grp + 1) * kTHi + jl) * 16);
        r.vr = ld16(pg + kOffVcHi + lane * 16);
        r.m0 = ld4(pg + kOffKmHi + (jl * kNG + grp) * 4);
        r.m1 = ld4(pg + kOffVmHi + (grp * kTHi + jl) * 4);
        r.m2 = r.m3 = 0;
    } else {
        r.k0 = ld16(pg + kOffKcLo + (grp * kTLo + jl) * 16);
        r.k1 = ld16(pg + kOffKcLo + (grp * kTLo + jl + 16) * 16);
        r.vr = ld16(pg + kOffVcLo + lane * 16);
        r.m0 = ld4(pg + kOffKmLo + (jl * kNG + grp) * 4);
        r.m1 = ld4(pg + kOffKmLo + ((jl + 16) * kNG + grp) * 4);
        r.m2 = ld4(pg + kOffVmLo + (grp * kTLo + jl) * 4);
        r.m3 = ld4(pg + kOffVmLo + (grp * kTLo + jl + 16) * 4);
    }
}

template <int GQ>
struct WaveState {
    float m[GQ];       // running max (log2 domain), wave-uniform
    float l[GQ];       // this lane's share of the running sum
    float z[GQ];       // this lane's share of sum(p * z_v) for its row's group
    float acc[GQ][2];  // dims 2*lane, 2*lane+1
};

// LDS for the softmax weights of one page: [row][token][head] fp32, rows
// padded by four floats so the four rows' broadcast reads hit different banks.
template <int GQ>
struct CoefLds {
    static constexpr int kH = GQ <= 4 ? 4 : 8;
    static constexpr int kRow = kTLo * kH + 4;
    float v[kAttnWaves][4 * kRow];
};

template <int GQ>
__device__ __forceinline__ void read_coef(const float* row, int j, float (&c)[GQ])
{
    const float* p = row + j * CoefLds<GQ>::kH;
    float t[8];
    const float4 v0 = *reinterpret_cast<const float4*>(p);
    t[0] = v0.x; t[1] = v0.y; t[2] = v0.z; t[3] = v0.w;
    if constexpr (GQ > 4) {
        const float4 v1 = *reinterpret_cast<const float4*>(p + 4);
        t[4] = v1.x; t[5] = v1.y; t[6] = v1.z; t[7] = v1.w;
    }
#pragma unroll
    for (int h = 0; h < GQ; ++h) c[h] = t[h];
}

// Softmax weights are exp2(logit - m) with a running max m that is only
// raised when a logit exceeds it by more than kSlack (weights stay <= 2^8).
constexpr float kSlack = 8.0f;

// One page: logits, online softmax, weighted value sum.  NT = tokens per lane.
template <int GQ, int NT>
__device__ __forceinline__ void do_page(WaveState<GQ>& st, const PageRaw& r, const half2_t (&q2)[GQ][16],
                                        const float (&qsum)[GQ], float sl2, int n_valid, int lane,
                                        float* coef_row)
{
    const int jl = lane & 15;
    float lg[NT][GQ];
#pragma unroll
    for (int tk = 0; tk < NT; ++tk) {
        const uint32_t km = tk ? r.m1 : r.m0;
        const float ks = h2f(km & 0xffffu) * (kTwo24 * sl2), kz = h2f(km >> 16) * sl2;
        float dlo[GQ], dhi[GQ];
#pragma unroll
        for (int hh = 0; hh < GQ; ++hh) dlo[hh] = dhi[hh] = 0.f;
        if (NT == 1) {
            // K8: two dwords (8 dims) -> four (d, d+4) pairs, one v_perm each
            const uint32_t w[8] = {r.k0.x, r.k0.y, r.k0.z, r.k0.w, r.k1.x, r.k1.y, r.k1.z, r.k1.w};
#pragma unroll
            for (int m = 0; m < 4; ++m) {
#pragma unroll
                for (int a2 = 0; a2 < 4; ++a2) {
                    const uint32_t x = perm_pair(w[2 * m + 1], w[2 * m], a2);
#pragma unroll
                    for (int hh = 0; hh < GQ; ++hh) dlo[hh] = dot2(q2[hh][4 * m + a2], x, dlo[hh]);
                }
            }
        } else {
            // K4: one dword (8 dims); nibbles a and a+4 sit in the two halves
            const uint4 kk = tk ? r.k1 : r.k0;
            const uint32_t w[4] = {kk.x, kk.y, kk.z, kk.w};
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const uint32_t v = w[m], v8 = w[m] >> 8;
                const uint32_t x0 = v & 0x000F000Fu, x1 = v & 0x00F000F0u;
                const uint32_t x2 = v8 & 0x000F000Fu, x3 = v8 & 0x00F000F0u;
#pragma unroll
                for (int hh = 0; hh < GQ; ++hh) {
                    dlo[hh] = dot2(q2[hh][4 * m + 0], x0, dlo[hh]);
                    dhi[hh] = dot2(q2[hh][4 * m + 1], x1, dhi[hh]);
                    dlo[hh] = dot2(q2[hh][4 * m + 2], x2, dlo[hh]);
                    dhi[hh] = dot2(q2[hh][4 * m + 3], x3, dhi[hh]);
                }
            }
        }
        const bool valid = jl + 16 * tk < n_valid;
#pragma unroll
        for (int hh = 0; hh < GQ; ++hh) {
            const float d = NT == 1 ? dlo[hh] : fmaf(dhi[hh], 0.0625f, dlo[hh]);
            const float part = rows_sum4(fmaf(ks, d, kz * qsum[hh]));
            lg[tk][hh] = valid ? part : -INFINITY;
        }
    }
    // online softmax with a lazily raised max
    bool raise = false;
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh)
#pragma unroll
        for (int tk = 0; tk < NT; ++tk) raise |= lg[tk][hh] > st.m[hh] + kSlack;
    if (__builtin_amdgcn_ballot_w64(raise)) {
#pragma unroll
        for (int hh = 0; hh < GQ; ++hh) {
            float mx = lg[0][hh];
            if (NT > 1) mx = fmax_sel(mx, lg[NT - 1][hh]);
            mx = row_max16(mx);
            const float mnew = fmax_sel(st.m[hh], mx);
            const float alpha = __builtin_amdgcn_exp2f(st.m[hh] - mnew);
            st.m[hh] = mnew;
            st.l[hh] *= alpha;
            st.z[hh] *= alpha;
            st.acc[hh][0] *= alpha;
            st.acc[hh][1] *= alpha;
        }
    }
    float p[NT][GQ];
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh) {
#pragma unroll
        for (int tk = 0; tk < NT; ++tk) {
            p[tk][hh] = __builtin_amdgcn_exp2f(lg[tk][hh] - st.m[hh]);
            st.l[hh] += p[tk][hh];
        }
    }
    // Weights p*s_v (fp32) to LDS for the row's lanes; zero-point term sum(p*z_v)
    // in registers.
    constexpr int kH = CoefLds<GQ>::kH;
#pragma unroll
    for (int tk = 0; tk < NT; ++tk) {
        const uint32_t vm = NT == 1 ? r.m1 : (tk ? r.m3 : r.m2);
        const float vs = h2f(vm & 0xffffu), vz = h2f(vm >> 16);
        float c[kH];
#pragma unroll
        for (int hh = 0; hh < kH; ++hh) c[hh] = hh < GQ ? p[tk][hh] * vs : 0.f;
#pragma unroll
        for (int hh = 0; hh < GQ; ++hh) st.z[hh] = fmaf(p[tk][hh], vz, st.z[hh]);
        float* dst = coef_row + (jl + 16 * tk) * kH;
#pragma unroll
        for (int i = 0; i < kH; i += 4)
            *reinterpret_cast<float4*>(dst + i) = make_float4(c[i], c[i + 1], c[i + 2], c[i + 3]);
    }
    __builtin_amdgcn_wave_barrier();
    // value phase: tokens of this row's group, codes of dims 2*lane, 2*lane+1.
    // The weights of 16 tokens are read from LDS in one burst before their
    // FMAs, so the reads overlap each other instead of stalling per token.
    const uint32_t w[4] = {r.vr.x, r.vr.y, r.vr.z, r.vr.w};
#pragma unroll
    for (int half = 0; half < NT; ++half) {
        float cf[16][GQ];
#pragma unroll
        for (int j = 0; j < 16; ++j) read_coef<GQ>(coef_row, 16 * half + j, cf[j]);
        if constexpr (NT == 1) {
            // 16 tokens x 4 bits per 64-bit row: dword (j >> 3), nibble (j & 7)
#pragma unroll
            for (int dw = 0; dw < 2; ++dw) {
                const uint32_t a = w[dw], b = w[2 + dw];
                const uint32_t alo = a & 0x0F0F0F0Fu, ahi = (a >> 4) & 0x0F0F0F0Fu;
                const uint32_t blo = b & 0x0F0F0F0Fu, bhi = (b >> 4) & 0x0F0F0F0Fu;
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const int j = 8 * dw + k;
                    const uint32_t sa = (k & 1) ? ahi : alo, sb = (k & 1) ? bhi : blo;
                    const float c0 = (float)((sa >> (8 * (k >> 1))) & 0xFFu);
                    const float c1 = (float)((sb >> (8 * (k >> 1))) & 0xFFu);
#pragma unroll
                    for (int hh = 0; hh < GQ; ++hh) {
                        st.acc[hh][0] = fmaf(cf[j][hh], c0, st.acc[hh][0]);
                        st.acc[hh][1] = fmaf(cf[j][hh], c1, st.acc[hh][1]);
                    }
                }
            }
        } else {
            // 32 tokens x 2 bits per 64-bit row: tokens 16*half.. in dword `half`, crumb j & 15
            const uint32_t a = w[half], b = w[2 + half];
#pragma unroll
            for (int sh = 0; sh < 4; ++sh) {
                const uint32_t sa = (a >> (2 * sh)) & 0x03030303u, sb = (b >> (2 * sh)) & 0x03030303u;
#pragma unroll
                for (int by = 0; by < 4; ++by) {
                    const int j = 4 * by + sh;
                    const float c0 = (float)((sa >> (8 * by)) & 0xFFu);
                    const float c1 = (float)((sb >> (8 * by)) & 0xFFu);
#pragma unroll
                    for (int hh = 0; hh < GQ; ++hh) {
                        st.acc[hh][0] = fmaf(cf[j][hh], c0, st.acc[hh][0]);
                        st.acc[hh][1] = fmaf(cf[j][hh], c1, st.acc[hh][1]);
                    }
                }
            }
        }
    }
    __builtin_amdgcn_wave_barrier();
}

template <int GQ>
__global__ __launch_bounds__(kAttnThreads) void attn_decode(AttnArgs a)
{
    const int split = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int t = b * a.Hkv + h;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int grp = lane >> 4;
    const int P = a.p_max;
    const int len_hi = a.len[2 * t], len_lo = a.len[2 * t + 1];
    // page counts from the section lengths, clamped to the table width
    int ph = (len_hi + kTHi - 1) / kTHi;
    int pl = (len_lo + kTLo - 1) / kTLo;
    ph = ph < 0 ? 0 : (ph > P ? P : ph);
    pl = pl < 0 ? 0 : (pl > P - ph ? P - ph : pl);
    const int np = ph + pl;
    const int p0 = (int)(((long long)split * np) / a.splits);
    const int p1 = (int)(((long long)(split + 1) * np) / a.splits);
    const int nmine = p1 - p0 > wave ? (p1 - p0 - wave + kAttnWaves - 1) / kAttnWaves : 0;
    const int32_t* trow = a.page_table + (long long)t * P;

    __shared__ CoefLds<GQ> s_coef;
    float* coef_row = &s_coef.v[wave][grp * CoefLds<GQ>::kRow];

    // q of this lane's group as fp16 pairs (d, d+4) of each 8-dim block, and its sum
    half2_t q2[GQ][16];
    float qsum[GQ];
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh) {
        const uint4* qp = reinterpret_cast<const uint4*>(a.q + ((long long)b * a.Hq + h * GQ + hh) * kD + grp * kG);
        float s = 0.f;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const uint4 v = qp[m];  // dims 8m .. 8m+7 as four fp16 pairs (d, d+1)
#pragma unroll
            for (int a2 = 0; a2 < 4; ++a2) {
                const uint32_t lo = a2 < 2 ? v.x : v.y, hi = a2 < 2 ? v.z : v.w;
                const uint32_t sh = (a2 & 1) * 16;
                const uint32_t pr = ((lo >> sh) & 0xffffu) | (((hi >> sh) & 0xffffu) << 16);
                q2[hh][4 * m + a2] = __builtin_bit_cast(half2_t, pr);
                s += (float)q2[hh][4 * m + a2].x + (float)q2[hh][4 * m + a2].y;
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
    const long long npool = a.num_pages;
    const long long page_bytes = a.page_bytes;

    // page IDs of this wave's pages, 64 per VGPR load
    auto page_of = [&](int i) { return p0 + wave + kAttnWaves * i; };
    auto slot_of = [&](int p) { return p < ph ? p : P - 1 - (p - ph); };
    int idv = -1;
    auto load_ids = [&](int i0) {
        const int i = i0 + lane;
        idv = i < nmine ? trow[slot_of(page_of(i))] : -1;
    };
    PageRaw cur, nxt;
    int id_cur = -1;
    if (nmine > 0) {
        load_ids(0);
        id_cur = __builtin_amdgcn_readfirstlane(idv);
        if ((unsigned long long)id_cur < (unsigned long long)npool)
            load_page(cur, a.pool + id_cur * page_bytes, page_of(0) < ph, lane);
    }
    for (int i = 0; i < nmine; ++i) {
        const int p = page_of(i);
        const bool hi = p < ph;
        int id_nxt = -1;
        if (i + 1 < nmine) {
            if (((i + 1) & 63) == 0) load_ids(i + 1);
            id_nxt = __builtin_amdgcn_readlane(idv, (i + 1) & 63);
            if ((unsigned long long)id_nxt < (unsigned long long)npool)
                load_page(nxt, a.pool + id_nxt * page_bytes, page_of(i + 1) < ph, lane);
        }
        if ((unsigned long long)id_cur < (unsigned long long)npool) {  // never read outside the pool
            if (hi) {
                do_page<GQ, 1>(st, cur, q2, qsum, sl2, len_hi - p * kTHi, lane, coef_row);
            } else {
                do_page<GQ, 2>(st, cur, q2, qsum, sl2, len_lo - (p - ph) * kTLo, lane, coef_row);
            }
        }
        cur = nxt;
        id_cur = id_nxt;
    }

    // ---- finish the wave: row sums of l and of the zero-point term ----------
    __shared__ float s_m[kAttnWaves][8];
    __shared__ float s_l[kAttnWaves][8];
    __shared__ float s_acc[kAttnWaves][8][kD];
#pragma unroll
    for (int hh = 0; hh < GQ; ++hh) {
        const float l = row_sum16(st.l[hh]);
        const float z = row_sum16(st.z[hh]);
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
        for (int w = 0; w < kAttnWaves; ++w) M = fmax_sel(M, s_m[w][hh]);
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
    for (int s = 0; s < a.splits; ++s) M = fmax_sel(M, pr[s * stride]);
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

bool attention_layout_matches(const diffkv_layout* L)
{
    return L->off_kcode[0] == kOffKcHi && L->off_kmeta[0] == kOffKmHi && L->off_vcode[0] == kOffVcHi &&
           L->off_vmeta[0] == kOffVmHi && L->off_kcode[1] == kOffKcLo && L->off_kmeta[1] == kOffKmLo &&
           L->off_vcode[1] == kOffVcLo && L->off_vmeta[1] == kOffVmLo;
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
