// k_prompt.hip -- prompt-phase significance (Sec. 4) on the matrix cores.
//
// Token p of an N-token prompt is scored by the mean, over the queries
// j = p..N-1, of the causal softmax probability query j gives it, the KV
// head's g query heads combined by their maximum per query.  Two passes over
// the prompt's fp16 q and k, both built on v_mfma_f32_16x16x32_f16 tiles
// (fp16 products, exact in fp32, fp32 sums):
//
//   ps_rows  per (sequence, KV head, block of query positions): the log2-sum-
//            exp of every query row of the group's heads over keys 0..j.  The
//            queries sit in registers as MFMA B operands (all g heads of 16
//            positions per wave, more positions when g is small so that every
//            key fragment read from LDS feeds at least four MFMAs); key blocks
//            of 64 rows are staged through LDS, double buffered, the next one
//            fetched into registers while the current one is multiplied.  The
//            running max is raised lazily (only when a row's new logits pass
//            it by more than 2^8, a wave-uniform branch), so most key tiles
//            cost one exp per logit and no rescale.
//   ps_cols  per (sequence, KV head, block of 256 keys): the keys sit in
//            registers as A operands (64 per wave); tiles of 16 query
//            positions x g heads, with their row log2-sum-exps, are staged
//            through LDS.  Per (key, query) the g logits are reduced by max
//            after subtracting each head's row normalizer, so one exp2 gives
//            the group's maximum probability; column sums stay per lane until
//            a single cross-lane reduction at the end, so no atomics and a
//            fixed summation order.
//
// Work order: the blocks of one (sequence, KV head) are numbered contiguously
// and mapped to one XCD (consecutive workgroups go round-robin over the 8
// XCDs), so that the key and query tiles they re-read stay in that XCD's L2;
// within a pair the heaviest blocks start first.

#include "internal.hpp"

namespace dkv {

namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kPsThreads = 256;         // 4 waves
constexpr int kKeyBlock = 64;           // keys per LDS stage of the row pass
constexpr int kColKeys = 256;           // keys per workgroup of the column pass (64 per wave)
constexpr int kRowChunks = 17;          // 16-byte chunks per LDS row: 128 halfs + 16 B pad
constexpr float kSlack = 8.0f;          // lazy-max slack of the row pass (log2 units)
constexpr float kLog2e = 1.4426950408889634f;

template <int G>
struct PsShape {
    static constexpr int QI = G <= 4 ? 32 : 16;      // query positions per LDS stage of the column pass
    static constexpr int QT = G >= 3 ? 1 : 4 / G;   // 16-position query tiles per head per wave
    static constexpr int PW = 16 * QT;               // query positions per wave
    static constexpr int PB = 4 * PW;                // query positions per workgroup
};

__device__ __forceinline__ f4 mfma16(h8 a, h8 b, f4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float max3f(float a, float b, float c) { return __builtin_fmaxf(__builtin_fmaxf(a, b), c); }

// Logical block of workgroup i among n: XCD x = i % 8 runs the logical range
// [x * (n / 8) + min(x, n % 8), ...) in order.  A bijection of [0, n).
__device__ __forceinline__ long long xcd_block(long long i, long long n)
{
    const long long per = n / 8, rem = n % 8, x = i % 8, k = i / 8;
    return x * per + (x < rem ? x : rem) + k;
}

__device__ __forceinline__ h8 zero8()
{
    h8 z;
    for (int i = 0; i < 8; i++) z[i] = (_Float16)0.0f;
    return z;
}

}  // namespace

// Row starts and lengths: off[b] = sum of the clamped lengths before b; a
// sequence's rows are cut at total_new, so no pass touches a row >= total_new.
__global__ __launch_bounds__(kPsThreads) void ps_offsets(PromptArgs a)
{
    __shared__ long long part[kPsThreads];
    const int tid = threadIdx.x;
    const int per = (a.B + kPsThreads - 1) / kPsThreads;
    const int b0 = tid * per, b1 = min(a.B, b0 + per);
    long long s = 0;
    for (int b = b0; b < b1; b++) s += min(max(a.new_len[b], 0), a.max_new);
    part[tid] = s;
    __syncthreads();
    for (int d = 1; d < kPsThreads; d <<= 1) {
        const long long v = tid >= d ? part[tid - d] : 0;
        __syncthreads();
        part[tid] += v;
        __syncthreads();
    }
    long long off = part[tid] - s;
    for (int b = b0; b < b1; b++) {
        const int n = min(max(a.new_len[b], 0), a.max_new);
        const long long room = a.total_new - off;
        a.off[b] = off;
        a.nlen[b] = (int)(room <= 0 ? 0 : (n < room ? n : room));
        off += n;
    }
}

// Pass 1: lse2[row][hq] = log2 sum_{p <= j} exp2(scale_log2 * q_j . k_p).
template <int G>
__global__ __launch_bounds__(kPsThreads) void ps_rows(PromptArgs a)
{
    constexpr int QT = PsShape<G>::QT, PW = PsShape<G>::PW, PB = PsShape<G>::PB;
    __shared__ h8 sk[2][kKeyBlock][kRowChunks];

    const int nqb = (a.max_new + PB - 1) / PB;
    const long long nblk = (long long)a.B * a.Hkv * nqb;
    const long long lb = xcd_block(blockIdx.x, nblk);
    const int bh = (int)(lb / nqb);
    const int qb = nqb - 1 - (int)(lb - (long long)bh * nqb);
    const int b = bh / a.Hkv, h = bh - b * a.Hkv;
    const int N = a.nlen[b];
    const long long off = a.off[b];
    const int q0 = qb * PB;
    if (q0 >= N) return;

    const int lane = threadIdx.x & (kWave - 1);
    const int w = wave_index();
    const int col = lane & 15, grp = lane >> 4;
    const int wq0 = q0 + w * PW;
    const float c = a.scale_log2;

    h8 qf[QT][G][4];
    for (int qt = 0; qt < QT; qt++) {
        const int j = wq0 + qt * 16 + col;
        for (int t = 0; t < G; t++) {
            const h8* src = reinterpret_cast<const h8*>(a.q + ((off + j) * a.Hq + h * G + t) * kD);
            for (int s = 0; s < 4; s++) qf[qt][t][s] = j < N ? src[4 * s + grp] : zero8();
        }
    }
    float m[QT][G], sum[QT][G];
    for (int qt = 0; qt < QT; qt++)
        for (int t = 0; t < G; t++) {
            m[qt][t] = -1e30f;
            sum[qt][t] = 0.0f;
        }

    const int last = min(N, q0 + PB) - 1;
    const int nkb = last / kKeyBlock + 1;
    constexpr int kPer = kKeyBlock * 16 / kPsThreads;    // 16-byte chunks staged per thread
    const int srow = threadIdx.x / (16 / kPer), spart = threadIdx.x % (16 / kPer);
    h8 pre[kPer];
    auto fetch = [&](int kb) {
        const int p = kb * kKeyBlock + srow;
        const h8* src = reinterpret_cast<const h8*>(a.k + ((off + p) * a.Hkv + h) * kD) + spart * kPer;
        for (int i = 0; i < kPer; i++) pre[i] = p < N ? src[i] : zero8();
    };
    auto stash = [&](int buf) {
        for (int i = 0; i < kPer; i++) sk[buf][srow][spart * kPer + i] = pre[i];
    };
    fetch(0);
    stash(0);
    __syncthreads();
    for (int kb = 0; kb < nkb; kb++) {
        const int buf = kb & 1;
        if (kb + 1 < nkb) fetch(kb + 1);
        const int kbase = kb * kKeyBlock;
        // waves whose positions all precede the block skip it; a block whose last
        // key passes the wave's first position needs the causal mask (which also
        // removes keys >= N: those lie after every valid position)
        if (kbase < wq0 + PW && wq0 < N) {
            const bool need_mask = kbase + kKeyBlock - 1 > wq0;
            for (int kt = 0; kt < kKeyBlock / 16; kt++) {
                h8 af[4];
                for (int s = 0; s < 4; s++) af[s] = sk[buf][kt * 16 + col][4 * s + grp];
                const int key0 = kbase + kt * 16 + 4 * grp;
                for (int qt = 0; qt < QT; qt++) {
                    const int j = wq0 + qt * 16 + col;
                    for (int t = 0; t < G; t++) {
                        f4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
                        for (int s = 0; s < 4; s++) acc = mfma16(af[s], qf[qt][t][s], acc);
                        if (need_mask)
                            for (int i = 0; i < 4; i++)
                                if (key0 + i > j) acc[i] = -__builtin_huge_valf();
                        const float bm = max3f(acc[0], acc[1], fmaxf(acc[2], acc[3])) * c;
                        if (__builtin_amdgcn_ballot_w64(bm > m[qt][t] + kSlack)) {
                            const float mn = fmaxf(m[qt][t], bm);
                            sum[qt][t] *= fast_exp2(m[qt][t] - mn);
                            m[qt][t] = mn;
                        }
                        const float nm = -m[qt][t];
                        sum[qt][t] += (fast_exp2(fmaf(acc[0], c, nm)) + fast_exp2(fmaf(acc[1], c, nm))) +
                                      (fast_exp2(fmaf(acc[2], c, nm)) + fast_exp2(fmaf(acc[3], c, nm)));
                    }
                }
            }
        }
        if (kb + 1 < nkb) stash(buf ^ 1);
        __syncthreads();
    }
    // combine the four row groups of each column (lanes col, col+16, col+32, col+48)
    for (int qt = 0; qt < QT; qt++) {
        const int j = wq0 + qt * 16 + col;
        for (int t = 0; t < G; t++) {
            float mx = fmaxf(m[qt][t], __shfl_xor(m[qt][t], 16));
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            float sm = sum[qt][t] * fast_exp2(m[qt][t] - mx);
            sm += __shfl_xor(sm, 16);
            sm += __shfl_xor(sm, 32);
            if (grp == 0 && j < N) a.lse2[(off + j) * a.Hq + h * G + t] = mx + __builtin_amdgcn_logf(sm);
        }
    }
}

// Pass 2: score[row][h] = (1 / (N - p)) sum_{j >= p} max_t exp2(scale_log2 * q_j,t . k_p - lse2[j][t]).
template <int G>
__global__ __launch_bounds__(kPsThreads) void ps_cols(PromptArgs a)
{
    constexpr int QI = PsShape<G>::QI;
    constexpr int NR = G * QI * 16 / kPsThreads;     // 16-byte chunks of q staged per thread
    __shared__ h8 sq[2][G][QI][kRowChunks];
    __shared__ float sl[2][G][QI];

    const int nkb = (a.max_new + kColKeys - 1) / kColKeys;
    const long long nblk = (long long)a.B * a.Hkv * nkb;
    const long long lb = xcd_block(blockIdx.x, nblk);
    const int bh = (int)(lb / nkb);
    const int kb = (int)(lb - (long long)bh * nkb);
    const int b = bh / a.Hkv, h = bh - b * a.Hkv;
    const int N = a.nlen[b];
    const long long off = a.off[b];
    const int k0 = kb * kColKeys;
    if (k0 >= N) return;

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int w = wave_index();
    const int col = lane & 15, grp = lane >> 4;
    const int wk0 = k0 + w * 64;
    const float c = a.scale_log2;
    const float inv_c = 1.0f / c;

    h8 kf[4][4];
    for (int kt = 0; kt < 4; kt++) {
        const int p = wk0 + kt * 16 + col;
        const h8* src = reinterpret_cast<const h8*>(a.k + ((off + p) * a.Hkv + h) * kD);
        for (int s = 0; s < 4; s++) kf[kt][s] = p < N ? src[4 * s + grp] : zero8();
    }
    float cs[4][4];
    for (int kt = 0; kt < 4; kt++)
        for (int i = 0; i < 4; i++) cs[kt][i] = 0.0f;

    const int nq = (N - k0 + QI - 1) / QI;
    h8 pq[NR];
    float pl = 0.0f;
    auto fetch = [&](int it) {
        const int j0 = k0 + it * QI;
        for (int r = 0; r < NR; r++) {
            const int cidx = r * kPsThreads + tid;
            const int row = cidx >> 4, pos = row / G, t = row - pos * G;
            const int j = j0 + pos;
            const h8* src = reinterpret_cast<const h8*>(a.q + ((off + j) * a.Hq + h * G + t) * kD);
            pq[r] = j < N ? src[cidx & 15] : zero8();
        }
        if (tid < QI * G) {
            const int pos = tid / G, t = tid - pos * G;
            const int j = j0 + pos;
            const long long e = (off + j) * a.Hq + h * G + t;
            pl = j >= N ? __builtin_huge_valf() : (a.lse ? a.lse[e] * kLog2e : a.lse2[e]);
        }
    };
    auto stash = [&](int buf) {
        for (int r = 0; r < NR; r++) {
            const int cidx = r * kPsThreads + tid;
            const int row = cidx >> 4, pos = row / G, t = row - pos * G;
            sq[buf][t][pos][cidx & 15] = pq[r];
        }
        if (tid < QI * G) {
            const int pos = tid / G, t = tid - pos * G;
            sl[buf][t][pos] = pl;
        }
    };
    fetch(0);
    stash(0);
    __syncthreads();
    for (int it = 0; it < nq; it++) {
        const int buf = it & 1;
        if (it + 1 < nq) fetch(it + 1);
        for (int sub = 0; sub < QI / 16; sub++) {
            const int j0 = k0 + it * QI + sub * 16;
            if (j0 + 15 < wk0 || wk0 >= N) continue;   // no query of the tile reaches the wave's keys
            const bool diag = j0 < wk0 + 63;
            // the MFMA accumulates onto -lse/c, so acc = S - lse/c and the maximum over the
            // heads needs no per-head arithmetic; exp2(c * max) is the group's probability
            f4 mx[4];
            for (int t = 0; t < G; t += 2) {
                const bool pair = t + 1 < G;
                h8 bf0[4], bf1[4];
                for (int s = 0; s < 4; s++) bf0[s] = sq[buf][t][sub * 16 + col][4 * s + grp];
                if (pair)
                    for (int s = 0; s < 4; s++) bf1[s] = sq[buf][t + 1][sub * 16 + col][4 * s + grp];
                const float z0 = -sl[buf][t][sub * 16 + col] * inv_c;
                const float z1 = pair ? -sl[buf][t + 1][sub * 16 + col] * inv_c : 0.0f;
                for (int kt = 0; kt < 4; kt++) {
                    f4 acc0 = {z0, z0, z0, z0};
                    for (int s = 0; s < 4; s++) acc0 = mfma16(kf[kt][s], bf0[s], acc0);
                    if (pair) {
                        f4 acc1 = {z1, z1, z1, z1};
                        for (int s = 0; s < 4; s++) acc1 = mfma16(kf[kt][s], bf1[s], acc1);
                        for (int i = 0; i < 4; i++)
                            mx[kt][i] = t == 0 ? fmaxf(acc0[i], acc1[i]) : max3f(mx[kt][i], acc0[i], acc1[i]);
                    } else {
                        for (int i = 0; i < 4; i++) mx[kt][i] = t == 0 ? acc0[i] : fmaxf(mx[kt][i], acc0[i]);
                    }
                }
            }
            const int j = j0 + col;
            for (int kt = 0; kt < 4; kt++)
                for (int i = 0; i < 4; i++) {
                    float v = fast_exp2(mx[kt][i] * c);
                    if (diag && wk0 + kt * 16 + 4 * grp + i > j) v = 0.0f;
                    cs[kt][i] += v;
                }
        }
        if (it + 1 < nq) stash(buf ^ 1);
        __syncthreads();
    }
    for (int kt = 0; kt < 4; kt++)
        for (int i = 0; i < 4; i++) {
            float v = cs[kt][i];
            v += __shfl_xor(v, 1);
            v += __shfl_xor(v, 2);
            v += __shfl_xor(v, 4);
            v += __shfl_xor(v, 8);
            const int p = wk0 + kt * 16 + 4 * grp + i;
            if (col == 0 && p < N) a.score[(off + p) * a.Hkv + h] = v / (float)(N - p);
        }
}

namespace {

template <int G>
hipError_t launch_prompt_g(const PromptArgs& a, hipStream_t st)
{
    hipError_t e;
    if (!a.lse) {
        const long long nqb = (a.max_new + PsShape<G>::PB - 1) / PsShape<G>::PB;
        const long long grid = (long long)a.B * a.Hkv * nqb;
        if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
        if ((e = launch1(ps_rows<G>, (unsigned)grid, kPsThreads, st, a)) != hipSuccess) return e;
    }
    const long long grid = (long long)a.B * a.Hkv * ((a.max_new + kColKeys - 1) / kColKeys);
    if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
    return launch1(ps_cols<G>, (unsigned)grid, kPsThreads, st, a);
}

}  // namespace

hipError_t launch_prompt_significance(const PromptArgs& a, int g, hipStream_t st)
{
    if (a.B <= 0 || a.max_new <= 0) return hipSuccess;
    hipError_t e = launch1(ps_offsets, 1, kPsThreads, st, a);
    if (e != hipSuccess) return e;
    switch (g) {
    case 1: return launch_prompt_g<1>(a, st);
    case 2: return launch_prompt_g<2>(a, st);
    case 3: return launch_prompt_g<3>(a, st);
    case 4: return launch_prompt_g<4>(a, st);
    case 5: return launch_prompt_g<5>(a, st);
    case 6: return launch_prompt_g<6>(a, st);
    case 7: return launch_prompt_g<7>(a, st);
    case 8: return launch_prompt_g<8>(a, st);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace dkv
