// k_generation.hip -- the generation-phase policy of DiffKV (Sec. 4,
// Algorithm 1) for gfx950: once per decode step, after the step's append has
// put the newest token of every sequence into the high section, each table
// decides what happens to the token that has just left the recent window.
//
// Three launches on the caller's stream:
//   gen_decide   one workgroup per table: finds the candidate (the high token
//                at position N - 1 - W), the victim of the section the rule
//                needs (lowest score, ties to the lowest position, among the
//                tokens outside the window), and the action; a table whose
//                low section grows past its pages asks for one page;
//   alloc_plan + alloc_write (the allocation kernels): one prefix sum over
//                the tables' page requests, all-or-nothing against the free
//                region and the table width;
//   gen_apply    one wave per table, only when the allocation was accepted:
//                reads the tokens it moves, then removes a token from the high
//                section (the section's last token takes its slot, the vacated
//                slot is cleared) and writes a re-quantized token into the low
//                section (at its end, or over the low victim it evicts).
//
// Thresholds alpha/N are fp32 quotients, as in the prompt phase.  A token
// moving to the low section is dequantized per element as fma(s, code, z) in
// fp32, rounded to fp16 (round to nearest even) and quantized at the low
// precision with the append's quantizer, so the result is bit-exact with the
// definition.
#include "internal.hpp"
#include "quant.hpp"

namespace dkv {

constexpr int kGenThreads = 256;
constexpr int kGenWaves = kGenThreads / kWave;

// A token in the victim search: ordered by score (-0 == +0), then position,
// then section index (only equal positions, i.e. a damaged table, reach it).
struct Pick {
    uint32_t key;  // order-preserving image of the score
    int32_t pos;
    int32_t u;     // section index; INT32_MAX when no token qualifies
    float s;
};

__device__ __forceinline__ uint32_t order_key(float s)
{
    uint32_t u = __float_as_uint(s);
    if (u == 0x80000000u) u = 0;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ bool pick_less(const Pick& x, const Pick& y)
{
    if (x.key != y.key) return x.key < y.key;
    if (x.pos != y.pos) return x.pos < y.pos;
    return x.u < y.u;
}

__device__ __forceinline__ Pick no_pick() { return Pick{0xffffffffu, INT32_MAX, INT32_MAX, 0.0f}; }

// Minimum over the workgroup; every thread gets it.  `lds` holds kGenWaves
// entries and is free again on return.
__device__ __forceinline__ Pick block_min_pick(Pick x, Pick* lds)
{
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        Pick y;
        y.key = (uint32_t)__shfl_xor((int)x.key, o, kWave);
        y.pos = __shfl_xor(x.pos, o, kWave);
        y.u = __shfl_xor(x.u, o, kWave);
        y.s = __shfl_xor(x.s, o, kWave);
        if (pick_less(y, x)) x = y;
    }
    if (lane_id() == 0) lds[threadIdx.x / kWave] = x;
    __syncthreads();
    Pick r = lds[0];
#pragma unroll
    for (int i = 1; i < kGenWaves; ++i)
        if (pick_less(lds[i], r)) r = lds[i];
    __syncthreads();
    return r;
}

// Scans section `sec` of a table: the lowest-ordered token with position <=
// pc (`best`) and, with `cand`, the lowest index whose position is pc.
// Tokens on page IDs outside the pool are skipped (never read).
template <int SEC>
__device__ __forceinline__ void scan_section(const GenArgs& a, const int32_t* row, int len, int pc,
                                             Pick& best, Pick* cand)
{
    constexpr int T = SEC == DIFFKV_HIGH ? kTHi : kTLo;
    constexpr int SH = SEC == DIFFKV_HIGH ? 4 : 5;
    const int lim = a.p_max * T;
    if (len > lim) len = lim;
    for (int u = threadIdx.x; u < len; u += kGenThreads) {
        const int pi = u >> SH;
        const int id = SEC == DIFFKV_HIGH ? row[pi] : row[a.p_max - 1 - pi];
        if (id < 0 || id >= a.num_pages) continue;
        const uint8_t* pg = a.pool + (long long)id * a.page_bytes;
        const int slot = u & (T - 1);
        const int32_t p = reinterpret_cast<const int32_t*>(pg + a.off_pos[SEC])[slot];
        if (p > pc) continue;
        const float s = reinterpret_cast<const float*>(pg + a.off_score[SEC])[slot];
        const Pick c{order_key(s), p, u, s};
        if (pick_less(c, best)) best = c;
        if (cand && p == pc && u < cand->u) *cand = Pick{0u, 0, u, s};
    }
}

__global__ __launch_bounds__(kGenThreads) void gen_decide(GenArgs a)
{
    __shared__ Pick s_pick[kGenWaves];
    const int t = blockIdx.x;
    const int N = a.seq_len[t / a.Hkv];
    const int pc = N - 1 - a.window;
    const int len0 = a.len[2 * t], len1 = a.len[2 * t + 1];
    const int32_t* row = a.page_table + (long long)t * a.p_max;
    int act = kGenNone, uc = 0, uv = -1;
    if (pc >= 0 && len0 > 0) {  // uniform over the workgroup
        Pick best = no_pick(), cand = no_pick();
        scan_section<DIFFKV_HIGH>(a, row, len0, pc, best, &cand);
        cand = block_min_pick(cand, s_pick);
        best = block_min_pick(best, s_pick);
        if (cand.u != INT32_MAX) {
            const float thr_h = a.alpha_h / (float)N;
            const float thr_l = a.alpha_l / (float)N;
            uc = cand.u;
            if (cand.s >= thr_h) {
                // the candidate qualifies itself, so the high victim exists
                uv = best.u;
                if (best.s >= thr_l && best.s < thr_h) act = kGenHighVictimToLow;
                else if (best.s < thr_l) act = kGenHighVictimOut;
            } else if (cand.s >= thr_l) {
                act = kGenCandToLow;
                Pick lo = no_pick();
                scan_section<DIFFKV_LOW>(a, row, len1, pc, lo, nullptr);
                lo = block_min_pick(lo, s_pick);
                uv = (lo.u != INT32_MAX && lo.s < thr_l) ? lo.u : -1;
            } else {
                act = kGenCandOut;
            }
        }
    }
    if (threadIdx.x == 0) {
        const bool grows = act == kGenHighVictimToLow || (act == kGenCandToLow && uv < 0);
        a.act[t] = make_int4(act, uc, uv, 0);
        a.demand[2 * t] = 0;
        a.demand[2 * t + 1] = (grows && len1 + 1 > a.pages[2 * t + 1] * kTLo) ? 1 : 0;
    }
}

__device__ __forceinline__ uint64_t lo64(uint4 r) { return ((uint64_t)r.y << 32) | r.x; }
__device__ __forceinline__ uint64_t hi64(uint4 r) { return ((uint64_t)r.w << 32) | r.z; }
__device__ __forceinline__ uint4 rows_of(uint64_t r0, uint64_t r1)
{
    return make_uint4((uint32_t)r0, (uint32_t)(r0 >> 32), (uint32_t)r1, (uint32_t)(r1 >> 32));
}

// fp16 pair of s * code + z (one fma in fp32, then round to nearest even)
__device__ __forceinline__ uint32_t dequant_pair(uint32_t sz, uint32_t c0, uint32_t c1)
{
    const float s = h2f(sz & 0xffffu), z = h2f(sz >> 16);
    return f2h_rne(__builtin_fmaf(s, (float)c0, z)) | (f2h_rne(__builtin_fmaf(s, (float)c1, z)) << 16);
}

// One wave per table.  Lane l owns dimensions 2l and 2l+1 (group l/16): their
// K codes, the 16 bytes of V code rows 2l and 2l+1, and -- lanes 0, 16, 32,
// 48 -- the group's metadata words.  Every byte is read before any is written
// (a barrier separates the phases) and written at most once, except a fresh
// low page, whose clearing completes before the token is written.
__global__ __launch_bounds__(kWave) void gen_apply(GenArgs a)
{
    if (!a.flags->ok) return;
    const int t = blockIdx.x;
    const int4 d = a.act[t];
    const int act = d.x;
    if (act == kGenNone) return;
    const int lane = threadIdx.x;
    const int g = lane >> 4;
    const bool lead = (lane & 15) == 0;
    const int P = a.p_max;
    const int32_t* row = a.page_table + (long long)t * P;
    const int len0 = a.len[2 * t], len1 = a.len[2 * t + 1];
    const bool victim_high = act == kGenHighVictimToLow || act == kGenHighVictimOut;
    const bool to_low = act == kGenHighVictimToLow || act == kGenCandToLow;
    const bool replace = act == kGenCandToLow && d.z >= 0;
    const int uh = victim_high ? d.z : d.y;  // the token leaving the high section
    const int last = len0 - 1;
    const int ul = replace ? d.z : len1;     // the low index it is written to
    // a damaged table (indices or page IDs out of range) is left alone
    if (uh < 0 || uh > last || (last >> 4) >= P) return;
    const int idh = row[uh >> 4], idl = row[last >> 4];
    if (idh < 0 || idh >= a.num_pages || idl < 0 || idl >= a.num_pages) return;
    int ido = 0;
    if (to_low) {
        if (ul < 0 || (ul >> 5) >= P || (replace && ul >= len1)) return;
        ido = row[P - 1 - (ul >> 5)];
        if (ido < 0 || ido >= a.num_pages) return;
    }
    uint8_t* hp = a.pool + (long long)idh * a.page_bytes;
    uint8_t* lp = a.pool + (long long)idl * a.page_bytes;
    uint8_t* op = a.pool + (long long)ido * a.page_bytes;
    const int hs = uh & 15, ls = last & 15, os = ul & 31;
    const bool moved = uh != last;
    const bool same = idh == idl;
    const bool fresh = to_low && !replace && os == 0;

    // K code bytes of dims 2l, 2l+1 in a high page: chunk l/8, byte 2l mod 16
    const int kc = a.off_kcode[0] + (lane >> 3) * kTHi * 16 + ((2 * lane) & 15);
    auto kmeta = [&](uint8_t* pg, int sec, int s) {
        return reinterpret_cast<uint32_t*>(pg + a.off_kmeta[sec] + (s * kNG + g) * 4);
    };
    auto vmeta = [&](uint8_t* pg, int sec, int s) {
        return reinterpret_cast<uint32_t*>(pg + a.off_vmeta[sec] + (g * (sec ? kTLo : kTHi) + s) * 4);
    };
    auto score = [&](uint8_t* pg, int sec, int s) { return reinterpret_cast<float*>(pg + a.off_score[sec]) + s; };
    auto posn = [&](uint8_t* pg, int sec, int s) { return reinterpret_cast<int32_t*>(pg + a.off_pos[sec]) + s; };
    auto vrows = [&](uint8_t* pg, int sec) { return reinterpret_cast<uint4*>(pg + a.off_vcode[sec] + lane * 16); };

    // ---- read: the leaving token, the section's last token, the low rows
    const uint32_t h_k = *reinterpret_cast<const uint16_t*>(hp + kc + hs * 16);
    const uint32_t h_km = *kmeta(hp, 0, hs), h_vm = *vmeta(hp, 0, hs);
    const float h_s = *score(hp, 0, hs);
    const int32_t h_p = *posn(hp, 0, hs);
    const uint4 hrow = *vrows(hp, 0);
    uint32_t l_k = 0, l_km = 0, l_vm = 0;
    float l_s = 0.0f;
    int32_t l_p = 0;
    uint4 lrow = hrow;
    if (moved) {
        l_k = *reinterpret_cast<const uint16_t*>(lp + kc + ls * 16);
        l_km = *kmeta(lp, 0, ls);
        l_vm = *vmeta(lp, 0, ls);
        l_s = *score(lp, 0, ls);
        l_p = *posn(lp, 0, ls);
        if (!same) lrow = *vrows(lp, 0);
    }
    uint4 orow = make_uint4(0, 0, 0, 0);
    if (to_low && !fresh) orow = *vrows(op, 1);
    __syncthreads();

    // ---- re-quantize the leaving token at the low precision
    uint32_t ksz = 0, kc0 = 0, kc1 = 0, vsz = 0, vc0 = 0, vc1 = 0;
    if (to_low) {  // uniform: the quantizer reduces over 16-lane rows
        const uint32_t xk = dequant_pair(h_km, h_k & 0xffu, h_k >> 8);
        const uint32_t xv = dequant_pair(h_vm, (uint32_t)(lo64(hrow) >> (hs * 4)) & 15u,
                                         (uint32_t)(hi64(hrow) >> (hs * 4)) & 15u);
        quant_pair(xk, 15, ksz, kc0, kc1);
        quant_pair(xv, 3, vsz, vc0, vc1);
    }

    // ---- remove it from the high section: the last token takes its slot
    const uint64_t nib = 0xfull;
    uint64_t h0 = lo64(hrow) & ~(nib << (hs * 4)), h1 = hi64(hrow) & ~(nib << (hs * 4));
    if (moved) {
        *reinterpret_cast<uint16_t*>(hp + kc + hs * 16) = (uint16_t)l_k;
        if (lead) {
            *kmeta(hp, 0, hs) = l_km;
            *vmeta(hp, 0, hs) = l_vm;
        }
        if (lane == 0) {
            *score(hp, 0, hs) = l_s;
            *posn(hp, 0, hs) = l_p;
        }
        uint64_t m0 = lo64(lrow), m1 = hi64(lrow);
        h0 |= ((m0 >> (ls * 4)) & nib) << (hs * 4);
        h1 |= ((m1 >> (ls * 4)) & nib) << (hs * 4);
        if (same) {
            h0 &= ~(nib << (ls * 4));
            h1 &= ~(nib << (ls * 4));
        } else {
            m0 &= ~(nib << (ls * 4));
            m1 &= ~(nib << (ls * 4));
            *vrows(lp, 0) = rows_of(m0, m1);
        }
    }
    *vrows(hp, 0) = rows_of(h0, h1);
    *reinterpret_cast<uint16_t*>(lp + kc + ls * 16) = 0;
    if (lead) {
        *kmeta(lp, 0, ls) = 0;
        *vmeta(lp, 0, ls) = 0;
    }
    if (lane == 0) {
        *score(lp, 0, ls) = 0.0f;
        *posn(lp, 0, ls) = 0;
    }

    // ---- write it into the low section
    if (to_low) {
        if (fresh) {
            for (long long o = lane * 16; o < a.page_bytes; o += kWave * 16)
                *reinterpret_cast<uint4*>(op + o) = make_uint4(0, 0, 0, 0);
            __syncthreads();  // the clearing completes before the token's bytes land
        }
        // K codes: chunk g (dims 32g..32g+31), byte l mod 16 holds dims 2l, 2l+1
        op[a.off_kcode[1] + (g * kTLo + os) * 16 + (lane & 15)] = (uint8_t)(kc0 | (kc1 << 4));
        if (lead) {
            *kmeta(op, 1, os) = ksz;
            *vmeta(op, 1, os) = vsz;
        }
        if (lane == 0) {
            *score(op, 1, os) = h_s;
            *posn(op, 1, os) = h_p;
        }
        const uint64_t two = 3ull;
        const uint64_t o0 = (lo64(orow) & ~(two << (os * 2))) | ((uint64_t)vc0 << (os * 2));
        const uint64_t o1 = (hi64(orow) & ~(two << (os * 2))) | ((uint64_t)vc1 << (os * 2));
        *vrows(op, 1) = rows_of(o0, o1);
    }
    if (lane == 0) {
        a.len[2 * t] = len0 - 1;
        if (to_low && !replace) a.len[2 * t + 1] = len1 + 1;
    }
}

hipError_t launch_generation(const GenArgs& g, const AllocArgs& a, hipStream_t st)
{
    if (g.num_tables == 0) return hipSuccess;
    hipLaunchKernelGGL(gen_decide, dim3(g.num_tables), dim3(kGenThreads), 0, st, g);
    const hipError_t e = launch_alloc(a, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(gen_apply, dim3(g.num_tables), dim3(kWave), 0, st, g);
    return hipGetLastError();
}

}  // namespace dkv
