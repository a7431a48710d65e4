// k_generation.hip -- the generation-phase policy of DiffKV (Sec. 4,
// Algorithm 1) for gfx950: once per decode step, after the step's append has
// put the newest token of every sequence into the high section, each table
// decides what happens to the token that has just left the recent window.
//
// Two launches on the caller's stream (three for very many tables):
//   gen_decide   one workgroup per table, one pass over the positions and
//                scores of both sections (16-byte loads, every load of a
//                thread in flight together): the candidate (the high token at
//                position N - 1 - W), the victim of each section (lowest
//                score, ties to the lowest position, among the tokens outside
//                the window), the action, and whether the low section needs
//                one more page;
//   gen_apply    one wave per table.  Every wave first derives the call's
//                allocation from all tables' page requests (total, its own
//                prefix, the all-or-nothing checks against the free region and
//                the table width), so no separate planning launch is needed;
//                above kGenFusedTables tables gen_scan does that once instead.
//                Then it reads the tokens it moves, removes a token from the
//                high section (the section's last token takes its slot, the
//                vacated slot is cleared) and writes a re-quantized token into
//                the low section (at its end, or over the low victim it evicts).
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
constexpr int kGenChunk = 4;           // groups of 4 tokens a thread loads before reducing them
constexpr int kGenFusedTables = 2048;  // up to this many tables each apply wave plans the allocation
constexpr int kGenScanThreads = 1024;
constexpr int kGenPlanIlp = 16;        // page requests a lane of an apply wave loads at once

// The victim search orders tokens by score (-0 == +0), then position, as one
// 64-bit key: the score's order-preserving image above the position.  Positions
// in a table are distinct, so the key names one token.
__device__ __forceinline__ uint32_t order_key(float s)
{
    uint32_t u = __float_as_uint(s);
    if (u == 0x80000000u) u = 0;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_score(uint64_t key)  // inverse of order_key (-0 reads +0)
{
    const uint32_t k = (uint32_t)(key >> 32);
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

constexpr uint64_t kNoKey = ~0ull;

template <int CTRL, int ROWS>
__device__ __forceinline__ uint64_t dpp_min_step(uint64_t x)
{
    // lanes without a source read the identity (all ones)
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)(uint32_t)x, CTRL, ROWS, 0xF, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)(uint32_t)(x >> 32), CTRL, ROWS, 0xF, false);
    const uint64_t y = ((uint64_t)hi << 32) | lo;
    return y < x ? y : x;
}

// Minimum over a full wave (row shifts, then row broadcasts; lane 63 holds it).
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x)
{
    x = dpp_min_step<0x111, 0xF>(x);  // row_shr:1
    x = dpp_min_step<0x112, 0xF>(x);  // row_shr:2
    x = dpp_min_step<0x114, 0xF>(x);  // row_shr:4
    x = dpp_min_step<0x118, 0xF>(x);  // row_shr:8
    x = dpp_min_step<0x142, 0xA>(x);  // row_bcast:15 into rows 1 and 3
    x = dpp_min_step<0x143, 0xC>(x);  // row_bcast:31 into rows 2 and 3
    return read_lane<unsigned long long>(x, kWave - 1);
}

// Threads 0-127 scan the high section, 128-255 the low one, 4 slots per load;
// a round covers kGenChunk groups of 4 per thread.  The first round's page IDs
// are loaded before the section lengths arrive (slots past a section's pages
// read -1 or a spare page, whose tokens the lengths then mask).  A section
// with no pages reads page 0 (never used: masked by the lengths).
constexpr int kGenHalf = kGenThreads / 2;

struct GenShared {
    uint64_t key[kGenWaves];  // each wave's lowest key (waves 0-1: high, 2-3: low)
    int32_t u[kGenWaves], id[kGenWaves];
    int32_t cu[2], cid[2];    // candidate found by a high wave (INT32_MAX: none)
    float cs[2];
};

__global__ __launch_bounds__(kGenThreads) void gen_decide(GenArgs a)
{
    __shared__ GenShared sh;
    const int t = blockIdx.x;
    const int P = a.p_max;
    const int32_t* row = a.page_table + (long long)t * P;
    const bool lo = threadIdx.x >= kGenHalf;  // this thread's section (uniform per wave)
    const int i = threadIdx.x & (kGenHalf - 1);
    const int tsh = lo ? 3 : 2;               // group of 4 slots -> page index
    // Loads are unconditional (clamped to a valid address, masked afterwards):
    // with no branch around them the compiler waits for each one alone.
    auto load_ids = [&](int jb, int* id) {
#pragma unroll
        for (int k = 0; k < kGenChunk; ++k) {
            const int pi = (jb + i + k * kGenHalf) >> tsh;
            const int pc_ = min(pi, P - 1);
            const int v = row[lo ? P - 1 - pc_ : pc_];
            id[k] = pi < P ? v : -1;
        }
    };
    int id[kGenChunk];
    load_ids(0, id);
    const int N = a.seq_len[t / a.Hkv];
    const int pc = N - 1 - a.window;
    const int len0 = a.len[2 * t], len1 = a.len[2 * t + 1];
    const int pg0 = a.pages[2 * t], pg1 = a.pages[2 * t + 1];
    int act = kGenNone, uh = 0, ul = 0, idh = -1, idl = -1, ido = -1;
    if (pc >= 0 && len0 > 0) {  // uniform over the workgroup
        // tokens read: this thread's section, clamped to the table width
        const int n = lo ? max(0, min(len1, P * kTLo)) : min(len0, P * kTHi);
        const int off_pos = lo ? a.off_pos[1] : a.off_pos[0];
        const int off_score = lo ? a.off_score[1] : a.off_score[0];
        const int smask = lo ? kTLo - 1 : kTHi - 1;
        // the last high token's page and the low section's append page, as
        // vector loads (a lane-varying zero) so no scalar-load wait holds back
        // the page loads below
        const int zv = (int)__builtin_amdgcn_mbcnt_lo(0u, 0u);
        const int plast = (len0 - 1) >> 4, papp = max(len1, 0) >> 5;
        const int v_last = row[min(plast, P - 1) + zv];
        const int v_app = row[P - 1 - min(papp, P - 1) + zv];
        uint64_t best = kNoKey;
        int bu = 0, bid = -1, cu = INT32_MAX, cid = -1;
        float cs = 0.0f;
        for (int jb = 0; 4 * jb < n; jb += kGenHalf * kGenChunk) {
            if (jb > 0) load_ids(jb, id);
            uint4 pv[kGenChunk], sv[kGenChunk];
            bool ok[kGenChunk];
#pragma unroll
            for (int k = 0; k < kGenChunk; ++k) {
                const int u0 = 4 * (jb + i + k * kGenHalf);
                ok[k] = u0 < n && id[k] >= 0 && id[k] < a.num_pages;
                const uint8_t* pg = a.pool + (long long)(ok[k] ? id[k] : 0) * a.page_bytes +
                                    (u0 & smask) * 4;
                pv[k] = *reinterpret_cast<const uint4*>(pg + off_pos);
                sv[k] = *reinterpret_cast<const uint4*>(pg + off_score);
            }
#pragma unroll
            for (int k = 0; k < kGenChunk; ++k) {
                if (!ok[k]) continue;
                const int u0 = 4 * (jb + i + k * kGenHalf);
                const uint32_t pp[4] = {pv[k].x, pv[k].y, pv[k].z, pv[k].w};
                const uint32_t ss[4] = {sv[k].x, sv[k].y, sv[k].z, sv[k].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int u = u0 + e;
                    const int32_t p = (int32_t)pp[e];
                    const bool in = u < n && p <= pc;
                    const uint64_t key = in ? (((uint64_t)order_key(__uint_as_float(ss[e])) << 32) | (uint32_t)p)
                                            : kNoKey;
                    if (key < best) {
                        best = key;
                        bu = u;
                        bid = id[k];
                    }
                    if (!lo && in && p == pc && u < cu) {
                        cu = u;
                        cid = id[k];
                        cs = __uint_as_float(ss[e]);
                    }
                }
            }
        }
        // per wave: the lowest key and the lane holding it; the candidate
        const int w = threadIdx.x / kWave;
        const uint64_t wmin = wave_min_u64(best);
        const uint64_t hit = __ballot(best == wmin);
        const int l0 = __ffsll((unsigned long long)hit) - 1;
        const int w_u = __builtin_amdgcn_readlane(bu, l0), w_id = __builtin_amdgcn_readlane(bid, l0);
        const uint64_t chit = __ballot(cu != INT32_MAX);
        const int lc = chit ? __ffsll((unsigned long long)chit) - 1 : 0;
        const int c_u = chit ? __builtin_amdgcn_readlane(cu, lc) : INT32_MAX;
        const int c_id = __builtin_amdgcn_readlane(cid, lc);
        const float c_sv = __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)__float_as_uint(cs), lc));
        if (lane_id() == 0) {
            sh.key[w] = wmin;
            sh.u[w] = w_u;
            sh.id[w] = w_id;
            if (!lo) {
                sh.cu[w] = c_u;
                sh.cid[w] = c_id;
                sh.cs[w] = c_sv;
            }
        }
        __syncthreads();
        const int wh = sh.key[1] < sh.key[0] ? 1 : 0, wl = sh.key[3] < sh.key[2] ? 3 : 2;
        const int wc = sh.cu[1] < sh.cu[0] ? 1 : 0;
        if (sh.cu[wc] != INT32_MAX) {
            const float thr_h = a.alpha_h / (float)N;
            const float thr_l = a.alpha_l / (float)N;
            const float c_s = sh.cs[wc];
            uh = sh.cu[wc];
            idh = sh.cid[wc];
            ul = len1;
            if (c_s >= thr_h) {
                // the candidate qualifies itself, so the high victim exists
                const float v_s = key_score(sh.key[wh]);
                if (v_s >= thr_l && v_s < thr_h) act = kGenHighVictimToLow;
                else if (v_s < thr_l) act = kGenHighVictimOut;
                uh = sh.u[wh];
                idh = sh.id[wh];
            } else if (c_s >= thr_l) {
                act = kGenCandToLow;
                if (sh.key[wl] != kNoKey && key_score(sh.key[wl]) < thr_l) {
                    ul = sh.u[wl];  // the low victim is evicted: its slot
                    ido = sh.id[wl];
                }
            } else {
                act = kGenCandOut;
            }
        }
        idl = plast < P ? v_last : -1;
        if (ul == len1) ido = papp < P ? v_app : -1;
    }
    if (threadIdx.x == 0) {
        if (t == 0) {  // ring pointers before the call, for the apply kernels
            a.flags->head_old = a.ring_ptr[0];
            a.flags->tail_old = a.ring_ptr[1];
        }
        const bool grows = act == kGenHighVictimToLow || (act == kGenCandToLow && ul == len1);
        const int need = (grows && len1 + 1 > pg1 * kTLo) ? 1 : 0;
        a.act[t] = make_int4(act, uh, ul, 0);
        a.ids[t] = make_int4(idh, idl, need ? -1 : ido, 0);
        a.demand[t] = need | (((long long)pg0 + pg1 + need > P) ? 2 : 0);
    }
}

// The allocation plan once, for many tables: ring offset of every table's
// page, the all-or-nothing checks, the new head.
__global__ __launch_bounds__(kGenScanThreads) void gen_scan(GenArgs a)
{
    __shared__ int32_t s_scan[kGenScanThreads / kWave];
    __shared__ uint32_t s_bits[kGenScanThreads / kWave];
    int carry = 0;
    uint32_t bad = 0;
    for (int t0 = 0; t0 < a.num_tables; t0 += kGenScanThreads) {
        const int t = t0 + threadIdx.x;
        const int d = t < a.num_tables ? a.demand[t] : 0;
        int tot;
        uint32_t b;
        const int off = block_excl_scan<int32_t>(d & 1, s_scan, &tot, (uint32_t)(d >> 1), s_bits, &b);
        if (t < a.num_tables) a.offset[t] = carry + off;
        carry += tot;
        bad |= b;
    }
    if (threadIdx.x == 0) {
        const long long head = a.flags->head_old, tail = a.flags->tail_old;
        uint32_t bits = bad ? DIFFKV_ST_TABLE_OVERFLOW : 0u;
        if (carry > tail - head) bits |= DIFFKV_ST_OUT_OF_PAGES;
        a.flags->ok = bits ? 0 : 1;
        if (bits) atomicOr(a.status, bits);
        else a.ring_ptr[0] = head + carry;
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
template <bool FUSED>
__global__ __launch_bounds__(kWave) void gen_apply(GenArgs a)
{
    const int t = blockIdx.x;
    const int lane = threadIdx.x;
    const int NT = a.num_tables;
    // Loads go out in two rounds, each unconditional (clamped addresses), so
    // none waits behind a branch: first the page requests and this table's
    // decision, then the page data and the ring entry of a new page.
    int dv[kGenPlanIlp];
    if constexpr (FUSED) {
#pragma unroll
        for (int k = 0; k < kGenPlanIlp; ++k) dv[k] = a.demand[min(lane + k * kWave, NT - 1)];
    }
    // this table's words as vector loads (a lane-varying zero in the index), so
    // they go out with the requests above instead of after the plan
    const int zv = (int)__builtin_amdgcn_mbcnt_lo(0u, 0u);
    const int4 d_v = a.act[t + zv];
    const int4 pid_v = a.ids[t + zv];
    const int dem_v = a.demand[t + zv];
    const int2 len_v = reinterpret_cast<const int2*>(a.len)[t + zv];
    const int pg1_v = a.pages[2 * t + 1 + zv];
    const long long head_v = (&a.flags->head_old)[zv];
    const long long tail_v = (&a.flags->tail_old)[zv];
    auto uni = [](int x) { return __builtin_amdgcn_readfirstlane(x); };
    // ---- the call's allocation: this table's ring offset, all-or-nothing
    int pre;
    if constexpr (FUSED) {
        int tot = 0, below = 0;
        uint32_t bad = 0;
        for (int base = 0; base < NT; base += kWave * kGenPlanIlp) {
            if (base > 0) {
#pragma unroll
                for (int k = 0; k < kGenPlanIlp; ++k) dv[k] = a.demand[min(base + lane + k * kWave, NT - 1)];
            }
#pragma unroll
            for (int k = 0; k < kGenPlanIlp; ++k) {
                const int i = base + lane + k * kWave;
                const int di = i < NT ? dv[k] : 0;
                tot += di & 1;
                below += (i < t) ? (di & 1) : 0;
                bad |= (uint32_t)di >> 1;
            }
        }
        tot = wave_isum_w<kWave>(tot);
        below = wave_isum_w<kWave>(below);
        bad = wave_or_u32(bad);
        const long long head = read_lane<long long>(head_v, 0);
        uint32_t bits = bad ? DIFFKV_ST_TABLE_OVERFLOW : 0u;
        if (tot > read_lane<long long>(tail_v, 0) - head) bits |= DIFFKV_ST_OUT_OF_PAGES;
        if (t == 0 && lane == 0) {
            if (bits) atomicOr(a.status, bits);
            else a.ring_ptr[0] = head + tot;
        }
        if (bits) return;
        pre = below;
    } else {
        if (!a.flags->ok) return;
        pre = a.offset[t];
    }
    // (uniform copies taken after the plan, so its loads are not held back)
    const int4 d = make_int4(uni(d_v.x), uni(d_v.y), uni(d_v.z), 0);
    const int4 pid = make_int4(uni(pid_v.x), uni(pid_v.y), uni(pid_v.z), 0);
    const int dem = uni(dem_v);
    const int len0 = uni(len_v.x), len1 = uni(len_v.y);
    const int pg1 = uni(pg1_v);
    const long long head = read_lane<long long>(head_v, 0);
    const int act = d.x;
    if (act == kGenNone) return;
    const int g = lane >> 4;
    const bool lead = (lane & 15) == 0;
    const int P = a.p_max;
    int32_t* row = a.page_table + (long long)t * P;
    const bool to_low = act == kGenHighVictimToLow || act == kGenCandToLow;
    const bool need = (dem & 1) != 0;  // this table takes a new low page
    const int uh = d.y;   // the token leaving the high section
    const int ul = d.z;   // the low index it is written to
    const bool replace = to_low && ul != len1;
    const int last = len0 - 1;
    const int idh = pid.x, idl = pid.y;
    // a damaged table (indices or page IDs out of range) is left alone
    if (uh < 0 || uh > last || idh < 0 || idh >= a.num_pages || idl < 0 || idl >= a.num_pages) return;
    if (to_low && (ul < 0 || ul > len1)) return;
    if (to_low && !need && (pid.z < 0 || pid.z >= a.num_pages)) return;
    if (need && (ul != pg1 * kTLo || pg1 < 0 || pg1 >= P)) return;
    uint8_t* hp = a.pool + (long long)idh * a.page_bytes;
    uint8_t* lp = a.pool + (long long)idl * a.page_bytes;
    const int hs = uh & 15, ls = last & 15, os = ul & 31;
    const bool moved = uh != last;
    const bool same = idh == idl;
    const bool fresh = to_low && !replace && os == 0;
    // the low rows are read from a page the decision named (a fresh page's are not read)
    uint8_t* orp = (to_low && !fresh) ? a.pool + (long long)pid.z * a.page_bytes : hp;

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

    // ---- read: the leaving token, the section's last token, the low rows, the ring
    const uint32_t h_k = *reinterpret_cast<const uint16_t*>(hp + kc + hs * 16);
    const uint32_t h_km = *kmeta(hp, 0, hs), h_vm = *vmeta(hp, 0, hs);
    const float h_s = *score(hp, 0, hs);
    const int32_t h_p = *posn(hp, 0, hs);
    const uint4 hrow = *vrows(hp, 0);
    const uint32_t l_k = *reinterpret_cast<const uint16_t*>(lp + kc + ls * 16);
    const uint32_t l_km = *kmeta(lp, 0, ls), l_vm = *vmeta(lp, 0, ls);
    const float l_s = *score(lp, 0, ls);
    const int32_t l_p = *posn(lp, 0, ls);
    const uint4 lrow_ld = *vrows(lp, 0);
    const uint4 orow_ld = *vrows(orp, to_low && !fresh ? 1 : 0);
    const int ring_id = a.ring[(head + pre) % a.num_pages];
    __syncthreads();
    const uint4 lrow = same ? hrow : lrow_ld;
    const uint4 orow = (to_low && !fresh) ? orow_ld : make_uint4(0, 0, 0, 0);
    int ido = pid.z;
    if (need) {
        ido = ring_id;
        if (ido < 0 || ido >= a.num_pages) return;  // a damaged ring
        if (lane == 0) {
            row[P - 1 - pg1] = ido;
            a.pages[2 * t + 1] = pg1 + 1;
        }
    }
    uint8_t* op = a.pool + (long long)(to_low ? ido : 0) * a.page_bytes;

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

hipError_t launch_generation(const GenArgs& g, hipStream_t st)
{
    if (g.num_tables == 0) return hipSuccess;
    hipError_t e = launch1(gen_decide, (unsigned)g.num_tables, kGenThreads, st, g);
    if (e != hipSuccess) return e;
    if (g.num_tables <= kGenFusedTables) return launch1(gen_apply<true>, (unsigned)g.num_tables, kWave, st, g);
    e = launch1(gen_scan, 1, kGenScanThreads, st, g);
    if (e != hipSuccess) return e;
    return launch1(gen_apply<false>, (unsigned)g.num_tables, kWave, st, g);
}

}  // namespace dkv
