// k_memory.hip -- KV compressor, page allocation and free-list compaction
// kernels for gfx950 (DiffKV Sec. 4, Sec. 5.2, Sec. 5.3).
//
// The compressor runs as two launches on the caller's stream:
//   append_classify  one workgroup per table: classes its new tokens (quota
//                    form by a two-target radix select on the score bits, or
//                    the Algorithm 1 threshold comparisons), ranks the kept
//                    tokens of each section in position order;
//   append_commit    every workgroup derives the plan from the classify
//                    results (page demand per table, one prefix sum over
//                    tables, all-or-nothing check against the free region and
//                    the table width); workgroup 0 writes the new state, and
//                    all take (table, section, page) jobs: resolve the page ID
//                    (new pages from the table's ring region), quantize each
//                    token's 32-dim groups and write the page.
//   append_one       a call of at most one new token per sequence (a decode
//                    step) in one launch: classes, plan and page jobs, the
//                    state written by the last workgroup to finish.
// Allocation alone (alloc_plan + alloc_write) and compaction (compact_count,
// compact_apply) follow the same planning/coordination split:
// per-table work is fully parallel, one prefix sum gives every table a
// disjoint ring region.
#include "internal.hpp"
#include "quant.hpp"

namespace dkv {

// ---------------------------------------------------------------------------
// shared small pieces
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t score_key(float s)
{
    uint32_t u = __float_as_uint(s);
    if (u == 0x80000000u) u = 0;  // -0 == +0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

// ---------------------------------------------------------------------------
// append_classify: grid B * Hkv (table t = b * Hkv + h), block 512
// ---------------------------------------------------------------------------
constexpr int kClsThreads = 512;
static_assert(kClsThreads >= 2 * kWave, "two waves scan the digit histograms");
constexpr int kClsPer = 8;                       // tokens per thread in one tile
static_assert(4 * kClsPer <= 32, "a thread keeps four flag bits per token of a tile in one 32-bit word");
constexpr int kClsTile = kClsThreads * kClsPer;  // the first tile's scores stay in registers
constexpr uint32_t kOffSat = 1u << 30;           // row offsets saturate here (above any total_new)

// Sum over the wave of values <= kOffSat, saturating at kOffSat (result in lane 63).
__device__ __forceinline__ uint32_t wave_sat_sum(uint32_t x)
{
    x = min(x + dpp_u32<0x111, 0xF>(x), kOffSat);
    x = min(x + dpp_u32<0x112, 0xF>(x), kOffSat);
    x = min(x + dpp_u32<0x114, 0xF>(x), kOffSat);
    x = min(x + dpp_u32<0x118, 0xF>(x), kOffSat);
    x = min(x + dpp_u32<0x142, 0xA>(x), kOffSat);
    x = min(x + dpp_u32<0x143, 0xC>(x), kOffSat);
    return (uint32_t)__builtin_amdgcn_readlane((int)x, kWave - 1);
}

// Class of one new token against the two cuts of Sec. 4.2 (the high set, and
// the high + low set).  Per cut: a = above it outright, e = tied with the cut
// key (only the first `need` ties in position order are above it).
// mode 0: nothing above the cut, 1: every non-window token, 2: cut at key K.
struct Cuts {
    int mode[2];
    uint32_t K[2];
    int need[2];
};

__global__ __launch_bounds__(kClsThreads) void append_classify(AppendArgs a)
{
    const int H = a.Hkv;
    const int t = blockIdx.x;
    const int b = t / H, h = t - b * H;
    const int tid = threadIdx.x;
    __shared__ long long s_scan[kClsThreads / kWave];
    __shared__ int s_hist[2][2][256];  // [buffer][cut][digit]
    __shared__ int s_sel[4];
    __shared__ uint32_t s_off;

    if (t == 0 && tid == 0) {  // ring pointers before this call (the commit kernel moves head)
        a.flags->head_old = a.ring_ptr[0];
        a.flags->tail_old = a.ring_ptr[1];
    }
    for (int i = tid; i < 512; i += kClsThreads) (&s_hist[0][0][0])[i] = 0;
    // row offset of this sequence: sum of new_len over lower sequences (wave 0).
    // Entries are clamped to [0, kOffSat] and the sum saturates: a call with an
    // entry outside [0, max_new] fails anyway (that table flags itself).
    if (tid < kWave) {
        uint32_t part = 0;
        for (int i = tid; i < b; i += kWave) {
            const int v = a.new_len[i];
            part = min(part + (uint32_t)(v < 0 ? 0 : (v > (int)kOffSat ? (int)kOffSat : v)), kOffSat);
        }
        part = wave_sat_sum(part);
        if (tid == 0) s_off = part;
    }
    const int n = a.new_len[b];
    TState* ts = a.tstate + t;
    if (tid == 0) {  // section lengths and pages before this call
        ts->lold[0] = a.len[2 * t];
        ts->lold[1] = a.len[2 * t + 1];
        ts->pold[0] = a.pages[2 * t];
        ts->pold[1] = a.pages[2 * t + 1];
    }
    const bool quota = a.quota != nullptr;
    int q0 = 0, q1 = 0;
    if (quota) {
        q0 = a.quota[2 * t];
        q1 = a.quota[2 * t + 1];
    }
    __syncthreads();
    const long long off_b = s_off;
    const bool bad = n < 0 || n > a.max_new || off_b + n > a.total_new ||
                     (b == a.B - 1 && off_b + n != a.total_new);
    if (bad) {
        if (tid == 0) {  // the commit kernel turns n < 0 into DIFFKV_ST_BAD_INPUT
            ts->cnt[0] = ts->cnt[1] = 0;
            ts->n = -1;
        }
        return;
    }
    if (h == 0 && tid == 0) {
        a.sold[b] = a.seq_len[b];
        a.row_off[b] = (int)off_b;
    }
    const int W = a.window < n ? a.window : n;
    const int avail = n - W;
    const float* sc = a.score + off_b * H + h;
    int32_t* ord = a.ord + off_b * H + (long long)h * n;

    // first tile: thread tid holds tokens tid*e .. tid*e + e - 1
    const int n0 = n < kClsTile ? n : kClsTile;
    const int e = (n0 + kClsThreads - 1) / kClsThreads;
    float sr[kClsPer];
#pragma unroll
    for (int i = 0; i < kClsPer; ++i) {
        const int j = tid * e + i;
        sr[i] = (i < e && j < avail) ? sc[(long long)j * H] : 0.f;
    }

    Cuts c = {{0, 0}, {0, 0}, {0, 0}};
    float thr_h = 0.f, thr_l = 0.f;
    if (quota) {
        const int nh = q0 < 0 ? 0 : (q0 > avail ? avail : q0);
        const int nl = q1 < 0 ? 0 : (q1 > avail - nh ? avail - nh : q1);
        const int cut[2] = {nh, nh + nl};
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) c.mode[s2] = cut[s2] <= 0 ? 0 : (cut[s2] >= avail ? 1 : 2);
        if (c.mode[0] == 2 || c.mode[1] == 2) {
            // two-target radix select (the cut[s]-th largest key), 8-bit digits
            // from the top; histograms double-buffered so each digit costs two barriers
            uint32_t prefix[2] = {0, 0}, mask = 0;
            int kk[2] = {c.mode[0] == 2 ? cut[0] : 0, c.mode[1] == 2 ? cut[1] : 0};
            uint32_t kr[kClsPer];
#pragma unroll
            for (int i = 0; i < kClsPer; ++i) kr[i] = score_key(sr[i]);
#pragma unroll
            for (int pass = 0; pass < 4; ++pass) {
                const int shift = 24 - 8 * pass;
                int* hist = &s_hist[pass & 1][0][0];
#pragma unroll
                for (int i = 0; i < kClsPer; ++i) {
                    if (i < e && tid * e + i < avail) {
                        const uint32_t key = kr[i];
                        const uint32_t dig = (key >> shift) & 255u;
#pragma unroll
                        for (int s2 = 0; s2 < 2; ++s2)
                            if (kk[s2] > 0 && (key & mask) == prefix[s2]) atomicAdd(&hist[s2 * 256 + dig], 1);
                    }
                }
                for (int j = kClsTile + tid; j < avail; j += kClsThreads) {  // beyond the first tile
                    const uint32_t key = score_key(sc[(long long)j * H]);
                    const uint32_t dig = (key >> shift) & 255u;
#pragma unroll
                    for (int s2 = 0; s2 < 2; ++s2)
                        if (kk[s2] > 0 && (key & mask) == prefix[s2]) atomicAdd(&hist[s2 * 256 + dig], 1);
                }
                for (int i = tid; i < 512; i += kClsThreads) (&s_hist[(pass + 1) & 1][0][0])[i] = 0;  // the next digit's buffer
                __syncthreads();
                if (tid < 2 * kWave) {  // two waves find the cut bins with a scan from the top
                    const int s2 = tid / kWave, l = tid & (kWave - 1);
                    if (kk[s2] > 0) {
                        // lane l owns bins 255-4l .. 252-4l (descending)
                        int cb[4], tot4 = 0;
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            cb[q] = hist[s2 * 256 + 255 - 4 * l - q];
                            tot4 += cb[q];
                        }
                        const int incl = wave_incl_scan(tot4);
                        int above = incl - tot4;
                        if (above < kk[s2] && incl >= kk[s2]) {
#pragma unroll
                            for (int q = 0; q < 4; ++q) {
                                if (above + cb[q] >= kk[s2]) {
                                    s_sel[2 * s2] = 255 - 4 * l - q;
                                    s_sel[2 * s2 + 1] = above;
                                    break;
                                }
                                above += cb[q];
                            }
                        }
                    }
                }
                __syncthreads();
#pragma unroll
                for (int s2 = 0; s2 < 2; ++s2) {
                    if (kk[s2] > 0) {
                        prefix[s2] |= (uint32_t)s_sel[2 * s2] << shift;
                        kk[s2] -= s_sel[2 * s2 + 1];
                    }
                }
                mask |= 255u << shift;
            }
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
                if (c.mode[s2] == 2) {
                    c.K[s2] = prefix[s2];
                    c.need[s2] = kk[s2];  // tokens with key == K that still belong above the cut
                }
            }
        }
    } else {
        const float N = (float)(a.seq_len[b] + n);
        thr_h = a.alpha_h / N;
        thr_l = a.alpha_l / N;
    }

    // ---- classes and in-section ranks, in position order ------------------
    // One block scan per tile of four counters (16 bits each): above cut 0,
    // tied at cut 0, above cut 1, tied at cut 1.  The high set is the cut-0
    // set; the low set is the cut-1 set minus it (cut 1's set contains cut 0's),
    // so a token's rank in either follows from the four prefix counts.
    int c_a0 = 0, c_e0 = 0, c_a1 = 0, c_e1 = 0;
    for (int base = 0; base < n; base += kClsTile) {
        const int tn = n - base < kClsTile ? n - base : kClsTile;
        const int et = (tn + kClsThreads - 1) / kClsThreads;
        uint32_t fl = 0;  // 4 flag bits per token
        long long cnt = 0;
#pragma unroll
        for (int i = 0; i < kClsPer; ++i) {
            const int j = base + tid * et + i;
            if (i < et && j < n) {
                bool a0, e0, a1, e1;
                if (j >= avail) {  // recent window: always high
                    a0 = a1 = true;
                    e0 = e1 = false;
                } else {
                    const float s = base == 0 ? sr[i] : sc[(long long)j * H];
                    if (quota) {
                        const uint32_t key = score_key(s);
                        a0 = c.mode[0] == 1 || (c.mode[0] == 2 && key > c.K[0]);
                        e0 = c.mode[0] == 2 && key == c.K[0];
                        a1 = c.mode[1] == 1 || (c.mode[1] == 2 && key > c.K[1]);
                        e1 = c.mode[1] == 2 && key == c.K[1];
                    } else {
                        a0 = s >= thr_h;
                        a1 = a0 || s >= thr_l;
                        e0 = e1 = false;
                    }
                }
                fl |= ((uint32_t)a0 | ((uint32_t)e0 << 1) | ((uint32_t)a1 << 2) | ((uint32_t)e1 << 3)) << (4 * i);
                cnt += (long long)a0 | ((long long)e0 << 16) | ((long long)a1 << 32) | ((long long)e1 << 48);
            }
        }
        long long tot;
        const long long ex = block_excl_scan<long long>(cnt, s_scan, &tot);
        int r_a0 = c_a0 + (int)(ex & 0xffff), r_e0 = c_e0 + (int)((ex >> 16) & 0xffff);
        int r_a1 = c_a1 + (int)((ex >> 32) & 0xffff), r_e1 = c_e1 + (int)((ex >> 48) & 0xffff);
#pragma unroll
        for (int i = 0; i < kClsPer; ++i) {
            const int j = base + tid * et + i;
            if (i < et && j < n) {
                const uint32_t f = fl >> (4 * i);
                const bool a0 = f & 1, e0 = f & 2, a1 = f & 4, e1 = f & 8;
                const int rh = r_a0 + min(r_e0, c.need[0]);  // high tokens before this one
                const int rt = r_a1 + min(r_e1, c.need[1]);  // high + low tokens before it
                // (the ranks stay inside the table's n slots; the bounds tests only guard memory)
                if (a0 || (e0 && r_e0 < c.need[0])) {
                    if (rh < n) ord[rh] = j;
                } else if (a1 || (e1 && r_e1 < c.need[1])) {
                    if ((unsigned)(rt - rh) < (unsigned)n) ord[n - 1 - (rt - rh)] = j;
                }
                r_a0 += a0;
                r_e0 += e0;
                r_a1 += a1;
                r_e1 += e1;
            }
        }
        c_a0 += (int)(tot & 0xffff);
        c_e0 += (int)((tot >> 16) & 0xffff);
        c_a1 += (int)((tot >> 32) & 0xffff);
        c_e1 += (int)((tot >> 48) & 0xffff);
    }
    if (tid == 0) {
        const int hi = c_a0 + min(c_e0, c.need[0]);
        ts->cnt[0] = hi;
        ts->cnt[1] = c_a1 + min(c_e1, c.need[1]) - hi;
        ts->n = n;
    }
}

constexpr int kPlanThreads = 1024;

// ---------------------------------------------------------------------------
// append_commit: plan + quantize in one launch.
// Every workgroup first derives the call's plan from the per-table state the
// classify kernel left (new tokens per section, section lengths and pages
// before the call): page demand, page jobs, one prefix sum over tables (ring
// region and first job of every table), and the all-or-nothing checks.  So no
// workgroup waits on another: workgroup 0 writes the new state (lengths,
// pages, seq_len, ring head) while all of them -- reading only the snapshot
// -- take page jobs (table, section, page) in job order.
// ---------------------------------------------------------------------------
constexpr int kQuantWaves = 4;
constexpr int kCommitThreads = kQuantWaves * kWave;
constexpr int kTokIlp = 4;    // tokens a wave quantizes side by side
constexpr int kTokLoad = 8;   // tokens a wave loads up front: a 32-token page in one round of loads
static_assert(kTokLoad * kQuantWaves >= 32, "one round of loads per page");

struct TablePlan {
    int need[2], jobs[2];
    bool held_over;  // more pages than p_max after the call
};

// Pages hold a power of two of tokens, so page indices are shifts; tsh packs
// the two sections' shifts (high section in bits 0-7, low in bits 8-15).
__device__ __forceinline__ int page_of(int x, int sec, int tsh) { return x >> (sec ? tsh >> 8 : tsh & 255); }

__device__ __forceinline__ TablePlan table_plan(const TState& s, int P, int tsh)
{
    TablePlan tp;
    int held = 0;
#pragma unroll
    for (int sec = 0; sec < 2; ++sec) {
        const int T = 1 << (sec ? tsh >> 8 : tsh & 255);
        const int want = page_of(s.lold[sec] + s.cnt[sec] + T - 1, sec, tsh);
        tp.need[sec] = want > s.pold[sec] ? want - s.pold[sec] : 0;
        held += want > s.pold[sec] ? want : s.pold[sec];
        tp.jobs[sec] =
            s.cnt[sec] ? page_of(s.lold[sec] + s.cnt[sec] - 1, sec, tsh) - page_of(s.lold[sec], sec, tsh) + 1 : 0;
    }
    tp.held_over = held > P;
    return tp;
}

__device__ __forceinline__ long long plan_word(const TablePlan& tp)  // new pages | jobs << 32
{
    return (long long)(tp.need[0] + tp.need[1]) | ((long long)(tp.jobs[0] + tp.jobs[1]) << 32);
}

struct JobDesc {
    int t, sec, p, u0, u1, lold, n, tslot;
    long long ring_idx;  // ring position of a new page, -1 for a page already held
    // one-token append: the sequence's row offset and length before the call
    // come with the job (no classify results); otherwise `one` is 0
    int one, off_b, sold;
};

// Job `job` of table t (its plan tp, its exclusive prefix pre = new pages |
// jobs << 32): section, page, token range, table slot and, for a new page, the
// ring index (the table's ring region, high pages first).
__device__ __forceinline__ void describe_job(JobDesc& d, int t, const TState& s, const TablePlan& tp,
                                             long long pre, int job, int P, long long head_old, int tsh)
{
    const int lj = job - (int)(pre >> 32);
    const int sec = lj < tp.jobs[0] ? 0 : 1;
    const int TT = 1 << (sec ? tsh >> 8 : tsh & 255);
    const int p = page_of(s.lold[sec], sec, tsh) + (sec ? lj - tp.jobs[0] : lj);
    const int lo = s.lold[sec], hi_end = s.lold[sec] + s.cnt[sec];
    d.t = t;
    d.sec = sec;
    d.p = p;
    d.u0 = lo > p * TT ? lo : p * TT;
    d.u1 = hi_end < (p + 1) * TT ? hi_end : (p + 1) * TT;
    d.lold = lo;
    d.n = s.n;
    d.tslot = sec ? P - 1 - p : p;
    d.ring_idx = p < s.pold[sec] ? -1 : head_old + (pre & 0xffffffffll) + (sec ? tp.need[0] : 0) + (p - s.pold[sec]);
    d.one = 0;
    d.off_b = 0;
    d.sold = 0;
}

// One page job: resolve the page ID (a new page from the table's ring region),
// quantize the job's tokens and write them, zero a fresh page's unused bytes.
// Called by every thread of the workgroup after `s_job` is described.
// V code rows: a lane owns dims 2*lane, 2*lane+1, i.e. 2 * T * vb / 8 bytes (8,
// 16 or 32) of the V code segment, kept as up to eight 32-bit words.
constexpr int kRowWords = 8;

template <int KB, int VB, int TT>
__device__ __forceinline__ void commit_job_fmt(const AppendArgs& a, const JobDesc& s_job,
                                               uint32_t (*s_rows)[kWave][kRowWords])
{
    const int tid = threadIdx.x;
    const int P = a.p_max;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = wave_index();
    const int grp = lane >> 4;
    const int H = a.Hkv;
    const long long page_bytes = a.page_bytes;
    const int t = __builtin_amdgcn_readfirstlane(s_job.t);
    const int sec = __builtin_amdgcn_readfirstlane(s_job.sec);
    const int p = __builtin_amdgcn_readfirstlane(s_job.p);
    const int u0 = __builtin_amdgcn_readfirstlane(s_job.u0);
    const int u1 = __builtin_amdgcn_readfirstlane(s_job.u1);
    const int lold = __builtin_amdgcn_readfirstlane(s_job.lold);
    const int n = __builtin_amdgcn_readfirstlane(s_job.n);
    const int tslot = __builtin_amdgcn_readfirstlane(s_job.tslot);
    const long long ring_idx = s_job.ring_idx;
    const int b = t / H, h = t - b * H;
    constexpr int kb = KB, vb = VB;
    constexpr int rw = TT * VB / 32;  // 32-bit words per dimension row (1, 2 or 4)
    static_assert(2 * rw <= kRowWords, "value rows");
    // the page ID (every wave reads the one entry), beside the token loads
    int32_t* trow = a.page_table + (long long)t * P;
    int id = ring_idx < 0 ? trow[tslot] : a.ring[ring_idx % a.num_pages];
    id = __builtin_amdgcn_readfirstlane(id);
    if (tid == 0 && ring_idx >= 0) trow[tslot] = id;
    // this wave's tokens u0 + wave + kQuantWaves*i, all loaded up front; token
    // u of the section is row ord[u - lold] (high, rank order) or
    // ord[n - 1 - (u - lold)] (low ranks are stored from the back)
    const bool one = __builtin_amdgcn_readfirstlane(s_job.one) != 0;  // the job's one token is row 0 of its sequence
    const int off_b = one ? __builtin_amdgcn_readfirstlane(s_job.off_b) : a.row_off[b];
    const int sold = one ? __builtin_amdgcn_readfirstlane(s_job.sold) : a.sold[b];
    const int32_t* ord = a.ord + (long long)off_b * H + (long long)h * n;
    int jj[kTokLoad];
    uint32_t kx[kTokLoad], vx[kTokLoad];
#pragma unroll
    for (int i = 0; i < kTokLoad; ++i) {
        const int u = u0 + wave + i * kQuantWaves;
        const int r = (u < u1 ? u : u0) - lold;
        jj[i] = one ? 0 : (sec ? ord[n - 1 - r] : ord[r]);
    }
#pragma unroll
    for (int i = 0; i < kTokLoad; ++i) {
        const long long row = (long long)(off_b + jj[i]) * H + h;
        kx[i] = reinterpret_cast<const uint32_t*>(a.k + row * kD)[lane];
        vx[i] = reinterpret_cast<const uint32_t*>(a.v + row * kD)[lane];
    }
    const int off_kc = a.off_kcode[sec], off_km = a.off_kmeta[sec];
    const int off_vc = a.off_vcode[sec], off_vm = a.off_vmeta[sec];
    const bool fresh = (u0 == p * TT);
    const bool page_ok = (unsigned)id < (unsigned)a.num_pages;  // never write outside the pool
    uint8_t* pg = a.pool + (long long)(page_ok ? id : 0) * page_bytes;
    // a page being continued keeps its earlier tokens' V code bits
    uint32_t vold[kRowWords] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (wave == 0 && page_ok && !fresh) {
        const uint32_t* src = reinterpret_cast<const uint32_t*>(pg + off_vc) + lane * 2 * rw;
#pragma unroll
        for (int w = 0; w < kRowWords; ++w)
            if (w < 2 * rw) vold[w] = src[w];
    }
    if (page_ok && fresh) {
        // A fresh page reads as zero wherever no token lies: zero the token
        // slots from u1 on in every per-token segment and the page tail.
        // These bytes are disjoint from the ones the tokens write (V code
        // rows are written whole, zeros included), so the stores need no
        // ordering among themselves.
        const int s_end = u1 - p * TT, nfill = TT - s_end;
        const uint4 z4 = make_uint4(0, 0, 0, 0);
        for (int i = tid; i < (kb + 1) * nfill; i += kCommitThreads) {
            const int c = i / nfill, sl = s_end + (i - c * nfill);  // K chunks (kb per token), then K meta
            uint8_t* dst = c < kb ? pg + off_kc + (c * TT + sl) * 16 : pg + off_km + sl * 16;
            *reinterpret_cast<uint4*>(dst) = z4;
        }
        for (int i = tid; i < (kNG + 2) * nfill; i += kCommitThreads) {
            const int g = i / nfill, sl = s_end + (i - g * nfill);  // V meta groups, score, pos
            uint8_t* dst = g < kNG ? pg + off_vm + (g * TT + sl) * 4
                                   : pg + (g == kNG ? a.off_score[sec] : a.off_pos[sec]) + sl * 4;
            *reinterpret_cast<uint32_t*>(dst) = 0;
        }
        for (long long o = a.off_pos[sec] + (long long)TT * 4 + tid * 16; o < page_bytes; o += kCommitThreads * 16)
            *reinterpret_cast<uint4*>(pg + o) = z4;
    }
    uint32_t rows[kRowWords] = {0, 0, 0, 0, 0, 0, 0, 0};  // dim 2*lane: words 0 .. rw-1, dim 2*lane+1: rw ..
    // two passes of kTokIlp tokens: quantize side by side, then store
#pragma unroll
    for (int pass = 0; pass < kTokLoad / kTokIlp; ++pass) {
        const int base_u = u0 + wave + pass * kTokIlp * kQuantWaves;
        if (base_u >= u1) break;  // wave-uniform: no token of this wave left in the page
        uint32_t ksz[kTokIlp], kc0[kTokIlp], kc1[kTokIlp], vsz[kTokIlp], vc0[kTokIlp], vc1[kTokIlp];
#pragma unroll
        for (int i = 0; i < kTokIlp; ++i) {
            if (base_u + i * kQuantWaves < u1) {
                quant_pair(kx[pass * kTokIlp + i], (1 << kb) - 1, ksz[i], kc0[i], kc1[i]);
                quant_pair(vx[pass * kTokIlp + i], (1 << vb) - 1, vsz[i], vc0[i], vc1[i]);
            }
        }
#pragma unroll
        for (int i = 0; i < kTokIlp; ++i) {
            const int u = base_u + i * kQuantWaves;
            if (u >= u1) break;
            const int sl = u - p * TT;
            const int bit = sl * vb;
#pragma unroll
            for (int w = 0; w < kRowWords / 2; ++w) {
                if (w == (bit >> 5) && w < rw) {
                    rows[w] |= vc0[i] << (bit & 31);
                    rows[rw + w] |= vc1[i] << (bit & 31);
                }
            }
            if (!page_ok) continue;
            const long long row = (long long)(off_b + jj[pass * kTokIlp + i]) * H + h;
            if (kb == 8) {
                uint16_t* dst = reinterpret_cast<uint16_t*>(pg + off_kc + ((lane >> 3) * TT + sl) * 16 +
                                                            ((2 * lane) & 15));
                *dst = (uint16_t)(kc0[i] | (kc1[i] << 8));
            } else {
                uint8_t* dst = pg + off_kc + (grp * TT + sl) * 16 + (lane & 15);
                *dst = (uint8_t)(kc0[i] | (kc1[i] << 4));
            }
            if ((lane & 15) == 0) {
                *reinterpret_cast<uint32_t*>(pg + off_km + (sl * kNG + grp) * 4) = ksz[i];
                *reinterpret_cast<uint32_t*>(pg + off_vm + (grp * TT + sl) * 4) = vsz[i];
            }
            if (lane == 0) {
                reinterpret_cast<float*>(pg + a.off_score[sec])[sl] = a.score[row];
                reinterpret_cast<int32_t*>(pg + a.off_pos[sec])[sl] = sold + jj[pass * kTokIlp + i];
            }
        }
    }
    // the page's dimension-major V code rows: OR of the waves' bits (and of the
    // bits already on a page being continued), one store per dimension pair
#pragma unroll
    for (int w = 0; w < kRowWords; ++w) s_rows[wave][lane][w] = rows[w];
    __syncthreads();
    if (wave == 0 && page_ok) {
        uint32_t* dst = reinterpret_cast<uint32_t*>(pg + off_vc) + lane * 2 * rw;
#pragma unroll
        for (int w = 0; w < kRowWords; ++w) {
            uint32_t x = vold[w];
#pragma unroll
            for (int q = 0; q < kQuantWaves; ++q) x |= s_rows[q][lane][w];
            if (w < 2 * rw) dst[w] = x;
        }
    }
}

// One page job in the page format of its section (the layouts' formats; see
// kLayoutFmts), so that row widths and bit positions are constants.
__device__ __forceinline__ void commit_job(const AppendArgs& a, const JobDesc& s_job,
                                           uint32_t (*s_rows)[kWave][kRowWords])
{
    const int sec = __builtin_amdgcn_readfirstlane(s_job.sec);
    const int kb = a.kb[sec], vb = a.vb[sec], T = a.T[sec];
    if (kb == 8 && vb == 4) commit_job_fmt<8, 4, 16>(a, s_job, s_rows);
    else if (kb == 4 && vb == 2 && T == 32) commit_job_fmt<4, 2, 32>(a, s_job, s_rows);
    else if (kb == 8 && vb == 8) commit_job_fmt<8, 8, 16>(a, s_job, s_rows);
    else if (kb == 8 && vb == 2) commit_job_fmt<8, 2, 16>(a, s_job, s_rows);
    else if (kb == 4 && vb == 1) commit_job_fmt<4, 1, 32>(a, s_job, s_rows);
    else commit_job_fmt<4, 2, 16>(a, s_job, s_rows);
}

constexpr int kPlanKeep = 2;  // tables per thread whose state stays in registers

__global__ __launch_bounds__(kCommitThreads) void append_commit(AppendArgs a)
{
    const int tid = threadIdx.x;
    const int NT = a.B * a.Hkv;
    const int P = a.p_max;
    __shared__ long long s_scan[kCommitThreads / kWave];
    __shared__ uint32_t s_bits[kCommitThreads / kWave];
    __shared__ JobDesc s_job;
    __shared__ uint32_t s_rows[kQuantWaves][kWave][kRowWords];
    const long long head_old = a.flags->head_old, tail_old = a.flags->tail_old;

    // ---- the plan, in every workgroup (each thread a contiguous run of tables)
    const int per = (NT + kCommitThreads - 1) / kCommitThreads;
    const int t0 = tid * per;
    const int t1 = t0 + per < NT ? t0 + per : NT;
    // the run's first two tables stay in registers (static indices: no scratch)
    static_assert(kPlanKeep == 2, "for_tables visits two kept states");
    const TState st0 = a.tstate[min(t0, NT - 1)], st1 = a.tstate[min(t0 + 1, NT - 1)];
    auto for_tables = [&](auto&& f) {
        if (t0 < t1) f(t0, st0);
        if (t0 + 1 < t1) f(t0 + 1, st1);
        for (int t = t0 + 2; t < t1; ++t) f(t, a.tstate[t]);
    };
    long long packed = 0;
    uint32_t bits = 0;
    for_tables([&](int, const TState& s) {
        if (s.n < 0) {
            bits |= DIFFKV_ST_BAD_INPUT;
            return;
        }
        const TablePlan tp = table_plan(s, P, a.tsh);
        if (tp.held_over) bits |= DIFFKV_ST_TABLE_OVERFLOW;
        packed += plan_word(tp);
    });
    long long tot;
    uint32_t all_bits;
    const long long before = block_excl_scan<long long>(packed, s_scan, &tot, bits, s_bits, &all_bits);
    bits = all_bits & (DIFFKV_ST_BAD_INPUT | DIFFKV_ST_TABLE_OVERFLOW);
    const long long total_need = tot & 0xffffffffll;
    const int njobs = (int)(tot >> 32);
    if (bits & DIFFKV_ST_BAD_INPUT) bits = DIFFKV_ST_BAD_INPUT;
    else if (total_need > tail_old - head_old) bits |= DIFFKV_ST_OUT_OF_PAGES;
    if (bits) {  // all or nothing: no state, table or page changes
        if (blockIdx.x == 0 && tid == 0) atomicOr(a.status, bits);
        return;
    }

    // ---- workgroup 0: the state after the call -------------------------------
    if (blockIdx.x == 0) {
        for_tables([&](int t, const TState& s) {
            const TablePlan tp = table_plan(s, P, a.tsh);
#pragma unroll
            for (int sec = 0; sec < 2; ++sec) {
                a.len[2 * t + sec] = s.lold[sec] + s.cnt[sec];
                a.pages[2 * t + sec] = s.pold[sec] + tp.need[sec];
            }
        });
        for (int b = tid; b < a.B; b += kCommitThreads) a.seq_len[b] = a.sold[b] + a.new_len[b];
        if (tid == 0) a.ring_ptr[0] = head_old + total_need;
    }

    // ---- page jobs ------------------------------------------------------------
    for (int job = blockIdx.x; job < njobs; job += gridDim.x) {
        // the thread whose run of tables holds this job describes it
        const int run_first = (int)(before >> 32);
        if (run_first <= job && job < run_first + (int)(packed >> 32)) {
            long long pre = before;
            for_tables([&](int t, const TState& s) {
                if (s.n < 0) return;
                const TablePlan tp = table_plan(s, P, a.tsh);
                const int jo = (int)(pre >> 32);
                if (jo <= job && job < jo + tp.jobs[0] + tp.jobs[1])
                    describe_job(s_job, t, s, tp, pre, job, P, head_old, a.tsh);
                pre += plan_word(tp);
            });
        }
        __syncthreads();
        commit_job(a, s_job, s_rows);
        if (job + (int)gridDim.x < njobs) __syncthreads();  // s_job and s_rows are reused by the next job
    }
}

// ---------------------------------------------------------------------------
// Many tables: the plan once (append_plan, one workgroup), then the jobs
// (append_commit_planned).  Every commit workgroup redoing the plan costs
// O(tables) each; past kAppendPlanTables tables one planning launch is cheaper.
// The plan writes each table's exclusive prefix, a job -> table map and the
// state after the call; a commit workgroup reads its job's table directly.
// ---------------------------------------------------------------------------
constexpr int kPlanLdsTables = 8192;  // up to this many tables the job map is built from LDS
constexpr int kMapIlp = 4;            // jobs a thread maps side by side

__global__ __launch_bounds__(kPlanThreads) void append_plan(AppendArgs a)
{
    const int tid = threadIdx.x;
    const int NT = a.B * a.Hkv;
    const int P = a.p_max;
    __shared__ long long s_scan[kPlanThreads / kWave];
    __shared__ uint32_t s_bits[kPlanThreads / kWave];
    __shared__ int32_t s_jobs[kPlanLdsTables + 1];  // first job of every table, then njobs
    const long long head_old = a.flags->head_old, tail_old = a.flags->tail_old;
    const int per = (NT + kPlanThreads - 1) / kPlanThreads;
    const int t0 = tid * per;
    const int t1 = t0 + per < NT ? t0 + per : NT;
    // the first two tables' states, loaded together and unconditionally (a
    // thread past the last table reloads table NT - 1 and ignores it)
    const TState st0 = a.tstate[min(t0, NT - 1)], st1 = a.tstate[min(t0 + 1, NT - 1)];
    auto for_tables = [&](auto&& f) {
        if (t0 < t1) f(t0, st0);
        if (t0 + 1 < t1) f(t0 + 1, st1);
        for (int t = t0 + 2; t < t1; ++t) f(t, a.tstate[t]);
    };
    long long packed = 0;
    uint32_t bits = 0;
    for_tables([&](int, const TState& s) {
        if (s.n < 0) {
            bits |= DIFFKV_ST_BAD_INPUT;
            return;
        }
        const TablePlan tp = table_plan(s, P, a.tsh);
        if (tp.held_over) bits |= DIFFKV_ST_TABLE_OVERFLOW;
        packed += plan_word(tp);
    });
    long long tot;
    uint32_t all_bits;
    const long long before = block_excl_scan<long long>(packed, s_scan, &tot, bits, s_bits, &all_bits);
    bits = all_bits & (DIFFKV_ST_BAD_INPUT | DIFFKV_ST_TABLE_OVERFLOW);
    const long long total_need = tot & 0xffffffffll;
    const int njobs = (int)(tot >> 32);
    if (bits & DIFFKV_ST_BAD_INPUT) bits = DIFFKV_ST_BAD_INPUT;
    else if (total_need > tail_old - head_old) bits |= DIFFKV_ST_OUT_OF_PAGES;
    if (njobs > a.job_cap) bits |= DIFFKV_ST_BAD_INPUT;  // never with the host's bound; keeps the map in bounds
    if (bits) {  // all or nothing: no state, table or page changes
        if (tid == 0) {
            atomicOr(a.status, bits);
            a.flags->ok = 0;
        }
        return;
    }
    const bool lds_map = NT <= kPlanLdsTables;  // job map by binary search in LDS
    long long pre = before;
    for_tables([&](int t, const TState& s) {
        const TablePlan tp = table_plan(s, P, a.tsh);
        a.tplan[t] = pre;
        const int j0 = (int)(pre >> 32);
        if (lds_map) s_jobs[t] = j0;
        else
            for (int k = 0; k < tp.jobs[0] + tp.jobs[1]; ++k) a.job_table[j0 + k] = t;
#pragma unroll
        for (int sec = 0; sec < 2; ++sec) {
            a.len[2 * t + sec] = s.lold[sec] + s.cnt[sec];
            a.pages[2 * t + sec] = s.pold[sec] + tp.need[sec];
        }
        pre += plan_word(tp);
    });
    for (int b = tid; b < a.B; b += kPlanThreads) a.seq_len[b] = a.sold[b] + a.new_len[b];
    if (tid == 0) {
        a.ring_ptr[0] = head_old + total_need;
        a.flags->njobs = njobs;
        a.flags->ok = 1;
    }
    if (lds_map) {
        // job j belongs to the last table whose first job is <= j (tables without
        // jobs share their successor's prefix); every thread maps kMapIlp jobs side
        // by side with a fixed-length search
        if (tid == 0) s_jobs[NT] = njobs;
        __syncthreads();
        int steps = 0;
        while ((1 << steps) < NT + 1) ++steps;
        for (int j0 = tid; j0 < njobs; j0 += kPlanThreads * kMapIlp) {
            int lo[kMapIlp];
#pragma unroll
            for (int i = 0; i < kMapIlp; ++i) lo[i] = 0;
            for (int st = steps - 1; st >= 0; --st) {
#pragma unroll
                for (int i = 0; i < kMapIlp; ++i) {
                    const int mid = lo[i] + (1 << st);
                    if (mid <= NT && s_jobs[mid] <= j0 + i * kPlanThreads) lo[i] = mid;
                }
            }
#pragma unroll
            for (int i = 0; i < kMapIlp; ++i)
                if (j0 + i * kPlanThreads < njobs) a.job_table[j0 + i * kPlanThreads] = lo[i];
        }
    }
}

__global__ __launch_bounds__(kCommitThreads) void append_commit_planned(AppendArgs a)
{
    __shared__ JobDesc s_job;
    __shared__ uint32_t s_rows[kQuantWaves][kWave][kRowWords];
    if (!a.flags->ok) return;
    const int njobs = a.flags->njobs;
    const long long head_old = a.flags->head_old;
    for (int job = blockIdx.x; job < njobs; job += gridDim.x) {
        if (threadIdx.x == 0) {
            const int t = a.job_table[job];
            const TState s = a.tstate[t];
            describe_job(s_job, t, s, table_plan(s, a.p_max, a.tsh), a.tplan[t], job, a.p_max, head_old, a.tsh);
        }
        __syncthreads();
        commit_job(a, s_job, s_rows);
        if (job + (int)gridDim.x < njobs) __syncthreads();  // s_job and s_rows are reused by the next job
    }
}

// ---------------------------------------------------------------------------
// append_one: the whole append of a call in which every sequence takes at most
// one new token (max_new <= 1) over at most kAppendPlanTables tables -- a
// decode step -- in one launch, one workgroup per table.  One token needs no
// selection: inside the recent window it is high; in the quota form it is
// high when the high quota (clamped to the one token) is 1, else low when the
// low quota is; in the threshold form its score is compared with alpha / N as
// in append_classify.  So every workgroup derives every table's class, the
// plan (page demand, one prefix sum over tables) and the all-or-nothing
// verdict from the state before the call, then does its own table's page job
// (at most one: one token lies on one page).  No workgroup writes what another
// reads: the state after the call (lengths, pages, seq_len, ring head) is
// written by the workgroup that arrives last (arrive_count, on two levels of
// words), after every workgroup has read the state before the call.
// Workgroup 0 claims the arrival words with the call's tag as it starts
// (arrive_claim), so the arrivals, all at about the same time, count with one
// add each.
// ---------------------------------------------------------------------------
constexpr int kOnePer = (kAppendPlanTables + kCommitThreads - 1) / kCommitThreads;  // tables per thread
constexpr int kOneGroups = 16;  // first-level arrival words

inline bool append_one_call(const AppendArgs& a) { return a.max_new <= 1 && !append_planned(a.B, a.Hkv); }

__global__ __launch_bounds__(kCommitThreads) void append_one(AppendArgs a)
{
    const int tid = threadIdx.x;
    const int H = a.Hkv, B = a.B, NT = B * H, P = a.p_max;
    __shared__ long long s_scan[kCommitThreads / kWave];
    __shared__ uint32_t s_bits[kCommitThreads / kWave];
    __shared__ JobDesc s_job;
    __shared__ uint32_t s_rows[kQuantWaves][kWave][kRowWords];
    __shared__ int s_off[kAppendPlanTables];  // row offset of each sequence (new tokens of the lower ones)
    __shared__ int s_job_here, s_last;
    const unsigned long long tag = call_tag();
    if (blockIdx.x == 0 && tid <= kOneGroups)  // before any arrival, as a rule
        arrive_claim(tid < kOneGroups ? &a.flags->arrive_group[tid] : &a.flags->arrive, tag);
    const long long head_old = a.ring_ptr[0], tail_old = a.ring_ptr[1];
    if (tid == 0) s_job_here = 0;

    // ---- row offsets; each thread a run of sequences (B <= NT <= kAppendPlanTables)
    const int pb = (B + kCommitThreads - 1) / kCommitThreads;
    const int b0 = tid * pb;
    int nb[kOnePer];
    long long nsum = 0;
    uint32_t bad = 0;
#pragma unroll
    for (int i = 0; i < kOnePer; ++i) {
        nb[i] = 0;
        if (i < pb && b0 + i < B) {
            const int v = a.new_len[b0 + i];
            if (v < 0 || v > a.max_new) bad = 1;
            nb[i] = v < 0 ? 0 : (v > 1 ? 1 : v);
            nsum += nb[i];
        }
    }
    long long ntot;
    uint32_t any_bad;
    long long off = block_excl_scan<long long>(nsum, s_scan, &ntot, bad, s_bits, &any_bad);
#pragma unroll
    for (int i = 0; i < kOnePer; ++i) {
        if (i < pb && b0 + i < B) {
            s_off[b0 + i] = (int)off;
            off += nb[i];
        }
    }
    __syncthreads();
    // every count in [0, max_new] and their sum total_new: the classify
    // kernel's per-sequence row checks, taken for the whole call
    const bool bad_call = any_bad != 0 || ntot != a.total_new;

    // ---- classes and plans of every table; each thread a run of tables
    const int pt = (NT + kCommitThreads - 1) / kCommitThreads;
    const int t0 = tid * pt;
    const bool quota = a.quota != nullptr;
    TState st[kOnePer];
    long long packed = 0;
    uint32_t bits = 0;
#pragma unroll
    for (int i = 0; i < kOnePer; ++i) {
        TState& s = st[i];
        s.cnt[0] = s.cnt[1] = 0;
        s.lold[0] = s.lold[1] = s.pold[0] = s.pold[1] = 0;
        s.ring_off = 0;
        s.n = 0;
        const int t = t0 + i;
        if (i < pt && t < NT) {
            const int b = t / H, h = t - b * H;
            const int v = a.new_len[b];
            const int n = v < 0 ? 0 : (v > 1 ? 1 : v);
            s.n = n;
            s.lold[0] = a.len[2 * t];
            s.lold[1] = a.len[2 * t + 1];
            s.pold[0] = a.pages[2 * t];
            s.pold[1] = a.pages[2 * t + 1];
            if (n == 1 && !bad_call) {  // (a bad call's row offsets may lie past total_new)
                if (a.window >= 1) {
                    s.cnt[0] = 1;
                } else if (quota) {
                    const int q0 = a.quota[2 * t], q1 = a.quota[2 * t + 1];
                    const int nh = q0 < 0 ? 0 : (q0 > 1 ? 1 : q0);
                    const int nl = q1 < 0 ? 0 : (q1 > 1 - nh ? 1 - nh : q1);
                    s.cnt[0] = nh;
                    s.cnt[1] = nl;
                } else {
                    const float sc = a.score[(long long)s_off[b] * H + h];
                    const float N = (float)(a.seq_len[b] + n);
                    const float thr_h = a.alpha_h / N, thr_l = a.alpha_l / N;
                    const bool a0 = sc >= thr_h;
                    const bool a1 = a0 || sc >= thr_l;
                    s.cnt[0] = a0 ? 1 : 0;
                    s.cnt[1] = (a1 && !a0) ? 1 : 0;
                }
            }
            const TablePlan tp = table_plan(s, P, a.tsh);
            if (tp.held_over) bits |= DIFFKV_ST_TABLE_OVERFLOW;
            packed += plan_word(tp);
        }
    }
    long long tot;
    uint32_t all_bits;
    const long long before = block_excl_scan<long long>(packed, s_scan, &tot, bits, s_bits, &all_bits);
    bits = all_bits & DIFFKV_ST_TABLE_OVERFLOW;
    const long long total_need = tot & 0xffffffffll;
    if (bad_call) bits = DIFFKV_ST_BAD_INPUT;
    else if (total_need > tail_old - head_old) bits |= DIFFKV_ST_OUT_OF_PAGES;
    if (bits) {  // all or nothing: no state, table or page changes
        if (blockIdx.x == 0 && tid == 0) atomicOr(a.status, bits);
        return;
    }

    // ---- this workgroup's table: its page job, if its token is kept
    {
        long long pre = before;
#pragma unroll
        for (int i = 0; i < kOnePer; ++i) {
            const int t = t0 + i;
            if (i < pt && t < NT) {
                const TablePlan tp = table_plan(st[i], P, a.tsh);
                if (t == (int)blockIdx.x && tp.jobs[0] + tp.jobs[1] > 0) {
                    describe_job(s_job, t, st[i], tp, pre, (int)(pre >> 32), P, head_old, a.tsh);
                    const int b = t / H;
                    s_job.one = 1;
                    s_job.off_b = s_off[b];
                    s_job.sold = a.seq_len[b];
                    s_job_here = 1;
                }
                pre += plan_word(tp);
            }
        }
    }
    __syncthreads();
    if (s_job_here) commit_job(a, s_job, s_rows);

    // ---- the workgroup arriving last writes the state after the call
    __syncthreads();
    if (tid == 0) {
        // two levels, so that no word takes more than a few dozen concurrent
        // adds: workgroup j counts in group j % kOneGroups, the last of a
        // group in the top word
        const int ng = NT < kOneGroups ? NT : kOneGroups, g = (int)blockIdx.x % kOneGroups;
        const unsigned long long gsize = NT / kOneGroups + (g < NT % kOneGroups ? 1 : 0);
        bool last = false;
        if (arrive_count(&a.flags->arrive_group[g], tag) == gsize)
            last = arrive_count(&a.flags->arrive, tag) == (unsigned long long)ng;
        s_last = last;
    }
    __syncthreads();
    if (!s_last) return;
#pragma unroll
    for (int i = 0; i < kOnePer; ++i) {
        const int t = t0 + i;
        if (i < pt && t < NT) {
            const TablePlan tp = table_plan(st[i], P, a.tsh);
#pragma unroll
            for (int sec = 0; sec < 2; ++sec) {
                a.len[2 * t + sec] = st[i].lold[sec] + st[i].cnt[sec];
                a.pages[2 * t + sec] = st[i].pold[sec] + tp.need[sec];
            }
        }
    }
#pragma unroll
    for (int i = 0; i < kOnePer; ++i)  // no other workgroup writes seq_len: this is still the length before the call
        if (i < pb && b0 + i < B) a.seq_len[b0 + i] = a.seq_len[b0 + i] + nb[i];
    if (tid == 0) a.ring_ptr[0] = head_old + total_need;
}

// ---------------------------------------------------------------------------
// Allocation alone: alloc_plan (one workgroup) + alloc_write (wave per table)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kPlanThreads) void alloc_plan(AllocArgs a)
{
    const int tid = threadIdx.x;
    const int NT = a.num_tables;
    __shared__ long long s_scan[kPlanThreads / kWave + 1];
    __shared__ long long s_head, s_tail;
    if (tid == 0) {
        s_head = a.ring_ptr[0];
        s_tail = a.ring_ptr[1];
    }
    __syncthreads();
    long long total = 0;
    uint32_t flags = 0;
    for (int t = tid; t < NT; t += kPlanThreads) {
        int d0 = a.demand[2 * t], d1 = a.demand[2 * t + 1];
        if (d0 < 0 || d1 < 0) flags |= DIFFKV_ST_BAD_INPUT;
        total += (long long)(d0 > 0 ? d0 : 0) + (d1 > 0 ? d1 : 0);
        if ((long long)a.pages[2 * t] + a.pages[2 * t + 1] + d0 + d1 > a.p_max)
            flags |= DIFFKV_ST_TABLE_OVERFLOW;
    }
    uint32_t bits;
    const long long total_all = block_sum_or(total, flags, s_scan, &bits);
    if (total_all > s_tail - s_head) bits |= DIFFKV_ST_OUT_OF_PAGES;
    if (bits) {
        if (tid == 0) {
            atomicOr(a.status, bits);
            a.flags->ok = 0;
        }
        return;
    }
    long long carry = 0;
    for (int t0 = 0; t0 < NT; t0 += kPlanThreads) {
        const int t = t0 + tid;
        int d0 = 0, d1 = 0;
        if (t < NT) {
            d0 = a.demand[2 * t];
            d1 = a.demand[2 * t + 1];
        }
        long long tr;
        long long off = block_excl_scan<long long>(d0 + d1, s_scan, &tr) + carry;
        carry += tr;
        if (t < NT) {
            int4 st = make_int4(a.pages[2 * t], a.pages[2 * t + 1], (int)off, d0);
            a.tstate[t] = st;
            a.pages[2 * t] = st.x + d0;
            a.pages[2 * t + 1] = st.y + d1;
        }
    }
    if (tid == 0) {
        a.flags->head_old = s_head;
        a.flags->ok = 1;
        a.ring_ptr[0] = s_head + carry;
    }
}

__global__ __launch_bounds__(kWave) void alloc_write(AllocArgs a)
{
    if (!a.flags->ok) return;
    const int t = blockIdx.x;
    const int4 st = a.tstate[t];
    const int d1 = a.pages[2 * t + 1] - st.y;
    const long long base = a.flags->head_old + st.z;
    int32_t* row = a.page_table + (long long)t * a.p_max;
    for (int i = threadIdx.x; i < st.w; i += kWave) row[st.x + i] = a.ring[(base + i) % a.num_pages];
    for (int i = threadIdx.x; i < d1; i += kWave)
        row[a.p_max - 1 - (st.y + i)] = a.ring[(base + st.w + i) % a.num_pages];
}

// ---------------------------------------------------------------------------
// Compaction in two launches: compact_count (a wave per table; a workgroup
// counts a group of group_tables tables and writes the group's total) and
// compact_apply (a wave per table).  An apply wave finds its ring offset from
// the totals of the groups before its own plus the counts of the earlier
// tables of its group; groups are sized so that neither exceeds kMaxGroups
// values, i.e. one round of loads per lane, so no scan launch runs between the
// two at any table count.
// ---------------------------------------------------------------------------
__device__ __forceinline__ bool slot_live(int slot, int ph, int pl, int P)
{
    return slot < ph || slot >= P - pl;
}

constexpr int kCountWaves = 4;       // waves of a compact_count workgroup
constexpr int kCompactPlanIlp = 16;  // values a lane loads at once
constexpr int kMaxGroups = kWave * kCompactPlanIlp;

// ONE: one table per wave (group_tables == kCountWaves, up to kMaxGroups * kCountWaves tables)
template <bool ONE>
__global__ __launch_bounds__(kCountWaves * kWave) void compact_count(CompactArgs a)
{
    __shared__ int s_c[kCountWaves];
    const int w = wave_index();
    const int lane = threadIdx.x & (kWave - 1);
    const int P = a.p_max;
    const int GT = ONE ? kCountWaves : a.group_tables;
    const int t0 = blockIdx.x * GT;
    const int t1 = ONE ? min(a.num_tables, t0 + w + 1) : min(a.num_tables, t0 + GT);
    int gsum = 0;
    for (int t = t0 + w; t < t1; t += kCountWaves) {
        int ph = a.pages[2 * t], pl = a.pages[2 * t + 1];
        ph = ph < 0 ? 0 : (ph > P ? P : ph);
        pl = pl < 0 ? 0 : (pl > P - ph ? P - ph : pl);
        const uint8_t* rel = a.release + (long long)t * P;
        int c = 0;
        for (int s = lane; s < P; s += kWave) c += (rel[s] != 0 && slot_live(s, ph, pl, P));
        c = wave_isum_w<kWave>(c);
        if (lane == 0) a.count[t] = c;
        gsum += c;
    }
    if (lane == 0) s_c[w] = gsum;
    __syncthreads();
    if (threadIdx.x == 0) {
        int g = 0;
#pragma unroll
        for (int i = 0; i < kCountWaves; ++i) g += s_c[i];
        a.offset[blockIdx.x] = g;  // the group's total
        // the end pointer before the call
        if (blockIdx.x == 0) a.flags->tail_old = a.ring_ptr[1];
    }
}

// sum of v[0 .. n) and of v[0 .. below) over the wave, n <= kMaxGroups: all
// loads in flight together (unconditional, clamped to the last element)
__device__ __forceinline__ void wave_sum_prefix(const int32_t* v, int n, int below, int lane, int& tot, int& pre)
{
    int cv[kCompactPlanIlp];
#pragma unroll
    for (int k = 0; k < kCompactPlanIlp; ++k) cv[k] = v[min(lane + k * kWave, n - 1)];
#pragma unroll
    for (int k = 0; k < kCompactPlanIlp; ++k) {
        const int i = lane + k * kWave;
        const int c = i < n ? cv[k] : 0;
        tot += c;
        pre += i < below ? c : 0;
    }
}

// One wave per table; the live part of the row is staged in LDS (dynamic
// shared memory of 2*p_max ints) with each slot's release flag in the sign bit
// of its page ID (IDs are non-negative), so the squeeze writes in place and no
// global load sits between the ring stores (a byte load may alias them, so the
// compiler would keep each after the last store).  The wave of table 0
// advances the end pointer by the call's total.
template <bool ONE>
__global__ __launch_bounds__(kWave) void compact_apply(CompactArgs a)
{
    extern __shared__ int32_t s_row[];  // [0, P): old IDs (sign bit: released), [P, 2P): new row
    const int t = blockIdx.x;
    const int lane = threadIdx.x;
    const int NT = a.num_tables;
    const int P = a.p_max;
    int ph = a.pages[2 * t], pl = a.pages[2 * t + 1];
    const int len0 = a.len[2 * t], len1 = a.len[2 * t + 1];
    const long long tail_old = a.flags->tail_old;
    const int GT = ONE ? kCountWaves : a.group_tables;
    const int ng = (NT + GT - 1) / GT, g = t / GT, t0 = g * GT;
    int tot = 0, before = 0;
    wave_sum_prefix(a.offset, ng, g, lane, tot, before);  // the groups before g
    if (ONE) {
        if (lane < t - t0) before += a.count[t0 + lane];  // its group's tables before t
    } else {
        for (int i = t0 + lane; i < t; i += kWave) before += a.count[i];
    }
    ph = ph < 0 ? 0 : (ph > P ? P : ph);  // same clamp as compact_count
    pl = pl < 0 ? 0 : (pl > P - ph ? P - ph : pl);
    const int T0 = a.T[0], T1 = a.T[1];
    const uint8_t* rel = a.release + (long long)t * P;
    int32_t* row = a.page_table + (long long)t * P;
    int32_t* s_new = s_row + P;
    // the whole row, without waiting for the page counts: every load of the
    // wave is then in flight at once (slots outside the sections are not read)
    for (int s = lane; s < P; s += kWave) s_row[s] = row[s] | (rel[s] != 0 ? (int32_t)0x80000000 : 0);
    tot = wave_isum_w<kWave>(tot);
    const int my_off = wave_isum_w<kWave>(before);
    if (t == 0 && lane == 0) a.ring_ptr[1] = tail_old + tot;
    const long long n = a.num_pages;
    // ring position of this table's first released ID, reduced once; later
    // positions pass n at most once (rank < released slots <= pages in the pool)
    const long long start = (tail_old % n + my_off) % n;
    const uint64_t below = (1ull << lane) - 1ull;
    __syncthreads();
    auto ring_at = [&](int k) -> int32_t& {
        long long i = start + k;
        i = i >= n ? i - n : i;
        return a.ring[i];
    };
    // released IDs to the ring in ascending slot order; kept high IDs packed left
    int rank = 0, hi_keep = 0, drop0 = 0, drop1 = 0;
    for (int c = 0; c < ph; c += kWave) {
        const int s = c + lane;
        const bool live = s < ph;
        const int32_t id = live ? s_row[s] : 0;
        const bool r = live && id < 0;
        const uint64_t mr = __ballot(r);
        const uint64_t mk = __ballot(live && !r);
        if (r) {
            ring_at(rank + __popcll(mr & below)) = id & 0x7fffffff;
            int f = len0 - s * T0;
            drop0 += f < 0 ? 0 : (f > T0 ? T0 : f);
        }
        if (live && !r) s_new[hi_keep + __popcll(mk & below)] = id;
        rank += __popcll(mr);
        hi_keep += __popcll(mk);
    }
    for (int c = P - pl; c < P; c += kWave) {
        const int s = c + lane;
        const int32_t id = s < P ? s_row[s] : 0;
        const bool r = s < P && id < 0;
        const uint64_t mr = __ballot(r);
        if (r) {
            ring_at(rank + __popcll(mr & below)) = id & 0x7fffffff;
            int f = len1 - (P - 1 - s) * T1;
            drop1 += f < 0 ? 0 : (f > T1 ? T1 : f);
        }
        rank += __popcll(mr);
    }
    // kept low IDs packed right, in section order (section page k sits at slot P-1-k)
    int lo_keep = 0;
    for (int c = 0; c < pl; c += kWave) {
        const int k = c + lane;
        const int s = P - 1 - k;
        const int32_t id = k < pl ? s_row[s] : -1;
        const bool keep = k < pl && id >= 0;
        const uint64_t mk = __ballot(keep);
        if (keep) s_new[P - 1 - (lo_keep + __popcll(mk & below))] = id;
        lo_keep += __popcll(mk);
    }
    __syncthreads();
    for (int s = lane; s < ph; s += kWave) row[s] = s < hi_keep ? s_new[s] : -1;
    for (int s = P - pl + lane; s < P; s += kWave) row[s] = s >= P - lo_keep ? s_new[s] : -1;
    drop0 = wave_isum_w<kWave>(drop0);
    drop1 = wave_isum_w<kWave>(drop1);
    if (lane == 0) {
        a.pages[2 * t] = hi_keep;
        a.pages[2 * t + 1] = lo_keep;
        a.len[2 * t] = len0 - drop0;
        a.len[2 * t + 1] = len1 - drop1;
    }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
hipError_t launch_append(const AppendArgs& a, int grid_quant, hipStream_t st)
{
    if (append_one_call(a)) return launch1(append_one, (unsigned)(a.Hkv * a.B), kCommitThreads, st, a);
    hipError_t e = launch1(append_classify, (unsigned)(a.Hkv * a.B), kClsThreads, st, a);
    if (e != hipSuccess) return e;
    if (append_planned(a.B, a.Hkv)) {
        e = launch1(append_plan, 1, kPlanThreads, st, a);
        if (e != hipSuccess) return e;
        return launch1(append_commit_planned, (unsigned)grid_quant, kCommitThreads, st, a);
    }
    return launch1(append_commit, (unsigned)grid_quant, kCommitThreads, st, a);
}

hipError_t launch_alloc(const AllocArgs& a, hipStream_t st)
{
    hipError_t e = launch1(alloc_plan, 1, kPlanThreads, st, a);
    if (e != hipSuccess || a.num_tables == 0) return e;
    return launch1(alloc_write, (unsigned)a.num_tables, kWave, st, a);
}

hipError_t launch_compact(const CompactArgs& args, hipStream_t st)
{
    if (args.num_tables == 0) return hipSuccess;
    CompactArgs a = args;
    // tables per count group: at least one per wave, and few enough groups that an
    // apply wave sums them (and its group's earlier counts) in one round of loads
    const long long per = ((long long)a.num_tables + kMaxGroups - 1) / kMaxGroups;
    a.group_tables = (int)(per < kCountWaves ? kCountWaves : per);
    if (a.group_tables > kMaxGroups) return hipErrorInvalidValue;
    const size_t lds = (size_t)2 * a.p_max * sizeof(int32_t);
    const unsigned groups = (unsigned)((a.num_tables + a.group_tables - 1) / a.group_tables);
    const bool one = a.group_tables == kCountWaves;
    hipError_t e = one ? launch1(compact_count<true>, groups, kCountWaves * kWave, st, a)
                       : launch1(compact_count<false>, groups, kCountWaves * kWave, st, a);
    if (e != hipSuccess) return e;
    return one ? launch1(compact_apply<true>, (unsigned)a.num_tables, kWave, st, a, lds)
               : launch1(compact_apply<false>, (unsigned)a.num_tables, kWave, st, a, lds);
}

}  // namespace dkv
